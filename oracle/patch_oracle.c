/*
 * Per-patch CPU oracle for the fragment-based image scan.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the definition the GPU scan must
 * reproduce; it is compiled and called by the test suite, the smoke check and
 * the benchmark's CPU-baseline leg, never by the library's product path.
 *
 * What it computes (Section 2.1, "Patch-level testing", with the outputs
 * wanted in Section 2.2: every window of size w_0 fully inside the image):
 * for each requested patch (image b, top-left row Y, column X) it crops the
 * w_0 x w_0 x C window and runs the net on it the plain way, layer by layer,
 * in double precision:
 *   - convolutional layer (Section 2.1.1): valid cross-correlation of all
 *     input maps with k x k kernels, plus bias, then the activation; the map
 *     size shrinks from w to w - (k - 1);
 *   - max-pooling layer (Section 2.1.2): non-overlapping k x k maxima; the
 *     map size must be divisible by k and becomes w / k;
 *   - fully connected layers (Section 2, "input, convolutional, max-pooling
 *     and fully-connected"): a dot product of the whole flattened map
 *     ([c][y][x] order) with each output neuron's weights, which is the
 *     convolution above with k equal to the map size;
 *   - the last layer's "softmax" activation turns the scores into class
 *     posterior probabilities (Section 1): exp(z - max z) / sum exp(z - max z).
 * Weights are OIHW, weight[co][ci][dy][dx]; image is [B][H][W][C].
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>

enum { O_CONV = 0, O_POOL = 1, O_FC = 2 };
enum { O_ACT_NONE = 0, O_ACT_TANH = 1, O_ACT_SOFTMAX = 2 };

typedef struct {
    int kind, k, c_in, c_out, act;
    const double *w; /* [c_out][c_in][k][k] */
    const double *b; /* [c_out] */
} olayer;

/* One layer on one patch.  `a` holds c_in maps of size w x w as [c][y][x];
 * the result goes to `o` and its size to *w_out.  Returns 0 or -1 on a shape
 * the patch-level definition does not allow. */
static int run_layer(const olayer *L, const double *a, int w, double *o, int *w_out)
{
    if (L->kind == O_POOL) {
        int k = L->k;
        if (k < 1 || w % k != 0) return -1;
        int wo = w / k;
        for (int c = 0; c < L->c_in; ++c)
            for (int y = 0; y < wo; ++y)
                for (int x = 0; x < wo; ++x) {
                    double m = a[((size_t)c * w + k * y) * w + k * x];
                    for (int i = 0; i < k; ++i)
                        for (int j = 0; j < k; ++j) {
                            double v = a[((size_t)c * w + k * y + i) * w + k * x + j];
                            if (v > m) m = v;
                        }
                    o[((size_t)c * wo + y) * wo + x] = m;
                }
        *w_out = wo;
        return 0;
    }
    /* convolution, or a fully connected layer seen as one */
    int k = L->k;
    if (k < 1 || k > w) return -1;
    if (L->kind == O_FC && k != w) return -1;
    int wo = w - (k - 1);
    for (int co = 0; co < L->c_out; ++co)
        for (int y = 0; y < wo; ++y)
            for (int x = 0; x < wo; ++x) {
                double s = L->b ? L->b[co] : 0.0;
                for (int ci = 0; ci < L->c_in; ++ci)
                    for (int dy = 0; dy < k; ++dy)
                        for (int dx = 0; dx < k; ++dx)
                            s += L->w[(((size_t)co * L->c_in + ci) * k + dy) * k + dx]
                               * a[((size_t)ci * w + y + dy) * w + x + dx];
                if (L->act == O_ACT_TANH) s = tanh(s);
                o[((size_t)co * wo + y) * wo + x] = s;
            }
    *w_out = wo;
    return 0;
}

static void softmax(double *z, int n)
{
    double m = z[0];
    for (int i = 1; i < n; ++i) if (z[i] > m) m = z[i];
    double s = 0.0;
    for (int i = 0; i < n; ++i) { z[i] = exp(z[i] - m); s += z[i]; }
    for (int i = 0; i < n; ++i) z[i] /= s;
}

/*
 * Run the net on `n` patches.  patches[3*p .. 3*p+2] = (b, Y, X), the image
 * index and the patch's top-left corner.  out[p * n_out + c] receives the last
 * layer's outputs (n_out = its c_out; the last map must be 1 x 1).
 * Returns 0, or -1 on an invalid net / patch (nothing is guaranteed in out).
 */
int oracle_patch_forward(const olayer *layers, int n_layers, const double *img,
                         int B, int H, int W, int C, int w0,
                         const int *patches, long n, double *out)
{
    if (n_layers < 1 || w0 < 1 || w0 > H || w0 > W) return -1;
    /* largest map any layer holds, for the scratch buffers */
    size_t cap = (size_t)C * w0 * w0;
    {
        int w = w0;
        for (int l = 0; l < n_layers; ++l) {
            const olayer *L = &layers[l];
            if (L->kind == O_POOL) { if (L->k < 1 || w % L->k) return -1; w /= L->k; }
            else { if (L->k < 1 || L->k > w) return -1; w -= L->k - 1; }
            size_t sz = (size_t)L->c_out * w * w;
            if (sz > cap) cap = sz;
        }
        if (w != 1) return -1;
    }
    int n_out = layers[n_layers - 1].c_out;
    int bad = 0;
#pragma omp parallel
    {
        double *a = (double *)malloc(cap * sizeof(double));
        double *o = (double *)malloc(cap * sizeof(double));
#pragma omp for schedule(dynamic, 1)
        for (long p = 0; p < n; ++p) {
            int b = patches[3 * p], Y = patches[3 * p + 1], X = patches[3 * p + 2];
            if (b < 0 || b >= B || Y < 0 || X < 0 || Y + w0 > H || X + w0 > W) { bad = 1; continue; }
            for (int c = 0; c < C; ++c)
                for (int y = 0; y < w0; ++y)
                    for (int x = 0; x < w0; ++x)
                        a[((size_t)c * w0 + y) * w0 + x] =
                            img[(((size_t)b * H + Y + y) * W + X + x) * C + c];
            int w = w0;
            double *cur = a, *nxt = o;
            for (int l = 0; l < n_layers; ++l) {
                int wo;
                if (run_layer(&layers[l], cur, w, nxt, &wo)) { bad = 1; break; }
                double *t = cur; cur = nxt; nxt = t; w = wo;
            }
            if (layers[n_layers - 1].act == O_ACT_SOFTMAX) softmax(cur, n_out);
            memcpy(out + p * n_out, cur, n_out * sizeof(double));
        }
        free(a);
        free(o);
    }
    return bad ? -1 : 0;
}
