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
 * h_0 x w_0 x C window and runs the net on it the plain way, layer by layer,
 * in double precision:
 *   - convolutional layer (Section 2.1.1): valid cross-correlation of all
 *     input maps with k_y x k_x kernels, plus bias, then the activation; each
 *     map side shrinks by its kernel side minus one;
 *   - max-pooling layer (Section 2.1.2): non-overlapping k_y x k_x maxima;
 *     each map side must be divisible by the pool side and is divided by it.
 *     Pools with a stride s other than their size k (a generalisation the
 *     paper does not treat) take the maxima of the k x k windows at rows
 *     s*y and columns s_x*x: a side w gives (w - k) / s + 1 and must leave
 *     no remainder, (w - k) mod s = 0, which for s = k is the rule above;
 *   - fully connected layers (Section 2, "input, convolutional, max-pooling
 *     and fully-connected"): a dot product of the whole flattened map
 *     ([c][y][x] order) with each output neuron's weights, which is the
 *     convolution above with k equal to the map size;
 *   - the last layer's "softmax" activation turns the scores into class
 *     posterior probabilities (Section 1): exp(z - max z) / sum exp(z - max z).
 * Section 2 states everything for square maps and kernels and notes that
 * rectangular ones follow directly; a layer's k_x = 0 means k_x = k_y.
 * Weights are OIHW, weight[co][ci][dy][dx]; image is [B][H][W][C].
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>

enum { O_CONV = 0, O_POOL = 1, O_FC = 2 };
enum { O_ACT_NONE = 0, O_ACT_TANH = 1, O_ACT_SOFTMAX = 2 };

typedef struct {
    int kind, k, kx, c_in, c_out, act; /* k: rows of the kernel / pool; kx: columns (0: k) */
    const double *w; /* [c_out][c_in][k][kx] */
    const double *b; /* [c_out] */
    int s, sx;       /* pools: row and column stride (0: the pool's rows k; columns: s if given, else kx) */
} olayer;

static int kcols(const olayer *L) { return L->kx ? L->kx : L->k; }
static int srows(const olayer *L) { return L->s ? L->s : L->k; }
static int scols(const olayer *L) { return L->sx ? L->sx : (L->s ? L->s : kcols(L)); }

/* One layer on one patch.  `a` holds c_in maps of h x w as [c][y][x]; the
 * result goes to `o` and its size to *h_out x *w_out.  Returns 0 or -1 on a
 * shape the patch-level definition does not allow. */
static int run_layer(const olayer *L, const double *a, int h, int w, double *o, int *h_out, int *w_out)
{
    const int ky = L->k, kx = kcols(L);
    if (L->kind == O_POOL) {
        const int sy = srows(L), sx = scols(L);
        if (ky < 1 || kx < 1 || sy < 1 || sx < 1 || h < ky || w < kx || (h - ky) % sy || (w - kx) % sx) return -1;
        int ho = (h - ky) / sy + 1, wo = (w - kx) / sx + 1;
        for (int c = 0; c < L->c_in; ++c)
            for (int y = 0; y < ho; ++y)
                for (int x = 0; x < wo; ++x) {
                    double m = a[((size_t)c * h + sy * y) * w + sx * x];
                    for (int i = 0; i < ky; ++i)
                        for (int j = 0; j < kx; ++j) {
                            double v = a[((size_t)c * h + sy * y + i) * w + sx * x + j];
                            if (v > m) m = v;
                        }
                    o[((size_t)c * ho + y) * wo + x] = m;
                }
        *h_out = ho;
        *w_out = wo;
        return 0;
    }
    /* convolution, or a fully connected layer seen as one */
    if (ky < 1 || kx < 1 || ky > h || kx > w) return -1;
    if (L->kind == O_FC && (ky != h || kx != w)) return -1;
    int ho = h - (ky - 1), wo = w - (kx - 1);
    for (int co = 0; co < L->c_out; ++co)
        for (int y = 0; y < ho; ++y)
            for (int x = 0; x < wo; ++x) {
                double s = L->b ? L->b[co] : 0.0;
                for (int ci = 0; ci < L->c_in; ++ci)
                    for (int dy = 0; dy < ky; ++dy)
                        for (int dx = 0; dx < kx; ++dx)
                            s += L->w[(((size_t)co * L->c_in + ci) * ky + dy) * kx + dx]
                               * a[((size_t)ci * h + y + dy) * w + x + dx];
                if (L->act == O_ACT_TANH) s = tanh(s);
                o[((size_t)co * ho + y) * wo + x] = s;
            }
    *h_out = ho;
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
                         int B, int H, int W, int C, int h0, int w0,
                         const int *patches, long n, double *out)
{
    if (n_layers < 1 || h0 < 1 || w0 < 1 || h0 > H || w0 > W) return -1;
    /* largest map any layer holds, for the scratch buffers */
    size_t cap = (size_t)C * h0 * w0;
    {
        int h = h0, w = w0;
        for (int l = 0; l < n_layers; ++l) {
            const olayer *L = &layers[l];
            const int ky = L->k, kx = kcols(L);
            if (ky < 1 || kx < 1) return -1;
            if (L->kind == O_POOL) {
                const int sy = srows(L), sx = scols(L);
                if (sy < 1 || sx < 1 || h < ky || w < kx || (h - ky) % sy || (w - kx) % sx) return -1;
                h = (h - ky) / sy + 1;
                w = (w - kx) / sx + 1;
            } else {
                if (ky > h || kx > w) return -1;
                h -= ky - 1;
                w -= kx - 1;
            }
            size_t sz = (size_t)L->c_out * h * w;
            if (sz > cap) cap = sz;
        }
        if (h != 1 || w != 1) return -1;
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
            if (b < 0 || b >= B || Y < 0 || X < 0 || Y + h0 > H || X + w0 > W) { bad = 1; continue; }
            for (int c = 0; c < C; ++c)
                for (int y = 0; y < h0; ++y)
                    for (int x = 0; x < w0; ++x)
                        a[((size_t)c * h0 + y) * w0 + x] =
                            img[(((size_t)b * H + Y + y) * W + X + x) * C + c];
            int h = h0, w = w0;
            double *cur = a, *nxt = o;
            for (int l = 0; l < n_layers; ++l) {
                int ho, wo;
                if (run_layer(&layers[l], cur, h, w, nxt, &ho, &wo)) { bad = 1; break; }
                double *t = cur; cur = nxt; nxt = t; h = ho; w = wo;
            }
            if (layers[n_layers - 1].act == O_ACT_SOFTMAX) softmax(cur, n_out);
            memcpy(out + p * n_out, cur, n_out * sizeof(double));
        }
        free(a);
        free(o);
    }
    return bad ? -1 : 0;
}
