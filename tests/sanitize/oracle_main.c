/* Driver for the sanitizer build of the per-patch oracle (oracle/patch_oracle.c):
 * every window of small square and rectangular nets, batches of two images,
 * and requests the oracle must refuse (a window past the image, a net whose
 * pool does not divide its map).  The layer record repeats the oracle's own. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

typedef struct {
    int kind, k, kx, c_in, c_out, act;
    const double *w;
    const double *b;
    int s, sx;
} olayer;

int oracle_patch_forward(const olayer *layers, int n_layers, const double *img, int B, int H, int W, int C, int h0,
                         int w0, const int *patches, long n, double *out);

static unsigned long long g_state = 1302;
static double rnd(void)
{
    g_state = g_state * 6364136223846793005ULL + 1442695040888963407ULL;
    return (double)(g_state >> 11) / 9007199254740992.0 - 0.5;
}

static double *fill(size_t n)
{
    double *p = malloc(n * sizeof(double));
    for (size_t i = 0; i < n; ++i) p[i] = rnd();
    return p;
}

static int run(olayer *L, int nl, int B, int H, int W, int C, int h0, int w0, int expect_ok)
{
    double *img = fill((size_t)B * H * W * C);
    const int ny = H - h0 + 1, nx = W - w0 + 1;
    long n = (long)B * ny * nx;
    int *pts = malloc(sizeof(int) * 3 * (n + 1));
    long p = 0;
    for (int b = 0; b < B; ++b)
        for (int y = 0; y < ny; ++y)
            for (int x = 0; x < nx; ++x) {
                pts[3 * p] = b;
                pts[3 * p + 1] = y;
                pts[3 * p + 2] = x;
                ++p;
            }
    const int nout = L[nl - 1].c_out;
    double *out = malloc(sizeof(double) * nout * (n + 1));
    int st = oracle_patch_forward(L, nl, img, B, H, W, C, h0, w0, pts, n, out);
    int ok = (st == 0) == (expect_ok != 0);
    if (st == 0)
        for (long i = 0; i < n * nout; ++i) ok = ok && isfinite(out[i]);
    /* one window past the image: refused */
    pts[3 * n] = 0;
    pts[3 * n + 1] = ny;
    pts[3 * n + 2] = 0;
    if (expect_ok) ok = ok && oracle_patch_forward(L, nl, img, B, H, W, C, h0, w0, pts + 3 * n, 1, out) == -1;
    free(img);
    free(pts);
    free(out);
    return ok;
}

int main(void)
{
    int ok = 1;
    /* conv 3x3 1->4 tanh, pool 2, conv 3x3 4->8 tanh, pool 2, fc 2x2 8->16 tanh, fc 16->2 softmax (w_0 = 14) */
    olayer sq[6] = {{0, 3, 0, 1, 4, 1, 0, 0}, {1, 2, 0, 4, 4, 0, 0, 0}, {0, 3, 0, 4, 8, 1, 0, 0},
                    {1, 2, 0, 8, 8, 0, 0, 0}, {2, 2, 0, 8, 16, 1, 0, 0}, {2, 1, 0, 16, 2, 2, 0, 0}};
    for (int i = 0; i < 6; ++i)
        if (sq[i].kind != 1) {
            const int kx = sq[i].kx ? sq[i].kx : sq[i].k;
            sq[i].w = fill((size_t)sq[i].c_out * sq[i].c_in * sq[i].k * kx);
            sq[i].b = fill(sq[i].c_out);
        }
    ok = ok && run(sq, 6, 2, 40, 33, 1, 14, 14, 1);
    /* a pool that does not divide its map: refused */
    ok = ok && run(sq, 6, 1, 40, 40, 1, 15, 15, 0);
    /* rectangular: conv 2x3 2->3 tanh, pool 2x3, conv 3x2 3->4 tanh, pool 1x2, fc 1x1 4->3 softmax (7 x 11) */
    olayer re[5] = {{0, 2, 3, 2, 3, 1, 0, 0}, {1, 2, 3, 3, 3, 0, 0, 0}, {0, 3, 2, 3, 4, 1, 0, 0},
                    {1, 1, 2, 4, 4, 0, 0, 0}, {2, 1, 1, 4, 3, 2, 0, 0}};
    for (int i = 0; i < 5; ++i)
        if (re[i].kind != 1) {
            re[i].w = fill((size_t)re[i].c_out * re[i].c_in * re[i].k * re[i].kx);
            re[i].b = fill(re[i].c_out);
        }
    ok = ok && run(re, 5, 2, 19, 23, 2, 7, 11, 1);
    /* pools with strides: conv 2x2 2->3 tanh, pool 3x2 stride 2x1, pool 2x2 stride 3, fc 1x2 3->2 softmax
     * (6 x 7) */
    olayer st[4] = {{0, 2, 2, 2, 3, 1, 0, 0, 0, 0}, {1, 3, 2, 3, 3, 0, 0, 0, 2, 1}, {1, 2, 2, 3, 3, 0, 0, 0, 3, 3},
                    {2, 1, 2, 3, 2, 2, 0, 0, 0, 0}};
    for (int i = 0; i < 4; i += 3) {
        st[i].w = fill((size_t)st[i].c_out * st[i].c_in * st[i].k * st[i].kx);
        st[i].b = fill(st[i].c_out);
    }
    ok = ok && run(st, 4, 2, 17, 15, 2, 6, 7, 1);
    for (int i = 0; i < 4; i += 3) {
        free((void *)st[i].w);
        free((void *)st[i].b);
    }
    for (int i = 0; i < 6; ++i) {
        free((void *)sq[i].w);
        free((void *)sq[i].b);
    }
    for (int i = 0; i < 5; ++i) {
        free((void *)re[i].w);
        free((void *)re[i].b);
    }
    if (!ok) {
        printf("oracle sanitizer run FAILED\n");
        return 1;
    }
    printf("oracle sanitizer run ok\n");
    return 0;
}
