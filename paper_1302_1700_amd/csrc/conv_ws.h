// Persistent, wave-specialised version of the fragment-batched convolution
// (same arithmetic and operand layout as conv_impl.h, vector path only).
//
// A workgroup has 8 waves: waves 0-3 run the matrix-core loop, waves 4-7 stage
// input windows.  The workgroup walks a list of tiles (tile = blockIdx.x,
// blockIdx.x + gridDim.x, ...) with two LDS window buffers: while the compute
// waves multiply tile i out of one buffer, the staging waves fill the other
// with tile i + 1's window, so the global-memory latency of the window, its
// zero fill and index arithmetic overlap the products instead of stalling
// them.  One workgroup-wide barrier per tile hands the buffers over.
#pragma once

#include "conv_impl.h"

namespace fs {
namespace conv {

struct TileGeo {
    bool valid;
    int q, fy, fx, hin, win, c0, twb, l0, lend, yfirst, R, Cc;
};

__device__ __forceinline__ TileGeo tile_geo(const ConvArgs &a, int tile)
{
    TileGeo T;
    T.valid = false;
    const int ntiles = a.nfrag * a.nbands * a.tiles_per_band;
    if (tile >= ntiles) return T;
    int bid = tile;
    const int t = bid % a.tiles_per_band;
    bid /= a.tiles_per_band;
    const int band = bid % a.nbands;
    T.q = bid / a.nbands;
    const int rem = T.q % a.F;
    T.fy = rem / a.Q;
    T.fx = rem - T.fy * a.Q;
    T.hin = a.ext.y[T.fy];
    T.win = a.ext.x[T.fx];
    const int hout = T.hin - a.k + 1, wout = T.win - a.k + 1;
    if (hout <= 0 || wout <= 0) return T;
    T.c0 = band * a.band_w;
    T.twb = min(a.band_w, wout - T.c0);
    if (T.twb <= 0) return T;
    const int npix = hout * T.twb;
    T.l0 = t * a.mt;
    if (T.l0 >= npix) return T;
    T.lend = min(T.l0 + a.mt, npix);
    T.yfirst = T.l0 / T.twb;
    T.R = (T.lend - 1) / T.twb - T.yfirst + a.k;
    T.Cc = T.twb + a.k - 1;
    T.valid = true;
    return T;
}

// Staging by the 256 threads of waves 4-7 (h = 0..255): the window rows
// [yfirst, yfirst + R) and columns [c0, c0 + Cc) of fragment q, all channels,
// zero outside the fragment's true size.
template <typename TC>
__device__ __forceinline__ void stage_window(const ConvArgs &a, const TileGeo &T, TC *dst, int h)
{
    constexpr int LPE = 16 / sizeof(TC);
    const TC *inp = reinterpret_cast<const TC *>(a.in) + (size_t)T.q * a.in_h * a.in_w * a.in_c;
    const int nvec = a.cin / LPE;
    const int per_row = T.Cc * nvec;
    const int total = T.R * per_row;
    const int CS = a.lds_cs;
    // batches of 8 loads in flight per thread before their LDS stores
    constexpr int UN = 8;
    for (int base = h; base < total; base += 256 * UN) {
        u4 val[UN];
        int dsto[UN];
#pragma unroll
        for (int u = 0; u < UN; ++u) {
            const int idx = base + u * 256;
            const int r = idx / per_row;
            const int rc = idx - r * per_row;
            const int c = rc / nvec;
            const int v = rc - c * nvec;
            const int gy = T.yfirst + r, gx = T.c0 + c;
            val[u] = u4{0u, 0u, 0u, 0u};
            if (idx < total && gy < T.hin && gx < T.win)
                val[u] = *reinterpret_cast<const u4 *>(inp + ((size_t)gy * a.in_w + gx) * a.in_c + v * LPE);
            dsto[u] = idx < total ? (r * T.Cc + c) * CS + v * LPE : -1;
        }
#pragma unroll
        for (int u = 0; u < UN; ++u)
            if (dsto[u] >= 0) *reinterpret_cast<u4 *>(dst + dsto[u]) = val[u];
    }
}

template <int MB, int NB, int WN, bool BF>
__global__ __launch_bounds__(512) void conv_frag_ws(ConvArgs a)
{
    using TC = typename Elem<BF>::T;
    constexpr int KSTEP = Elem<BF>::KSTEP;
    constexpr int LPE = KSTEP / 4;

    extern __shared__ __align__(16) unsigned char smem[];
    TC *buf[2] = {reinterpret_cast<TC *>(smem), reinterpret_cast<TC *>(smem + a.win_bytes)};
    float *red = reinterpret_cast<float *>(smem + 2 * a.win_bytes);

    const bool compute = threadIdx.x < 256;
    const int h = threadIdx.x - 256;

    int tile = blockIdx.x;
    TileGeo T = tile_geo(a, tile);
    if (!compute && T.valid) stage_window<TC>(a, T, buf[0], h);
    __syncthreads();

    const int lane = threadIdx.x & 63, wv = (threadIdx.x >> 6) & 3;
    const int wm = wv / WN, wn = wv - (wv / WN) * WN;
    const int lm = lane & 15, g = lane >> 4;
    const int nb0 = blockIdx.y * (WN * NB) + wn * NB;
    const u4 *wp = reinterpret_cast<const u4 *>(a.w) + (size_t)nb0 * 64 + lane;
    const size_t wstep = (size_t)a.nbt * 64;
    const int CS = a.lds_cs;
    const int ncc = a.cin / KSTEP;
    const int nsteps = a.ksteps;
    const int last = nsteps - 1;

    // tiles beyond a fragment's true size are skipped (not staged, not
    // computed); the walk ends past the last tile
    const int ntiles = a.nfrag * a.nbands * a.tiles_per_band;
    for (int it = 0; tile < ntiles; ++it) {
        const int ntile = tile + gridDim.x;
        const TileGeo N = tile_geo(a, ntile);
        TC *cur = buf[it & 1];
        if (!compute) {
            if (N.valid) stage_window<TC>(a, N, buf[(it + 1) & 1], h);
        } else if (T.valid) {
            const int Cc = T.Cc;
            int abase[MB];
#pragma unroll
            for (int i = 0; i < MB; ++i) {
                const int l = T.l0 + (wm * MB + i) * 16 + lm;
                if (l < T.lend) {
                    const int y = l / T.twb - T.yfirst, x = l - (l / T.twb) * T.twb;
                    abase[i] = (y * Cc + x) * CS + g * LPE;
                } else {
                    abase[i] = g * LPE;
                }
            }
            f4 acc[MB][NB];
#pragma unroll
            for (int i = 0; i < MB; ++i)
#pragma unroll
                for (int j = 0; j < NB; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

            auto mma = [&](const u4(&av)[MB], const u4(&bv)[NB]) {
                if constexpr (BF) {
#pragma unroll
                    for (int i = 0; i < MB; ++i)
#pragma unroll
                        for (int j = 0; j < NB; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                __builtin_bit_cast(bf8, av[i]), __builtin_bit_cast(bf8, bv[j]), acc[i][j], 0, 0, 0);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
#pragma unroll
                        for (int i = 0; i < MB; ++i)
#pragma unroll
                            for (int j = 0; j < NB; ++j)
                                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                    __uint_as_float(av[i][e]), __uint_as_float(bv[j][e]), acc[i][j], 0, 0, 0);
                }
            };
            int dy = 0, dx = 0, cc = 0;
            auto advance = [&]() {
                ++cc;
                const int w1 = cc == ncc;
                cc = w1 ? 0 : cc;
                dx += w1;
                const int w2 = dx == a.k;
                dx = w2 ? 0 : dx;
                dy += w2;
                return (dy * Cc + dx) * CS + cc * KSTEP;
            };
            u4 b0[NB], b1[NB], a0[MB], a1[MB];
#pragma unroll
            for (int j = 0; j < NB; ++j) b0[j] = wp[j * 64];
#pragma unroll
            for (int j = 0; j < NB; ++j) b1[j] = wp[(nsteps > 1 ? wstep : 0) + j * 64];
#pragma unroll
            for (int i = 0; i < MB; ++i) a0[i] = *reinterpret_cast<const u4 *>(cur + abase[i]);
            int off = 0;
            int s = 0;
            for (; s + 1 < nsteps; s += 2) {
                off = advance();  // step s + 1
#pragma unroll
                for (int i = 0; i < MB; ++i) a1[i] = *reinterpret_cast<const u4 *>(cur + abase[i] + off);
                __builtin_amdgcn_sched_barrier(0);
                mma(a0, b0);
                __builtin_amdgcn_sched_barrier(0);
                const size_t w2 = (size_t)min(s + 2, last) * wstep;
#pragma unroll
                for (int j = 0; j < NB; ++j) b0[j] = wp[w2 + j * 64];
                off = advance();  // step s + 2
                const int offa = s + 2 < nsteps ? off : 0;
#pragma unroll
                for (int i = 0; i < MB; ++i) a0[i] = *reinterpret_cast<const u4 *>(cur + abase[i] + offa);
                __builtin_amdgcn_sched_barrier(0);
                mma(a1, b1);
                __builtin_amdgcn_sched_barrier(0);
                const size_t w3 = (size_t)min(s + 3, last) * wstep;
#pragma unroll
                for (int j = 0; j < NB; ++j) b1[j] = wp[w3 + j * 64];
            }
            if (s < nsteps) mma(a0, b0);

            if (a.head_ncls == 0) {
                TC *outp = reinterpret_cast<TC *>(a.out) + (size_t)T.q * a.out_h * a.out_w * a.cout;
#pragma unroll
                for (int i = 0; i < MB; ++i) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int l = T.l0 + (wm * MB + i) * 16 + 4 * g + e;
                        if (l >= T.lend) continue;
                        const int y = l / T.twb, x = T.c0 + (l - (l / T.twb) * T.twb);
                        TC *row = outp + ((size_t)y * a.out_w + x) * a.cout;
#pragma unroll
                        for (int j = 0; j < NB; ++j) {
                            const int co = (nb0 + j) * 16 + lm;
                            if (co >= a.cout) continue;
                            float v = acc[i][j][e] + a.bias[co];
                            if (a.act == ACT_TANH) v = tanh_fast(v);
                            if constexpr (BF)
                                row[co] = f2bf(v);
                            else
                                row[co] = v;
                        }
                    }
                }
            } else {
                // fused last layer: per-lane partial class sums, reduced over
                // the 16 lanes of a row; the WN waves' parts go through LDS
                fused_head_partials<MB, NB, WN>(a, acc, nb0, wm, wn, lm, g, red);
            }
        }
        if (a.head_ncls > 0) {
            __syncthreads();  // partial sums of the compute waves are in LDS
            if (T.valid) fused_head_finish<WN>(a, T.q, T.fy, T.fx, T.l0, T.lend, T.twb, T.c0, red);
        }
        __syncthreads();  // window i consumed, window i + 1 staged
        tile = ntile;
        T = N;
    }
}

template <int MB, int NB, int WN, bool BF>
hipError_t launch_ws(const ConvArgs &a, int gx, int gy, hipStream_t s)
{
    auto kern = conv_frag_ws<MB, NB, WN, BF>;
    if (a.lds_bytes > 65536) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, a.lds_bytes);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3(gx, gy), dim3(512), a.lds_bytes, s, a);
    return hipGetLastError();
}

#define FS_CONV_TILES_WS(X)                                                                     \
    X(1, 1, 1) X(2, 1, 1) X(4, 1, 1) X(1, 2, 1) X(2, 2, 1) X(4, 2, 1) X(1, 3, 1) X(2, 3, 1)       \
    X(4, 3, 1) X(1, 4, 1) X(2, 4, 1) X(4, 4, 1) X(2, 7, 2) X(2, 4, 2) X(4, 4, 2) X(4, 7, 2)       \
    X(2, 8, 1) X(2, 2, 2)

template <bool BF>
hipError_t dispatch_ws(const ConvArgs &a, int mb, int nb, int wn, int gx, int gy, hipStream_t s)
{
#define FS_WS_CASE(M, N, W) \
    if (mb == M && nb == N && wn == W) return launch_ws<M, N, W, BF>(a, gx, gy, s);
    FS_CONV_TILES_WS(FS_WS_CASE)
#undef FS_WS_CASE
    return hipErrorInvalidValue;
}

}  // namespace conv
}  // namespace fs
