// Fragmenting max-pool (Section 2.2.2).
//
// A k x k max-pooling layer turns every input fragment into k^2 output
// fragments, one per offset (o_x, o_y) in {0..k-1}^2.  Child pixel
// (xbar, ybar) is the maximum of the parent's pixels with
//   o_x + k*xbar <= x <= o_x + k*xbar + k - 1 and the same in y       (Eq. 5)
// and the child's size is div(s - o, k) per axis (Eqs. 6-7), never below 0.
// A rectangular k_y x k_x pool (Section 2: the square case generalizes
// directly) has k_y * k_x children and the same rules per axis.  A pool whose
// windows step by s instead of k (overlapping for s < k, with gaps for s > k;
// the paper's pools have s = k) has s_y * s_x children, child pixel xbar
// covering o_x + s*xbar .. o_x + s*xbar + k - 1, and holds
// div(n - o - k + s, s) pixels of a parent of n.
//
// One workgroup writes one row of one child: the row is a contiguous run of
// w_c * C elements, so stores are fully coalesced; the k parent rows it reads
// are contiguous runs too (neighbouring threads take neighbouring channel
// vectors, then neighbouring pixels), and the k^2 siblings that read the same
// parent rows are adjacent in the grid, so the overlap is served from cache.
// Max is exact in any precision: bf16 values are compared as floats and
// stored back unchanged.
#include "fs_internal.h"

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <type_traits>

namespace fs {
namespace {

typedef uint32_t u4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }
__device__ __forceinline__ uint16_t f2bf(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// V = elements per thread per access (4 x f32 or 8 x bf16 = 16 bytes; 1 = scalar)
template <bool BF, bool IN_F32, int V>
__global__ __launch_bounds__(256) void pool_frag(PoolArgs a)
{
    using TO = typename std::conditional<BF, uint16_t, float>::type;
    using TI = typename std::conditional<IN_F32, float, TO>::type;

    const int kk = a.sy * a.sx;
    // blockIdx.x = ((b * F + f) * sy*sx + o) * out_h + ybar, grouped so that
    // the children of a parent row band are neighbours:
    const int ybar = blockIdx.x % a.out_h;
    const int rest = blockIdx.x / a.out_h;
    const int o = rest % kk;
    const int p = rest / kk;            // parent batch index b * F + fy * Qx + fx
    const int oy = o / a.sx, ox = o - (o / a.sx) * a.sx;
    const int b = p / a.F;
    const int rem = p - b * a.F;
    const int fy = rem / a.Qx, fx = rem - (rem / a.Qx) * a.Qx;
    const int hp = a.ext.y[fy], wp = a.ext.x[fx];
    const int hc = hp - oy - a.ky >= 0 ? (hp - oy - a.ky) / a.sy + 1 : 0;
    const int wc = wp - ox - a.kx >= 0 ? (wp - ox - a.kx) / a.sx + 1 : 0;
    if (ybar >= hc || wc <= 0) return;

    // child batch index in the (fy * sy + oy, fx * sx + ox) grid (Qx * sx per row)
    const int Qc = a.Qx * a.sx;
    const size_t child = (size_t)b * a.F * kk + (size_t)(fy * a.sy + oy) * Qc + (fx * a.sx + ox);

    const TI *src = reinterpret_cast<const TI *>(a.in) +
                    ((size_t)p * a.in_h + (oy + a.sy * ybar)) * a.in_w * a.C;
    TO *dst = reinterpret_cast<TO *>(a.out) + (child * a.out_h + ybar) * a.out_w * a.C;
    const size_t prow = (size_t)a.in_w * a.C;

    const int nv = a.C / V;
    const int total = wc * nv;
    [[maybe_unused]] const int nparents = a.n_children / kk;
    for (int idx = threadIdx.x; idx < total; idx += 256) {
        const int xbar = idx / nv;
        const int cv = idx - xbar * nv;
        // the window's last parent row and column lie inside the parent's
        // true size; the child pixel inside the child's storage
        [[maybe_unused]] const int ly = oy + a.sy * ybar + a.ky - 1, lx = ox + a.sx * xbar + a.kx - 1;
        if (!FS_DBG_OK(a.dbg, p < nparents && ly < hp - a.dbg_shrink && lx < wp - a.dbg_shrink && ly < a.in_h &&
                                  lx < a.in_w, DBG_POOL_READ))
            continue;
        if (!FS_DBG_OK(a.dbg, child < (size_t)a.n_children && ybar < a.out_h && xbar < a.out_w, DBG_POOL_WRITE))
            continue;
        const size_t base = (size_t)(ox + a.sx * xbar) * a.C + cv * V;
        float m[V];
#pragma unroll
        for (int e = 0; e < V; ++e) m[e] = -INFINITY;
        for (int i = 0; i < a.ky; ++i) {
            for (int j = 0; j < a.kx; ++j) {
                const TI *s = src + i * prow + base + (size_t)j * a.C;
                if constexpr (V == 1) {
                    float v;
                    if constexpr (!BF || IN_F32) v = s[0]; else v = bf2f(s[0]);
                    m[0] = fmaxf(m[0], v);
                } else {
                    u4 raw = *reinterpret_cast<const u4 *>(s);
                    if constexpr (BF) {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            m[2 * e] = fmaxf(m[2 * e], bf2f((uint16_t)(raw[e] & 0xffffu)));
                            m[2 * e + 1] = fmaxf(m[2 * e + 1], bf2f((uint16_t)(raw[e] >> 16)));
                        }
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e) m[e] = fmaxf(m[e], __uint_as_float(raw[e]));
                    }
                }
            }
        }
        TO *d = dst + (size_t)xbar * a.C + cv * V;
        if constexpr (V == 1) {
            if constexpr (BF) d[0] = f2bf(m[0]); else d[0] = m[0];
        } else {
            u4 w;
            if constexpr (BF) {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    w[e] = (uint32_t)f2bf(m[2 * e]) | ((uint32_t)f2bf(m[2 * e + 1]) << 16);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) w[e] = __float_as_uint(m[e]);
            }
            *reinterpret_cast<u4 *>(d) = w;
        }
    }
}

// Row-band version for pool sizes 2..4 (the common case).  The k x k maxima
// at every position of the parent, M[y][x] = max_{i,j<k} P[y+i][x+j], are
// exactly the children's pixels: M[y][x] is pixel (y div k, x div k) of the
// child with offset (x mod k, y mod k).  A thread owns one (x, channel vector)
// column of a band of RB rows of M: it walks the parent rows once, keeps the
// last k horizontal maxima in registers, and writes each M row to its child.
// So a parent element is fetched from memory once (its k horizontal
// neighbours share it through the cache) and every child row is written with
// contiguous stores; the k^2 siblings no longer re-read the parent.
template <int K, int RB, bool BF, bool IN_F32, int V>
__global__ __launch_bounds__(256) void pool_frag_rows(PoolArgs a, int nbands, int nchunks, int nblocks)
{
    using TO = typename std::conditional<BF, uint16_t, float>::type;
    using TI = typename std::conditional<IN_F32, float, TO>::type;
    // Workgroups are dealt to the 8 XCDs round-robin; renumber them so each
    // XCD takes a contiguous run of bands, and the K - 1 parent rows that
    // neighbouring bands share are read from that XCD's L2 rather than twice
    // from HBM (the grid is padded to a multiple of 8; the padding exits).
    int bid = (blockIdx.x % 8) * (gridDim.x / 8) + blockIdx.x / 8;
    if (bid >= nblocks) return;
    const int chunk = bid % nchunks;
    bid /= nchunks;
    const int band = bid % nbands;
    const int p = bid / nbands;  // parent batch index b * F + fy * Qx + fx
    const int b = p / a.F;
    const int rem = p - b * a.F;
    const int fy = rem / a.Qx, fx = rem - (rem / a.Qx) * a.Qx;
    const int hp = a.ext.y[fy], wp = a.ext.x[fx];
    const int nv = a.C / V;
    const int pi = chunk * 256 + threadIdx.x;
    const int x = pi / nv, cv = pi - (pi / nv) * nv;
    const int y0 = band * RB;
    const int yend = min(y0 + RB, hp - K + 1);  // M rows [y0, yend)
    if (x > wp - K || y0 >= yend) return;
    // the parent rows and columns the thread reads lie inside the parent's true size
    [[maybe_unused]] const int lastrow = min(y0 + RB + K - 2, hp - 1), lastcol = x + K - 1;
    if (!FS_DBG_OK(a.dbg, p < a.n_children / (K * K) && lastrow < hp - a.dbg_shrink && lastcol < wp - a.dbg_shrink &&
                              lastrow < a.in_h && lastcol < a.in_w, DBG_POOL_READ))
        return;

    const TI *src = reinterpret_cast<const TI *>(a.in) + (size_t)p * a.in_h * a.in_w * a.C + (size_t)x * a.C + cv * V;
    const size_t prow = (size_t)a.in_w * a.C;
    const int Qc = a.Qx * K;
    const size_t cbase = (size_t)b * a.F * K * K;
    TO *out = reinterpret_cast<TO *>(a.out);

    // The RB + K - 1 parent rows this thread reads, every load issued before
    // any maximum is taken (rows past the band's last are clamped to the
    // fragment's last row: in bounds, and unused), so a thread has all its
    // loads in flight at once.
    u4 raw[RB + K - 1][K];
    float sc[RB + K - 1][K];
#pragma unroll
    for (int r = 0; r < RB + K - 1; ++r) {
        const TI *row = src + (size_t)min(y0 + r, hp - 1) * prow;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            if constexpr (V == 1) {
                if constexpr (!BF || IN_F32)
                    sc[r][j] = row[(size_t)j * a.C];
                else
                    sc[r][j] = bf2f(row[(size_t)j * a.C]);
            } else {
                raw[r][j] = *reinterpret_cast<const u4 *>(row + (size_t)j * a.C);
            }
        }
    }
    // horizontal maxima of each row, then the K-row maxima
    float h[RB + K - 1][V];
#pragma unroll
    for (int r = 0; r < RB + K - 1; ++r) {
#pragma unroll
        for (int e = 0; e < V; ++e) h[r][e] = -INFINITY;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            if constexpr (V == 1) {
                h[r][0] = fmaxf(h[r][0], sc[r][j]);
            } else if constexpr (BF) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    h[r][2 * e] = fmaxf(h[r][2 * e], bf2f((uint16_t)(raw[r][j][e] & 0xffffu)));
                    h[r][2 * e + 1] = fmaxf(h[r][2 * e + 1], bf2f((uint16_t)(raw[r][j][e] >> 16)));
                }
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) h[r][e] = fmaxf(h[r][e], __uint_as_float(raw[r][j][e]));
            }
        }
    }
    const int ox = x % K, xbar = x / K;
#pragma unroll
    for (int i = 0; i < RB; ++i) {
        const int y = y0 + i;
        if (y >= yend) break;
        float m[V];
#pragma unroll
        for (int e = 0; e < V; ++e) {
            m[e] = h[i][e];
#pragma unroll
            for (int t = 1; t < K; ++t) m[e] = fmaxf(m[e], h[i + t][e]);
        }
        const int oy = y % K, ybar = y / K;
        const size_t child = cbase + (size_t)(fy * K + oy) * Qc + (fx * K + ox);
        // inside the child: (s - o) div K pixels per axis of a parent of s (Eqs. 6-7)
        if (!FS_DBG_OK(a.dbg,
                       child < (size_t)a.n_children && ybar < (hp - oy) / K - a.dbg_shrink &&
                           xbar < (wp - ox) / K - a.dbg_shrink && ybar < a.out_h && xbar < a.out_w,
                       DBG_POOL_WRITE))
            continue;
        TO *d = out + ((child * a.out_h + ybar) * a.out_w + xbar) * a.C + cv * V;
        if constexpr (V == 1) {
            if constexpr (BF) d[0] = f2bf(m[0]); else d[0] = m[0];
        } else {
            u4 w;
            if constexpr (BF) {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    w[e] = (uint32_t)f2bf(m[2 * e]) | ((uint32_t)f2bf(m[2 * e + 1]) << 16);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) w[e] = __float_as_uint(m[e]);
            }
            *reinterpret_cast<u4 *>(d) = w;
        }
    }
}

template <int K, int RB, bool BF, bool IN_F32, int V>
hipError_t go_rows_rb(const PoolArgs &a, hipStream_t s)
{
    const int nv = a.C / V;
    const int nbands = (a.in_h + RB - 1) / RB;
    const int nchunks = (a.in_w * nv + 255) / 256;
    const long long grid = (long long)a.n_children / (K * K) * nbands * nchunks;
    const long long grid8 = (grid + 7) / 8 * 8;
    if (grid <= 0 || grid8 > 0x7fffffffLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((pool_frag_rows<K, RB, BF, IN_F32, V>), dim3((unsigned)grid8), dim3(256), 0, s, a, nbands,
                       nchunks, (int)grid);
    return hipGetLastError();
}

// Filter rows per thread: the planner's choice (PoolArgs::rows).
template <int K, bool BF, bool IN_F32, int V>
hipError_t go_rows(const PoolArgs &a, hipStream_t s)
{
    if (a.rows == 4) return go_rows_rb<K, 4, BF, IN_F32, V>(a, s);
    return go_rows_rb<K, 8, BF, IN_F32, V>(a, s);
}

template <bool BF, bool IN_F32, int V>
hipError_t go_k(const PoolArgs &a, int grid, hipStream_t s)
{
    if (a.ky == a.kx && a.sy == a.ky && a.sx == a.kx) {  // the paper's pools: stride = size
        if (a.ky == 2) return go_rows<2, BF, IN_F32, V>(a, s);
        if (a.ky == 3) return go_rows<3, BF, IN_F32, V>(a, s);
        if (a.ky == 4) return go_rows<4, BF, IN_F32, V>(a, s);
    }
    hipLaunchKernelGGL((pool_frag<BF, IN_F32, V>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}


}  // namespace

hipError_t launch_pool(const PoolArgs &a, int dtype, bool in_f32, int grid, hipStream_t s)
{
    if (dtype == DT_F32) return (a.C % 4 == 0) ? go_k<false, false, 4>(a, grid, s) : go_k<false, false, 1>(a, grid, s);
    if (in_f32) return go_k<true, true, 1>(a, grid, s);
    return (a.C % 8 == 0) ? go_k<true, false, 8>(a, grid, s) : go_k<true, false, 1>(a, grid, s);
}

std::string pool_kernel_name(int dtype, bool in_f32, int ky, int kx, int sy, int sx, int C, int rows)
{
    // the instance launch_pool picks, as the profiler names it
    const bool bf = dtype == DT_BF16, bin = bf && in_f32;
    const int v = !bf ? (C % 4 == 0 ? 4 : 1) : (in_f32 ? 1 : (C % 8 == 0 ? 8 : 1));
    const char *t = bf ? "true" : "false", *ti = bin ? "true" : "false";
    char buf[64];
    if (ky == kx && sy == ky && sx == kx && ky >= 2 && ky <= 4)
        snprintf(buf, sizeof buf, "pool_frag_rows<%d, %d, %s, %s, %d>", ky, rows == 4 ? 4 : 8, t, ti, v);
    else
        snprintf(buf, sizeof buf, "pool_frag<%s, %s, %d>", t, ti, v);
    return buf;
}

}  // namespace fs
