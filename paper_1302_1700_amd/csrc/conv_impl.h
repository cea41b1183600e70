// Fragment-batched convolution on the CDNA4 matrix cores (implicit GEMM).
// Included by conv_f32.hip and conv_bf16.hip, which instantiate it.
//
// Section 2.2.1: a convolutional layer keeps the fragment count and convolves
// each fragment's extended maps exactly as a patch is convolved; the sizes
// shrink by k - 1 per axis (Eqs. 3-4).  Fully connected layers run through the
// same kernel as convolutions whose kernel covers the patch-level map.
//
// As a matrix product, per layer: M = output pixels of all fragments (the
// fragments are the batch), N = c_out, K = c_in * k * k, with
//   out[q, y, x, co] = act(bias[co] + sum_{dy, dx, ci} W[co, ci, dy, dx] * in[q, y+dy, x+dx, ci]).
//
// Work split
//   - A fragment's output columns are cut into bands of `band_w` columns; the
//     pixels of a band are numbered row-major and cut into tiles of `mt`
//     pixels.  Tiles follow the fragment's true size, with waste only at the
//     end of a band.
//   - The workgroup (4 waves) stages the input window its tile needs (the
//     rows its pixels touch plus k - 1, band + k - 1 columns, all c_in
//     channels) in LDS once, zero-filled outside the fragment's true size.
//   - The 4 waves form a WM x WN grid: wave (wm, wn) computes MB blocks of 16
//     pixels (m-blocks wm*MB ..) times NB blocks of 16 output channels
//     (n-blocks wn*NB ..), so waves in a row share pixels and waves in a
//     column share weights.  Products use v_mfma_f32_16x16x4_f32 (float32) or
//     v_mfma_f32_16x16x32_bf16 (bfloat16 operands, float32 accumulate), with
//     the weights as the row operand and the pixels as the column operand, so
//     the 16 x 16 result of a (channel block, pixel block) pair leaves row
//     4g + e (a channel) of column lm (a pixel) in lane lm + 16g, element e.
//   - A lane (lm = lane % 16, g = lane / 16) feeds pixel lm of each m-block and
//     16 bytes of consecutive K values starting at g * (KSTEP / 4); float32
//     uses element e of that vector in the e-th of 4 products, so each product
//     sums over K indices {4g + e}.  The weights are pre-arranged on the host
//     so that each (K step, channel block) is one contiguous 1 KB run, read by
//     a wave in one coalesced load; the next step's weights and pixels are
//     loaded while the current step's products run.  Which channel a block
//     row computes is fixed by the host's packing (api.hip: chan_of).
//   - Vector path (c_in a multiple of KSTEP): K is walked tap by tap, KSTEP
//     channels at a time, and a lane's A operand is one 16-byte LDS read.
//     Gather path (small c_in, e.g. the first layer): K = (tap, channel)
//     flattened and padded to KSTEP, gathered through an LDS offset table.
//   - Epilogue: bias and tanh in float32, then each lane stores its four
//     (bf16 with paired channel blocks: eight) consecutive channels of a
//     pixel straight from its registers (bf16: round to nearest even), only
//     inside the fragment's true size.
#pragma once

#include "fs_internal.h"

#include <algorithm>
#include <atomic>
#include <type_traits>

namespace fs {
namespace conv {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

typedef float f2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf2v __attribute__((ext_vector_type(2)));

// Two bfloat16 values -> two int16 keys with the same order (negative values
// get their 15 magnitude bits flipped), so a packed integer max picks the
// larger value of each half; the map is its own inverse.
typedef short s2v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16x2_key(uint32_t x)
{
    // per half: all ones for a negative value (arithmetic shift by 15), whose
    // 15 magnitude bits are then flipped
    const uint32_t neg = __builtin_bit_cast(uint32_t, __builtin_bit_cast(s2v, x) >> (short)15);
    return x ^ (neg & 0x7fff7fffu);
}
__device__ __forceinline__ uint32_t max_i16x2(uint32_t a, uint32_t b)
{
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(s2v, a), __builtin_bit_cast(s2v, b)));
}

// float -> bfloat16, round to nearest even (one v_cvt_pk_bf16_f32 per pair)
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2v{lo, hi}, bf2v));
}

// Quotient and remainder of the small non-negative integers of the tile
// index arithmetic (n < 2^20, 1 <= d < 2^16; the planner keeps tiles within
// that) by a divisor fixed for the tile: one multiply by a float reciprocal,
// truncated, then one correction either way (the product's error is below
// 1/4 for such n).  The general 32-bit division the compiler emits costs
// ~25 instructions; this ~7, which matters in the per-element loops.
struct Div {
    int d;
    float r;
    __device__ explicit Div(int d_) : d(d_), r(__builtin_amdgcn_rcpf((float)d_)) {}
    __device__ int quo(int n) const
    {
        int q = (int)((float)n * r);
        const int t = n - __mul24(q, d);
        return q + (t >= d) - (t < 0);
    }
    // n = q * d + m, 0 <= m < d
    __device__ void qr(int n, int &q, int &m) const
    {
        q = quo(n);
        m = n - __mul24(q, d);
    }
};

// tanh(x) = 1 - 2 / (exp(2x) + 1), with the hardware exp2 and reciprocal:
// absolute error a few 1e-7, saturates cleanly to +-1 for large |x|.
__device__ __forceinline__ float tanh_fast(float x)
{
    const float t = __builtin_amdgcn_exp2f(x * 2.8853900817779268f);  // exp(2x)
    return 1.0f - 2.0f * __builtin_amdgcn_rcpf(t + 1.0f);
}

template <bool BF>
struct Elem;
template <>
struct Elem<false> {
    using T = float;
    static constexpr int KSTEP = 16;
};
template <>
struct Elem<true> {
    using T = uint16_t;
    static constexpr int KSTEP = 32;
};

// Fused last layer.  The tile's activations act(acc + bias) never leave the
// registers: every lane multiplies its values (rows 4g .. 4g + 3 of each
// channel block, for pixel lm of each m-block) by the last layer's weights
// (stored over the same (block, row) order), the four lanes of a pixel add up
// with xor shuffles (fused_head_partials; bf16 tiles with paired blocks use a
// matrix-core product per block pair instead); the waves that split the channels
// add up through LDS and one thread per pixel applies the last activation
// (softmax: exp(z - max z) / sum) and writes the pixel's classes to the dense
// map at the window corner the pixel stands for: final fragment (fy, fx)
// position (y, x) holds window (base[fy] + S*y, base[fx] + S*x)
// (fused_head_finish).  A workgroup barrier separates the two.
// Whether the fused head keeps only z1 - z0 (two classes and softmax, per-lane
// products): fused_head_partials and fused_head_finish agree on it.
template <bool BF, int NB>
__device__ __forceinline__ bool head_two_class(const ConvArgs &a)
{
    return !(BF && NB % 2 == 0) && a.head_ncls == 2 && a.head_act == ACT_SOFTMAX;
}

template <int MB, int NB, int WN, bool BF>
__device__ __forceinline__ void fused_head_partials(const ConvArgs &a, const f4 (&acc)[MB][NB], int nb0, int wm,
                                                    int wn, int lm, int g, float *red)
{
    constexpr int NC = kMaxFusedClasses;
    float part[MB][NC];
    if constexpr (BF && NB % 2 == 0) {
        // bf16 with paired blocks: the activations, rounded to bf16 as the
        // layer would store them, are the column operand of one 16x16x32
        // product per block pair against the class weights (rows = classes):
        // lane (lm, g) supplies pixel lm's channels 8g .. 8g + 7 of the pair
        // and ends with classes 4g .. 4g + 3 of pixel lm.
        const u4 *hw = reinterpret_cast<const u4 *>(a.head_wbf) + (size_t)(nb0 / 2) * 64 + g * 16 + lm;
        f4 hacc[MB];
#pragma unroll
        for (int i = 0; i < MB; ++i) hacc[i] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int p = 0; p < NB / 2; ++p) {
            const u4 wv = hw[p * 64];
#pragma unroll
            for (int i = 0; i < MB; ++i) {
                float h[8];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    h[e] = acc[i][2 * p][e];
                    h[4 + e] = acc[i][2 * p + 1][e];
                }
                if (a.act == ACT_TANH) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) h[e] = tanh_fast(h[e]);
                }
                u4 pk;
#pragma unroll
                for (int e = 0; e < 4; ++e) pk[e] = pack_bf16(h[2 * e], h[2 * e + 1]);
                hacc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, wv), __builtin_bit_cast(bf8, pk),
                                                                  hacc[i], 0, 0, 0);
            }
        }
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
            for (int c = 0; c < NC; ++c) part[i][c] = hacc[i][c];
    } else if (head_two_class<BF, NB>(a)) {
        // two classes with softmax: only z1 - z0 is needed, one product per
        // value with the weight differences
        const int ldw = a.nbt * 16;
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
            for (int c = 0; c < NC; ++c) part[i][c] = 0.f;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int r0 = (nb0 + j) * 16 + 4 * g;
            const f4 w0 = *reinterpret_cast<const f4 *>(a.head_w + r0);
            const f4 w1 = *reinterpret_cast<const f4 *>(a.head_w + (size_t)ldw + r0);
#pragma unroll
            for (int i = 0; i < MB; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float v = acc[i][j][e];
                    if (a.act == ACT_TANH) v = tanh_fast(v);
                    part[i][0] = fmaf(w1[e] - w0[e], v, part[i][0]);
                }
        }
#pragma unroll
        for (int i = 0; i < MB; ++i) {
            float t = part[i][0];
            t += __shfl_xor(t, 16);
            t += __shfl_xor(t, 32);
            part[i][0] = t;
        }
    } else {
        const int ldw = a.nbt * 16;
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
            for (int c = 0; c < NC; ++c) part[i][c] = 0.f;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int r0 = (nb0 + j) * 16 + 4 * g;  // (block, row) index of element 0
            // (rows past head_ncls are zero on the device: unconditional loads)
            f4 w2[NC];
#pragma unroll
            for (int c = 0; c < NC; ++c) w2[c] = *reinterpret_cast<const f4 *>(a.head_w + (size_t)c * ldw + r0);
#pragma unroll
            for (int i = 0; i < MB; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float v = acc[i][j][e];
                    if (a.act == ACT_TANH) v = tanh_fast(v);
#pragma unroll
                    for (int c = 0; c < NC; ++c) part[i][c] = fmaf(w2[c][e], v, part[i][c]);
                }
        }
        // the four lanes of a pixel hold disjoint channels: add them up
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                float t = part[i][c];
                t += __shfl_xor(t, 16);
                t += __shfl_xor(t, 32);
                part[i][c] = t;
            }
    }
    if (g == 0) {
#pragma unroll
        for (int i = 0; i < MB; ++i) {
            const int m = (wm * MB + i) * 16 + lm;
#pragma unroll
            for (int c = 0; c < NC; ++c) red[((size_t)wn * a.mt + m) * NC + c] = part[i][c];
        }
    }
}

// Bounds check of a fused-head write: output (y, x) of final fragment
// (fy, fx) of image b lies inside the fragment's true size and its window
// (Y, X) inside the map.
__device__ __forceinline__ bool head_ok(const ConvArgs &a, int b, int fy, int fx, int y, int x, int Y, int X)
{
    return FS_DBG_OK(a.dbg,
                     b < a.nfrag / a.F && y < a.ext.y[fy] - a.ky + 1 - a.dbg_shrink &&
                         x < a.ext.x[fx] - a.kx + 1 - a.dbg_shrink && Y < a.ny && X < a.nx,
                     DBG_FUSED_HEAD);
}

// locate(m, fy, fx, y, x): fragment (fy, fx) of image b and output (y, x)
// in it of the tile's pixel m < npix.
template <int WN, class Locate>
__device__ __forceinline__ void fused_head_finish(const ConvArgs &a, int b, int npix, Locate locate,
                                                  const float *red, bool two_class)
{
    constexpr int NC = kMaxFusedClasses;
    const int ncls = a.head_ncls;
    const int mt = a.mt;
    for (int m = threadIdx.x; m < npix; m += blockDim.x) {
        float z[NC];
        if (two_class) {
            // softmax of two: p1 = 1 / (1 + exp(z0 - z1)), p0 = 1 / (1 + exp(z1 - z0))
            float d = a.head_b[1] - a.head_b[0];
#pragma unroll
            for (int w = 0; w < WN; ++w) d += red[((size_t)w * mt + m) * NC];
            z[0] = 1.0f / (1.0f + expf(d));
            z[1] = 1.0f / (1.0f + expf(-d));
            int fy, fx, y, x;
            locate(m, fy, fx, y, x);
            const int Y = a.base_y[fy] + a.Sy * y, X = a.base_x[fx] + a.Sx * x;
            if (!head_ok(a, b, fy, fx, y, x, Y, X)) continue;
            float *dst = a.head_out + (((size_t)b * a.ny + Y) * a.nx + X) * 2;
            *reinterpret_cast<float2 *>(dst) = float2{z[0], z[1]};
            continue;
        }
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            float t = c < ncls ? a.head_b[c] : 0.f;
#pragma unroll
            for (int w = 0; w < WN; ++w) t += red[((size_t)w * mt + m) * NC + c];
            z[c] = t;
        }
        if (a.head_act == ACT_SOFTMAX) {
            float mx = z[0];
#pragma unroll
            for (int c = 1; c < NC; ++c)
                if (c < ncls) mx = fmaxf(mx, z[c]);
            float sum = 0.f;
#pragma unroll
            for (int c = 0; c < NC; ++c)
                if (c < ncls) {
                    z[c] = expf(z[c] - mx);
                    sum += z[c];
                }
            const float inv = 1.0f / sum;
#pragma unroll
            for (int c = 0; c < NC; ++c) z[c] *= inv;
        } else if (a.head_act == ACT_TANH) {
#pragma unroll
            for (int c = 0; c < NC; ++c) z[c] = tanhf(z[c]);
        }
        int fy, fx, y, x;
        locate(m, fy, fx, y, x);
        const int Y = a.base_y[fy] + a.Sy * y, X = a.base_x[fx] + a.Sx * x;
        if (!head_ok(a, b, fy, fx, y, x, Y, X)) continue;
        float *dst = a.head_out + (((size_t)b * a.ny + Y) * a.nx + X) * ncls;
#pragma unroll
        for (int c = 0; c < NC; ++c)
            if (c < ncls) dst[c] = z[c];
    }
}

// RUN: run tiles (ConvArgs::run = 1, no fused pool); the other instances
// take one band of one fragment per tile sequence.  Float32 tiles of one
// channel block and up to four pixel blocks (16-channel layers, whose
// launches wait on memory) are compiled for six workgroups per CU (at most
// 80 registers: six waves per SIMD instead of five; 4-5% faster on the
// 2x2 16 -> 16 + pool layers; larger tiles would spill).
template <int MB, int NB, int WN, int WK, bool BF, bool IN_F32, bool VEC, bool RUN>
__global__ __launch_bounds__(256, (!BF && NB == 1 && MB <= 4) ? 6 : 1) void conv_frag_mfma(ConvArgs a)
{
    using TC = typename Elem<BF>::T;                                // LDS / operand element
    using TI = typename std::conditional<IN_F32, float, TC>::type;  // global input element
    constexpr int KSTEP = Elem<BF>::KSTEP;
    constexpr int LPE = KSTEP / 4;  // elements per lane per K step (16 bytes)

    extern __shared__ __align__(16) unsigned char smem[];

    // Workgroups are dealt to the 8 XCDs round-robin; renumber them so each
    // XCD gets a contiguous run of tiles, whose shared window rows and
    // columns then meet in that XCD's L2 (the grid is padded to a multiple of
    // 8; the padding tiles exit).
    const int per_xcd = gridDim.x / 8;
    int bid = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    const int nunit = RUN ? a.nfrag / a.F : a.nfrag;  // images (run tiles) or fragments
    if (bid >= nunit * a.nbands * a.tiles_per_band) return;
    // the tile's channel blocks (weights, bias, last-layer weights) lie in the layer's packing
    if (!FS_DBG_OK(a.dbg, (int)(blockIdx.y + 1) * (WN * NB) <= a.nbt, DBG_CONV_WEIGHT)) return;
    int sib = 0;  // xsib: the fragment's column index
    if (!RUN && a.xsib) {
        sib = bid % a.Qx;
        bid /= a.Qx;
    }
    const int t = bid % a.tiles_per_band;
    bid /= a.tiles_per_band;
    const int band = bid % a.nbands;

    // The tile's convolution outputs: segment 0 numbers them l in [l0, lend),
    // pixel l at row l / twb, column c0 + l % twb of fragment q's output; a
    // run tile that reaches the end of its fragment continues with the first
    // n1 pixels of the next fragment q1 (segment 1, width twb1).
    int q, fy, fx, l0, lend, twb;
    int q1 = 0, fy1 = 0, fx1 = 0, n1 = 0, twb1 = 1;
    int c0 = 0;
    int y0 = 0, rtM = 0, twM = 0;  // fused pool: max-filter rows [y0, y0 + rtM), columns [c0, c0 + twM)
    int hin, win;
    if constexpr (RUN) {
        const int b = bid / a.nbands;
        const int p0 = t * a.mt;
        if (p0 >= a.run_pix) return;
        const int np = min(a.mt, a.run_pix - p0);
        // row of fragments: the last fy with ypre[fy] * wsum <= p0
        const int v = p0 / a.run_wsum;
        int lo = 0, hi = a.Qy - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if ((int)a.run_ypre[mid] <= v) lo = mid; else hi = mid - 1;
        }
        fy = lo;
        const int ho = a.run_ypre[fy + 1] - a.run_ypre[fy];
        const int r0 = p0 - (int)a.run_ypre[fy] * a.run_wsum;
        const int u = r0 / ho;
        lo = 0;
        hi = a.Qx - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if ((int)a.run_xpre[mid] <= u) lo = mid; else hi = mid - 1;
        }
        fx = lo;
        twb = a.run_xpre[fx + 1] - a.run_xpre[fx];
        l0 = r0 - ho * (int)a.run_xpre[fx];
        lend = min(ho * twb, l0 + np);
        n1 = np - (lend - l0);
        q = b * a.F + fy * a.Qx + fx;
        if (n1 > 0) {  // every fragment holds at least mt pixels: one more segment at most
            fy1 = fy;
            fx1 = fx + 1;
            if (fx1 == a.Qx) {
                fx1 = 0;
                ++fy1;
            }
            q1 = b * a.F + fy1 * a.Qx + fx1;
            twb1 = a.run_xpre[fx1 + 1] - a.run_xpre[fx1];
        }
        hin = a.ext.y[fy];
        win = a.ext.x[fx];
    } else {
        if (a.xsib) {
            const int row = bid / a.nbands;  // b * Qy + fy
            fy = row % a.Qy;
            fx = sib;
            q = (row / a.Qy) * a.F + fy * a.Qx + fx;
        } else {
            q = bid / a.nbands;
            const int rem = q % a.F;
            fy = rem / a.Qx;
            fx = rem - (rem / a.Qx) * a.Qx;
        }
        hin = a.ext.y[fy];
        win = a.ext.x[fx];
        const int hout = hin - a.ky + 1, wout = win - a.kx + 1;
        if (hout <= 0 || wout <= 0) return;
        c0 = band * a.band_w;
        if (a.pool_ky) {
            // Section 2.2.2: child (o_x, o_y) of a k x k pool holds the stride-1
            // k x k max filter M of its parent at (o_y + k*ybar, o_x + k*xbar),
            // so every filter position y < hout - k + 1 (and likewise x) feeds
            // exactly one child.  The tile computes the convolution outputs its
            // filter positions need: k - 1 more rows and columns (per axis,
            // for a k_y x k_x pool).
            const int hM = hout - a.pool_ky + 1, wM = wout - a.pool_kx + 1;
            if (hM <= 0 || wM <= 0) return;
            twM = min(a.band_w, wM - c0);
            if (twM <= 0) return;
            y0 = t * a.pool_rt;
            if (y0 >= hM) return;
            rtM = min(a.pool_rt, hM - y0);
            twb = twM + a.pool_kx - 1;
            l0 = y0 * twb;
            lend = l0 + (rtM + a.pool_ky - 1) * twb;
        } else {
            twb = min(a.band_w, wout - c0);
            if (twb <= 0) return;
            const int npix = hout * twb;
            const int tpx = a.tile_rows ? a.tile_rows * twb : a.mt;  // pixels per tile
            l0 = t * tpx;
            if (l0 >= npix) return;
            lend = min(l0 + tpx, npix);
        }
    }
    const int n0 = lend - l0;
    const int yfirst = l0 / twb;
    const int ylast = (lend - 1) / twb;
    const int R = ylast - yfirst + a.ky;                     // window rows of segment 0
    const int R1 = n1 > 0 ? (n1 - 1) / twb1 + a.ky : 0;      // then those of segment 1
    const int Cc = max(twb, n1 > 0 ? twb1 : 0) + a.kx - 1;   // window columns
    const int hin1 = n1 > 0 ? a.ext.y[fy1] : 0, win1 = n1 > 0 ? a.ext.x[fx1] : 0;
    const int CS = a.lds_cs;
    const int kk_total = a.ksteps * KSTEP;

    int *offtab = reinterpret_cast<int *>(smem);
    TC *win_lds = reinterpret_cast<TC *>(smem + (VEC ? 0 : ((kk_total * 4 + 15) & ~15)));

    // ---- stage the input window ----------------------------------------------
    // window rows [0, R) come from fragment q (rows yfirst ..), rows
    // [R, R + R1) from fragment q1 (rows 0 ..); columns c0 .. of both
    const size_t fsz = (size_t)a.in_h * a.in_w * a.in_c;
    const TI *inp = reinterpret_cast<const TI *>(a.in) + (size_t)q * fsz;
    const TI *inp1 = reinterpret_cast<const TI *>(a.in) + (size_t)q1 * fsz;
    // nrows window rows from row row0 on: rows gy0 .. of fragment src (batch
    // index fq), whose true size is hh x ww (outside it, zeros)
    auto stage = [&](const TI *src, int fq, int gy0, int hh, int ww, int row0, int nrows) {
        const int rowp = a.in_w * a.in_c;  // elements per input row (fragments stay below 2^31)
        const int npx = nrows * Cc;        // window pixels to stage
        auto read_ok = [&](int gy, int gx) {
            return FS_DBG_OK(a.dbg, fq < a.nfrag && gy < hh - a.dbg_shrink && gx < ww - a.dbg_shrink && gy < a.in_h &&
                                        gx < a.in_w, DBG_CONV_READ);
        };
        // Fast form (up to 64 loads per pixel): a thread owns load v of
        // window pixels p, p + P, p + 2P, ... (P = 256 / loads per pixel);
        // the pixel's (row, column) and both addresses advance by constants,
        // with at most one carry into the next row per step.  UN loads are
        // in flight per thread before their LDS stores.
        auto walk = [&](int nvec, int width, auto load) {
            // Loads in flight per thread before their LDS stores: two for the
            // float32 tiles of three or more channel blocks whose waves split
            // the channels or the K steps in two (FC1's 7 x 2 and the split-K
            // 4 x 3 of 48 -> 48 layers), whose window staging runs beside
            // the K walk of another resident workgroup and delays its weight
            // loads less that way (N4 on 8 x 1024^2: FC1 + head 1.4% and the
            // 48 -> 48 layers up to 0.9% faster than with eight); eight for
            // the rest, where two measured 3-4% slower.
            constexpr int UN = (!BF && VEC && NB >= 3 && (WN == 2 || WK == 2)) ? 2 : 8;
            const int P = 256 / nvec;
            int p, v;
            Div(nvec).qr(threadIdx.x, p, v);
            if (p >= P) return;  // threads past P * nvec idle
            int r, c;
            Div(Cc).qr(p, r, c);
            const int dr = P / Cc, dc = P - dr * Cc;
            int soff = (gy0 + r) * rowp + __mul24(c0 + c, a.in_c) + v * width;
            const int sstep = dr * rowp + dc * a.in_c, swrap = rowp - Cc * a.in_c;
            int doff = __mul24(__mul24(row0, Cc) + p, CS) + v * width;
            const int dstep = P * CS;
            while (p < npx) {
                decltype(load(0)) val[UN];
                int dsto[UN];
#pragma unroll
                for (int u = 0; u < UN; ++u) {
                    const bool in = p < npx;
                    // A tile of one fragment never reaches past its true
                    // size: its last window row is at most hout - 1 + k_y - 1
                    // = hh - 1, its last column c0 + twb - 1 + k_x - 1 <= ww - 1
                    // (also for the fused pool's filter tiles).  Run tiles
                    // stage two fragments with the wider one's columns.
                    if constexpr (RUN) {
                        val[u] = {};
                        if (in && gy0 + r < hh && c0 + c < ww && read_ok(gy0 + r, c0 + c)) val[u] = load(soff);
                    } else {
                        if (in && read_ok(gy0 + r, c0 + c)) val[u] = load(soff);
                    }
                    dsto[u] = in ? doff : -1;
                    p += P;
                    doff += dstep;
                    soff += sstep;
                    r += dr;
                    c += dc;
                    if (c >= Cc) {
                        c -= Cc;
                        ++r;
                        soff += swrap;
                    }
                }
#pragma unroll
                for (int u = 0; u < UN; ++u)
                    if (dsto[u] >= 0) *reinterpret_cast<decltype(load(0)) *>(win_lds + dsto[u]) = val[u];
            }
        };
        if constexpr (VEC && !IN_F32) {
            const int nvec = a.cin / LPE;
            if (nvec <= 64) {
                walk(nvec, LPE, [&](int off) { return *reinterpret_cast<const u4 *>(src + off); });
                return;
            }
            // batches of 8 loads in flight per thread before their LDS stores
            const int total = npx * nvec;
            const Div dnv(nvec), dcc(Cc);
            constexpr int UN = 8;
            for (int base = threadIdx.x; base < total; base += 256 * UN) {
                u4 val[UN];
                int dsto[UN];
#pragma unroll
                for (int u = 0; u < UN; ++u) {
                    const int idx = base + u * 256;
                    int p, v, r, c;
                    dnv.qr(idx, p, v);
                    dcc.qr(p, r, c);
                    const int gy = gy0 + r, gx = c0 + c;
                    val[u] = u4{0u, 0u, 0u, 0u};
                    if (idx < total && gy < hh && gx < ww && read_ok(gy, gx))
                        val[u] = *reinterpret_cast<const u4 *>(src + (gy * rowp + __mul24(gx, a.in_c) + v * LPE));
                    dsto[u] = idx < total ? __mul24(__mul24(row0 + r, Cc) + c, CS) + v * LPE : -1;
                }
#pragma unroll
                for (int u = 0; u < UN; ++u)
                    if (dsto[u] >= 0) *reinterpret_cast<u4 *>(win_lds + dsto[u]) = val[u];
            }
        } else {
            if (a.cin <= 64) {
                walk(a.cin, 1, [&](int off) -> TC {
                    if constexpr (BF && IN_F32)
                        return f2bf(src[off]);
                    else
                        return src[off];
                });
                return;
            }
            const int total = npx * a.cin;
            const Div dci(a.cin), dcc(Cc);
            for (int idx = threadIdx.x; idx < total; idx += 256) {
                int p, ci, r, c;
                dci.qr(idx, p, ci);
                dcc.qr(p, r, c);
                const int gy = gy0 + r, gx = c0 + c;
                TC val = 0;
                if (gy < hh && gx < ww && read_ok(gy, gx)) {
                    TI x = src[gy * rowp + __mul24(gx, a.in_c) + ci];
                    if constexpr (BF && IN_F32)
                        val = f2bf(x);
                    else
                        val = x;
                }
                win_lds[__mul24(__mul24(row0 + r, Cc) + c, CS) + ci] = val;
            }
        }
    };
    stage(inp, q, yfirst, hin, win, 0, R);
    if constexpr (RUN)
        if (R1 > 0) stage(inp1, q1, 0, hin1, win1, R, R1);
    if constexpr (!VEC) {
        const Div dci(a.cin), dk(a.kx);
        for (int kk = threadIdx.x; kk < kk_total; kk += 256) {
            int tap, ci;
            dci.qr(kk, tap, ci);
            int off = -1;
            if (tap < a.ky * a.kx) {
                int dy, dx;
                dk.qr(tap, dy, dx);
                off = (dy * Cc + dx) * CS + ci;
            }
            offtab[kk] = off;
        }
    }
    __syncthreads();

    // ---- matrix-core main loop ----------------------------------------------
    // wave (wm, wn, wk): pixel blocks wm*MB.., channel blocks wn*NB.., and the
    // wk-th of WK equal parts of the K steps (their partial sums are added up
    // through LDS after the loop)
    constexpr int WMN = 4 / WK;
    // the wave index is the same in every lane of a wave; read it from the
    // first lane so that everything derived from it (the wave's K range,
    // the step counters and LDS offsets of the K walk, its weight and bias
    // addresses) is computed once per wave in scalar registers
    const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wk = wv / WMN, wmn = wv - (wv / WMN) * WMN;
    const int wm = wmn / WN, wn_raw = wmn - (wmn / WN) * WN;
    // Float32 layers whose two wave columns own unequal work -- the second
    // half ends in a padding block, whose products it skips (FC1 with the
    // fused head: 200 outputs in 14 blocks) -- swap the halves between the
    // columns in every other workgroup of an XCD's run (ConvArgs::swapn), so
    // the two workgroups sharing a CU tend to load each SIMD with one heavy
    // and one light wave (N4's FC1 on 8x1024^2 4% faster).  The channel sums
    // and their order are those of the unswapped tile.
    const bool swap = !BF && WN == 2 && WK == 1 && a.swapn && ((blockIdx.x / 8) & 1);
    const int wn = swap ? 1 - wn_raw : wn_raw;
    const int lm = lane & 15, g = lane >> 4;
    const int nb0 = blockIdx.y * (WN * NB) + wn * NB;

    // tile pixel m < npix: segment seg, output row y and column c0 + x of
    // fragment q (seg 0) or q1 (seg 1; c0 = 0 there)
    const int npix = n0 + n1;
    const Div dtw(twb), dtw1(twb1);
    auto locate = [&](int m, int &seg, int &y, int &x) {
        seg = RUN && m >= n0;
        if (seg)
            dtw1.qr(m - n0, y, x);
        else
            dtw.qr(l0 + m, y, x);
    };
    // output (y, x) of segment seg's fragment: inside its true size (Eqs. 3-4)
    auto write_ok = [&](int seg, int y, int x) {
        [[maybe_unused]] const int hh = (seg ? hin1 : hin) - a.ky + 1 - a.dbg_shrink,
                                   ww = (seg ? win1 : win) - a.kx + 1 - a.dbg_shrink;
        return FS_DBG_OK(a.dbg, (seg ? q1 : q) < a.nfrag && y < hh && x < ww && y < a.out_h && x < a.out_w,
                         DBG_CONV_WRITE);
    };
    int abase[MB];
#pragma unroll
    for (int i = 0; i < MB; ++i) {
        const int m = (wm * MB + i) * 16 + lm;
        if (m < n0) {
            int y, x;
            dtw.qr(l0 + m, y, x);
            abase[i] = ((y - yfirst) * Cc + x) * CS + g * LPE;
        } else {
            abase[i] = g * LPE;  // any in-window address; the result is not stored
        }
    }
    if (RUN && n1 > 0) {
#pragma unroll
        for (int i = 0; i < MB; ++i) {
            const int m = (wm * MB + i) * 16 + lm;
            if (m >= n0 && m < npix) {
                int y, x;
                dtw1.qr(m - n0, y, x);
                abase[i] = ((y + R) * Cc + x) * CS + g * LPE;
            }
        }
    }

    // The accumulators start from the bias (rows 4g .. 4g + 3 of each block;
    // the waves with wk > 0 from zero, their sums are added to wk == 0's), so
    // the epilogue has no bias to add.
    f4 acc[MB][NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        f4 b0 = f4{0.f, 0.f, 0.f, 0.f};
        if (wk == 0) b0 = *reinterpret_cast<const f4 *>(a.bias + (nb0 + j) * 16 + 4 * g);
#pragma unroll
        for (int i = 0; i < MB; ++i) acc[i][j] = b0;
    }

    const u4 *wp = reinterpret_cast<const u4 *>(a.w) + (size_t)nb0 * 64 + lane;
    const size_t wstep = (size_t)a.nbt * 64;  // u4 per K step

    // nbac: the blocks whose products are taken (the rest are padding)
    auto mma = [&](const u4(&av)[MB], const u4(&bv)[NB], auto nbac) {
        constexpr int NBA = decltype(nbac)::value;
        if constexpr (BF) {
#pragma unroll
            for (int i = 0; i < MB; ++i)
#pragma unroll
                for (int j = 0; j < NBA; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf8, bv[j]), __builtin_bit_cast(bf8, av[i]), acc[i][j], 0, 0, 0);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int i = 0; i < MB; ++i)
#pragma unroll
                    for (int j = 0; j < NBA; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                            __uint_as_float(bv[j][e]), __uint_as_float(av[i][e]), acc[i][j], 0, 0, 0);
        }
    };

    if constexpr (VEC) {
        auto kwalk = [&](auto nbac) {
            // K step s covers tap (dy, dx) and channels cc*KSTEP ..; the three
            // indices advance incrementally.  Weights are loaded PD steps ahead
            // (a ring of PD register buffers, the loop unrolled by PD) and pixels
            // one step ahead, so the products of a step never wait on the loads
            // it needs.
            // (four-deep rings measured slower for bf16: the extra registers
            // cost a wave per SIMD)
            constexpr int PD = 2;
            static_assert(PD % 2 == 0, "the pixel double buffer needs an even unroll");
            const int ncc = a.cin / KSTEP;
            const int s_begin = (a.ksteps * wk) / WK, s_end = (a.ksteps * (wk + 1)) / WK;
            const int nsteps = s_end - s_begin;
            // (branch-free: a straight-line loop body lets the compiler wait only
            // for the operands each product needs)
            int cc = s_begin % ncc, dx = (s_begin / ncc) % a.kx, dy = (s_begin / ncc) / a.kx;
            auto advance = [&](int) {
                ++cc;
                const int w1 = cc == ncc;
                cc = w1 ? 0 : cc;
                dx += w1;
                const int w2 = dx == a.kx;
                dx = w2 ? 0 : dx;
                dy += w2;
                return (dy * Cc + dx) * CS + cc * KSTEP;
            };
            u4 b[PD][NB], av[2][MB];
            const u4 *wpk = wp + (size_t)s_begin * wstep;
            const int off0 = (dy * Cc + dx) * CS + cc * KSTEP;
            const int last = nsteps - 1;
            // unconditional (clamped) so every path reaches the loop with the same
            // loads in flight
#pragma unroll
            for (int t = 0; t < PD; ++t)
#pragma unroll
                for (int j = 0; j < NB; ++j) b[t][j] = wpk[(size_t)min(t, last) * wstep + j * 64];
#pragma unroll
            for (int i = 0; i < MB; ++i) av[0][i] = *reinterpret_cast<const u4 *>(win_lds + abase[i] + off0);
            // The prefetches are issued on every step (past the end they re-read
            // the last step's weights and the window's first pixel), so every
            // path through the loop has the same loads in flight and the waits
            // before the products only cover the operands they use.
            int off = off0;
            int s = 0;
            // Interleaved form (all tiles but the float32 one-block ones): the
            // step's bookkeeping for later steps -- the tap and channel counters
            // of step s + t + 2 and the weight pointer of step s + t + PD + 1 --
            // runs between its products (two scalar instructions after each),
            // where a lone wave per SIMD would otherwise leave the matrix core
            // idle; only the loads stay between steps (N4's 48 -> 48 layers and
            // FC1 2-5% faster, workload 5 2%; the float32 one-block tiles, held to
            // 80 registers, would spill).
            constexpr bool IL = BF || NB > 1;
            int offn = IL ? advance(off) : 0;                       // step 1's offset
            const u4 *wnx = wpk + (size_t)min(PD, last) * wstep;    // step PD's weights
            int kw = min(PD, last);                                 // ... their step (clamped)
            for (; s + PD <= nsteps; s += PD) {
#pragma unroll
                for (int t = 0; t < PD; ++t) {
                    // scheduling barriers keep each prefetch ahead of the products
                    // that do not need it (left alone, the compiler sinks the
                    // loads below them to share registers, exposing their latency)
                    if constexpr (IL) {
                        const int offa = s + t + 1 < nsteps ? offn : off0;
#pragma unroll
                        for (int i = 0; i < MB; ++i)
                            av[(t + 1) & 1][i] = *reinterpret_cast<const u4 *>(win_lds + abase[i] + offa);
                        __builtin_amdgcn_sched_barrier(0);
                        const u4 *wcur = wnx;  // step s + t + PD (clamped to the last)
                        offn = advance(offn);
                        const bool more = kw < last;
                        wnx += more ? wstep : 0;
                        kw += more;
                        mma(av[t & 1], b[t], nbac);
#pragma unroll
                        for (int k = 0; k < 16; ++k) {
                            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one product
                            __builtin_amdgcn_sched_group_barrier(0x004, 2, 0);  // two scalar instructions
                        }
                        __builtin_amdgcn_sched_group_barrier(0x008, MB * NB * (BF ? 1 : 4), 0);
                        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                        for (int j = 0; j < NB; ++j) b[t][j] = wcur[j * 64];
                    } else {
                        off = advance(off);  // step s + t + 1
                        const int offa = s + t + 1 < nsteps ? off : off0;
#pragma unroll
                        for (int i = 0; i < MB; ++i)
                            av[(t + 1) & 1][i] = *reinterpret_cast<const u4 *>(win_lds + abase[i] + offa);
                        __builtin_amdgcn_sched_barrier(0);
                        mma(av[t & 1], b[t], nbac);
                        __builtin_amdgcn_sched_barrier(0);
                        const size_t wn2 = (size_t)min(s + t + PD, last) * wstep;
#pragma unroll
                        for (int j = 0; j < NB; ++j) b[t][j] = wpk[wn2 + j * 64];
                    }
                }
            }
            if constexpr (IL) off = offn;  // the tail advances from the next step's offset
            // the last nsteps % PD steps (their weights are already loaded)
#pragma unroll
            for (int t = 0; t + 1 < PD; ++t) {
                if (s + t < nsteps) {
                    int offa;
                    if constexpr (IL) {
                        offa = s + t + 1 < nsteps ? off : off0;
                        off = advance(off);
                    } else {
                        off = advance(off);
                        offa = s + t + 1 < nsteps ? off : off0;
                    }
#pragma unroll
                    for (int i = 0; i < MB; ++i)
                        av[(t + 1) & 1][i] = *reinterpret_cast<const u4 *>(win_lds + abase[i] + offa);
                    mma(av[t & 1], b[t], nbac);
                }
            }
        };
        // a wave whose last block is padding (ConvArgs::nbu) skips its products
        if constexpr (!BF && WN == 2 && WK == 1 && NB >= 2) {
            if (nb0 + NB - 1 >= a.nbu)
                kwalk(std::integral_constant<int, NB - 1>());
            else
                kwalk(std::integral_constant<int, NB>());
        } else {
            kwalk(std::integral_constant<int, NB>());
        }
    } else {
        const int s_begin = (a.ksteps * wk) / WK, s_end = (a.ksteps * (wk + 1)) / WK;
        u4 bcur[NB], bnxt[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j) bcur[j] = wp[(size_t)s_begin * wstep + j * 64];
        for (int s = s_begin; s < s_end; ++s) {
            const bool more = s + 1 < s_end;
            if (more) {
#pragma unroll
                for (int j = 0; j < NB; ++j) bnxt[j] = wp[(size_t)(s + 1) * wstep + j * 64];
            }
            int offs[LPE];
#pragma unroll
            for (int e = 0; e < LPE; ++e) offs[e] = offtab[s * KSTEP + g * LPE + e];
            u4 av[MB];
#pragma unroll
            for (int i = 0; i < MB; ++i) {
                TC v[LPE];
                const int base = abase[i] - g * LPE;
#pragma unroll
                for (int e = 0; e < LPE; ++e) v[e] = offs[e] >= 0 ? win_lds[base + offs[e]] : TC(0);
                __builtin_memcpy(&av[i], v, 16);
            }
            mma(av, bcur, std::integral_constant<int, NB>());
            if (more) {
#pragma unroll
                for (int j = 0; j < NB; ++j) bcur[j] = bnxt[j];
            }
        }
    }

    // ---- split-K reduction ----------------------------------------------------
    if constexpr (WK > 1) {
        constexpr int RV = MB * NB * 4;  // accumulator floats per lane
        float *part = reinterpret_cast<float *>(smem);
        __syncthreads();  // the window is no longer read
        if (wk > 0) {
            float *dst = part + ((size_t)((wk - 1) * WMN + wmn) * RV) * 64 + lane;
#pragma unroll
            for (int i = 0; i < MB; ++i)
#pragma unroll
                for (int j = 0; j < NB; ++j)
#pragma unroll
                    for (int e = 0; e < 4; ++e) dst[(size_t)((i * NB + j) * 4 + e) * 64] = acc[i][j][e];
        }
        __syncthreads();
        if (wk == 0) {
#pragma unroll
            for (int w = 1; w < WK; ++w) {
                const float *src = part + ((size_t)((w - 1) * WMN + wmn) * RV) * 64 + lane;
#pragma unroll
                for (int i = 0; i < MB; ++i)
#pragma unroll
                    for (int j = 0; j < NB; ++j)
#pragma unroll
                        for (int e = 0; e < 4; ++e) acc[i][j][e] += src[(size_t)((i * NB + j) * 4 + e) * 64];
            }
        }
    }

    // ---- epilogue (only the wk == 0 waves hold the sums) ----------------------
    if (a.head_ncls > 0) {
        float *red = reinterpret_cast<float *>(smem);
        __syncthreads();  // the LDS window / partial sums (which red reuses) are no longer read
        if (wk == 0) fused_head_partials<MB, NB, WN, BF>(a, acc, nb0, wm, wn, lm, g, red);
        __syncthreads();
        fused_head_finish<WN>(
            a, q / a.F, npix,
            [&](int m, int &hy, int &hx, int &y, int &x) {
                int seg;
                locate(m, seg, y, x);
                x += c0;
                hy = seg ? fy1 : fy;
                hx = seg ? fx1 : fx;
            },
            red, head_two_class<BF, NB>(a));
        return;
    }
    // Lane (lm, g) holds, for pixel lm of each m-block, rows 4g .. 4g + 3 of
    // each channel block: four consecutive channels (float32: 16 bytes) or,
    // with paired blocks in bf16, eight (16 bytes); other bf16 tiles hold 8
    // bytes per block.  Channels past c_out (padding blocks) and pixels past
    // the tile are not written.
    const bool act_tanh = a.act == ACT_TANH;
    auto act = [&](float v) { return act_tanh ? tanh_fast(v) : v; };
    constexpr bool PAIRED = BF && (NB % 2) == 0;
    constexpr int CRUN = PAIRED ? 8 : 4;  // consecutive channels per lane and block (pair)

    // LDS [pixel][channel] tile of act(acc + bias) (one 8- or 16-byte write per
    // run), for the restaged stores and the fused pool
    constexpr int NW = WN * NB * 16;            // channels this workgroup owns
    constexpr int TPAD = 16 / (int)sizeof(TC);  // 16 bytes of row padding
    constexpr int TS = NW + TPAD;
    // keys: bf16 runs are written as order keys (bf16x2_key), for the pool
    auto stage_tile = [&](TC *tile, bool keys) {
        if (wk != 0) return;
#pragma unroll
        for (int i = 0; i < MB; ++i) {
            TC *row = tile + ((wm * MB + i) * 16 + lm) * TS;
            if constexpr (PAIRED) {
#pragma unroll
                for (int p = 0; p < NB / 2; ++p) {
                    // channels 8g .. 8g + 3 from block 2p, 8g + 4 .. 8g + 7 from 2p + 1
                    float h[8];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        h[e] = act(acc[i][2 * p][e]);
                        h[4 + e] = act(acc[i][2 * p + 1][e]);
                    }
                    u4 pk;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        pk[e] = pack_bf16(h[2 * e], h[2 * e + 1]);
                        if (keys) pk[e] = bf16x2_key(pk[e]);
                    }
                    *reinterpret_cast<u4 *>(row + (wn * NB + 2 * p) * 16 + 8 * g) = pk;
                }
            } else {
#pragma unroll
                for (int j = 0; j < NB; ++j) {
                    TC *dst = row + (wn * NB + j) * 16 + 4 * g;
                    if constexpr (BF) {
                        uint2 pk;
                        pk.x = pack_bf16(act(acc[i][j][0]), act(acc[i][j][1]));
                        pk.y = pack_bf16(act(acc[i][j][2]), act(acc[i][j][3]));
                        if (keys) {
                            pk.x = bf16x2_key(pk.x);
                            pk.y = bf16x2_key(pk.y);
                        }
                        *reinterpret_cast<uint2 *>(dst) = pk;
                    } else {
                        *reinterpret_cast<f4 *>(dst) = f4{act(acc[i][j][0]), act(acc[i][j][1]), act(acc[i][j][2]),
                                                          act(acc[i][j][3])};
                    }
                }
            }
        }
    };

    if (!RUN && a.pool_ky) {
        // Fused k x k pool (the workgroup owns every channel): the filter
        // value at fragment position (y, x) = (y0 + r, c0 + c) is the
        // maximum over the tile's k x k outputs from (r, c), and goes to
        // child (o_y, o_x) = (y mod k, x mod k) at (y div k, x div k); the
        // child of (fy, fx) is fragment (fy*k + o_y, fx*k + o_x) of the next
        // layer (Qx*k fragments per row of its grid).  Per axis for a
        // k_y x k_x pool.  Same values as a separate pool kernel reading this
        // layer's stored (rounded) outputs.
        TC *tile = reinterpret_cast<TC *>(smem);
        __syncthreads();  // every wave is done with the window / partial sums
        stage_tile(tile, true);
        __syncthreads();
        const int kpy = a.pool_ky, kpx = a.pool_kx, ew = twb;
        const int Qc = a.Qx * kpx;
        const size_t child_px = (size_t)a.pool_oh * a.pool_ow;
        const size_t cbase = (size_t)(q / a.F) * a.F * kpy * kpx;  // first child of image b
        const Div dky(kpy), dkx(kpx), dtm(twM);
        auto child_ptr = [&](int r, int c) {
            int ybar, oy, xbar, ox;
            dky.qr(y0 + r, ybar, oy);
            dkx.qr(c0 + c, xbar, ox);
            const size_t qc = cbase + (size_t)(fy * kpy + oy) * Qc + (fx * kpx + ox);
            return reinterpret_cast<TC *>(a.out) + (qc * child_px + (size_t)ybar * a.pool_ow + xbar) * a.cout;
        };
        // filter value (y0 + r, c0 + c) lies inside its child (size (s - o) div k
        // per axis of a parent of s, Eqs. 6-7) and the child batch
        auto child_ok = [&](int r, int c) {
            int ybar, oy, xbar, ox;
            dky.qr(y0 + r, ybar, oy);
            dkx.qr(c0 + c, xbar, ox);
            [[maybe_unused]] const int hc = (hin - a.ky + 1 - oy) / kpy - a.dbg_shrink,
                                       wc = (win - a.kx + 1 - ox) / kpx - a.dbg_shrink;
            return FS_DBG_OK(a.dbg,
                             q < a.nfrag && ybar < hc && xbar < wc && ybar < a.pool_oh && xbar < a.pool_ow,
                             DBG_FUSED_POOL);
        };
        if ((a.cout % TPAD) == 0) {
            // A thread owns one 16-byte channel chunk v of one filter column
            // c and walks a run of consecutive filter rows, so its LDS source
            // and child addresses only advance: a row down in the tile, and
            // the next child row (o_y + 1, or o_y = 0 and ybar + 1).  With
            // fewer (column, chunk) pairs than threads the rows are shared
            // out as well.
            const int nv = a.cout / TPAD;
            const int items = twM * nv;
            const int nrg = max(1, 256 / items);   // row runs per (column, chunk)
            const int rpt = (rtM + nrg - 1) / nrg;  // rows per run
            const Div dit(items), dnv(nv);
            const long long d_oy = (long long)Qc * child_px * a.cout;  // next o_y: the child Qc fragments on
            const long long d_yb = (long long)a.pool_ow * a.cout;      // next ybar
            auto walk = [&](auto kc) {
                constexpr int KC = decltype(kc)::value;  // square pool size if known here, else 0
                const int KY = KC ? KC : kpy, KX = KC ? KC : kpx;
                for (int w = threadIdx.x; w < items * nrg; w += 256) {
                    int rg, it, c, v;
                    dit.qr(w, rg, it);
                    dnv.qr(it, c, v);
                    const int r0 = rg * rpt, r1 = min(r0 + rpt, rtM);
                    if (r0 >= r1) continue;
                    int ybar, oy;
                    dky.qr(y0 + r0, ybar, oy);
                    TC *dst = child_ptr(r0, c) + v * TPAD;
                    const TC *src = tile + __mul24(__mul24(r0, ew) + c, TS) + v * TPAD;
                    auto vmax = [&](u4 m, const u4 x) {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            if constexpr (BF)
                                m[e] = max_i16x2(m[e], x[e]);
                            else
                                m[e] = __float_as_uint(fmaxf(__uint_as_float(m[e]), __uint_as_float(x[e])));
                        }
                        return m;
                    };
                    auto put = [&](u4 m, int r) {
                        if constexpr (BF) {
#pragma unroll
                            for (int e = 0; e < 4; ++e) m[e] = bf16x2_key(m[e]);
                        }
                        if (child_ok(r, c)) *reinterpret_cast<u4 *>(dst) = m;
                        if (++oy == KY) {
                            oy = 0;
                            dst += d_yb - (KY - 1) * d_oy;
                        } else {
                            dst += d_oy;
                        }
                    };
                    if constexpr (KC > 0) {
                        // Separable: the filter value at row r is the maximum
                        // of the KC row maxima h(r) .. h(r + KC - 1), where
                        // h(rr) = max_j tile[rr][c + j]; a run keeps the last
                        // KC - 1 row maxima, so each row is read once per run
                        // (KC reads and 2 (KC - 1) maxima per value instead of
                        // KC^2 reads and KC^2 - 1 maxima).  max is exact, so
                        // the values are those of the direct form.
                        auto hrow = [&](const TC *row) {
                            u4 h = *reinterpret_cast<const u4 *>(row);
#pragma unroll
                            for (int j = 1; j < KC; ++j) h = vmax(h, *reinterpret_cast<const u4 *>(row + j * TS));
                            return h;
                        };
                        const int rstep = ew * TS;
                        u4 hr[KC];
#pragma unroll
                        for (int i = 0; i + 1 < KC; ++i) hr[i] = hrow(src + i * rstep);
                        src += (KC - 1) * rstep;
                        for (int r = r0; r < r1; ++r) {
                            hr[KC - 1] = hrow(src);
                            u4 m = hr[0];
#pragma unroll
                            for (int i = 1; i < KC; ++i) m = vmax(m, hr[i]);
                            put(m, r);
#pragma unroll
                            for (int i = 0; i + 1 < KC; ++i) hr[i] = hr[i + 1];
                            src += rstep;
                        }
                    } else {
                        for (int r = r0; r < r1; ++r) {
                            u4 m = *reinterpret_cast<const u4 *>(src);
                            for (int i = 0; i < KY; ++i)
                                for (int j = 0; j < KX; ++j)
                                    m = vmax(m, *reinterpret_cast<const u4 *>(src + __mul24(__mul24(i, ew) + j, TS)));
                            put(m, r);
                            src += ew * TS;
                        }
                    }
                }
            };
            if (kpy == 2 && kpx == 2)
                walk(std::integral_constant<int, 2>());
            else if (kpy == 3 && kpx == 3)
                walk(std::integral_constant<int, 3>());
            else
                walk(std::integral_constant<int, 0>());
        } else {
            const Div dco(a.cout);
            const int total = rtM * twM * a.cout;
            for (int idx = threadIdx.x; idx < total; idx += 256) {
                int p, ch, r, c;
                dco.qr(idx, p, ch);
                dtm.qr(p, r, c);
                const TC *src = tile + __mul24(__mul24(r, ew) + c, TS) + ch;
                TC m = src[0];
                for (int i = 0; i < kpy; ++i)
                    for (int j = 0; j < kpx; ++j) {
                        const TC x = src[__mul24(__mul24(i, ew) + j, TS)];
                        if constexpr (BF)
                            m = (TC)max_i16x2(m, x);  // keys in the low half
                        else
                            m = fmaxf(m, x);
                    }
                if constexpr (BF) m = (TC)bf16x2_key(m);
                if (child_ok(r, c)) child_ptr(r, c)[ch] = m;
            }
        }
        return;
    }

    if (!a.direct_store) {
        // Restaged: all threads copy the tile out in 16-byte pieces; the
        // pixels of a band row are contiguous in memory, so a tile row leaves
        // as one contiguous run.
        const int nbase = blockIdx.y * NW;
        TC *tile = reinterpret_cast<TC *>(smem);
        __syncthreads();  // every wave is done with the window / partial sums
        stage_tile(tile, false);
        __syncthreads();
        const size_t osz = (size_t)a.out_h * a.out_w * a.cout;
        TC *outp = reinterpret_cast<TC *>(a.out) + (size_t)q * osz + nbase;
        TC *outp1 = reinterpret_cast<TC *>(a.out) + (size_t)q1 * osz + nbase;
        const int orow = a.out_w * a.cout;
        const int nch = min(NW, a.cout - nbase);
        if ((a.cout % TPAD) == 0 && (nch % TPAD) == 0) {
            const int nv = nch / TPAD;
            const Div dnv(nv);
            for (int idx = threadIdx.x; idx < npix * nv; idx += 256) {
                int m, v, seg, y, x;
                dnv.qr(idx, m, v);
                locate(m, seg, y, x);
                x += c0;
                if (!write_ok(seg, y, x)) continue;
                *reinterpret_cast<u4 *>((seg ? outp1 : outp) + (y * orow + __mul24(x, a.cout) + v * TPAD)) =
                    *reinterpret_cast<const u4 *>(tile + __mul24(m, TS) + v * TPAD);
            }
        } else {
            const Div dnc(nch);
            for (int idx = threadIdx.x; idx < npix * nch; idx += 256) {
                int m, c, seg, y, x;
                dnc.qr(idx, m, c);
                locate(m, seg, y, x);
                x += c0;
                if (!write_ok(seg, y, x)) continue;
                (seg ? outp1 : outp)[y * orow + __mul24(x, a.cout) + c] = tile[__mul24(m, TS) + c];
            }
        }
        return;
    }

    // Direct: every lane writes its runs straight from registers.
    if (wk != 0) return;
    const size_t osz = (size_t)a.out_h * a.out_w * a.cout;
    TC *outp = reinterpret_cast<TC *>(a.out) + (size_t)q * osz;
    TC *outp1 = reinterpret_cast<TC *>(a.out) + (size_t)q1 * osz;
    const int orow = a.out_w * a.cout;
    const bool full = (a.cout % CRUN) == 0;
#pragma unroll
    for (int i = 0; i < MB; ++i) {
        const int m = (wm * MB + i) * 16 + lm;
        if (m >= npix) continue;
        int seg, y, x;
        locate(m, seg, y, x);
        x += c0;
        if (!write_ok(seg, y, x)) continue;
        TC *px = (seg ? outp1 : outp) + (y * orow + __mul24(x, a.cout));
        if constexpr (PAIRED) {
#pragma unroll
            for (int p = 0; p < NB / 2; ++p) {
                const int ch = (nb0 + 2 * p) * 16 + 8 * g;
                if (ch >= a.cout) continue;
                float h[8];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    h[e] = act(acc[i][2 * p][e]);
                    h[4 + e] = act(acc[i][2 * p + 1][e]);
                }
                u4 pk;
#pragma unroll
                for (int e = 0; e < 4; ++e) pk[e] = pack_bf16(h[2 * e], h[2 * e + 1]);
                if (full) {
                    *reinterpret_cast<u4 *>(px + ch) = pk;
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (ch + e < a.cout) px[ch + e] = (uint16_t)(pk[e / 2] >> (16 * (e % 2)));
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const int ch = (nb0 + j) * 16 + 4 * g;
                if (ch >= a.cout) continue;
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = act(acc[i][j][e]);
                if constexpr (BF) {
                    uint2 pk;
                    pk.x = pack_bf16(v[0], v[1]);
                    pk.y = pack_bf16(v[2], v[3]);
                    if (full) {
                        *reinterpret_cast<uint2 *>(px + ch) = pk;
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (ch + e < a.cout) px[ch + e] = (uint16_t)((e < 2 ? pk.x : pk.y) >> (16 * (e % 2)));
                    }
                } else {
                    if (full) {
                        *reinterpret_cast<f4 *>(px + ch) = f4{v[0], v[1], v[2], v[3]};
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (ch + e < a.cout) px[ch + e] = v[e];
                    }
                }
            }
        }
    }
}

template <int MB, int NB, int WN, int WK, bool BF, bool IN_F32, bool VEC, bool RUN>
hipError_t launch_one(const ConvArgs &a, int gx, int gy, hipStream_t s)
{
    auto kern = conv_frag_mfma<MB, NB, WN, WK, BF, IN_F32, VEC, RUN>;
    if (a.lds_bytes > 65536) {
        // the instance may take up to a whole CU's LDS: set once per device
        // (a runtime call per launch cost tens of microseconds of host time)
        static std::atomic<uint64_t> done{0};
        int dev = 0;
        (void)hipGetDevice(&dev);
        const uint64_t bit = 1ull << (dev & 63);
        if (!(done.load(std::memory_order_acquire) & bit)) {
            hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLdsBytes);
            if (e != hipSuccess) {
                (void)hipGetLastError();  // do not leave it to be reported by a later launch
                return e;
            }
            done.fetch_or(bit, std::memory_order_acq_rel);
        }
    }
    hipLaunchKernelGGL(kern, dim3(gx, gy), dim3(256), a.lds_bytes, s, a);
    return hipGetLastError();
}

// The register tiles each operand variant is built for: (MB, NB, WN, WK).
#define FS_CONV_TILES_VEC(X)                                                                    \
    X(1, 1, 1, 1) X(1, 2, 1, 1) X(1, 3, 1, 1) X(1, 4, 1, 1) X(2, 1, 1, 1) X(2, 2, 1, 1)          \
    X(2, 3, 1, 1) X(2, 4, 1, 1) X(4, 1, 1, 1) X(4, 2, 1, 1) X(4, 3, 1, 1) X(4, 4, 1, 1)          \
    X(1, 7, 1, 1) X(1, 8, 1, 1) X(1, 13, 1, 1) X(2, 7, 1, 1) X(2, 8, 1, 1) X(2, 13, 1, 1)        \
    X(2, 2, 2, 1) X(2, 4, 2, 1) X(2, 7, 2, 1) X(4, 2, 2, 1) X(4, 4, 2, 1) X(4, 7, 2, 1)          \
    X(4, 2, 4, 1) X(4, 4, 4, 1) X(8, 2, 4, 1) X(8, 4, 4, 1)                                      \
    X(4, 1, 1, 2) X(4, 2, 1, 2) X(4, 3, 1, 2) X(4, 4, 1, 2) X(8, 1, 1, 4) X(8, 2, 1, 4)          \
    X(8, 3, 1, 4) X(8, 4, 1, 4) X(4, 7, 2, 2) X(4, 4, 2, 2) X(4, 2, 2, 2) X(4, 7, 1, 2)          \
    X(2, 13, 1, 2) X(8, 1, 1, 1) X(8, 2, 1, 1) X(4, 7, 1, 1) X(4, 8, 1, 1) X(8, 2, 2, 1)
#define FS_CONV_TILES_GATHER(X)                                                                 \
    X(1, 1, 1, 1) X(1, 2, 1, 1) X(1, 3, 1, 1) X(1, 4, 1, 1) X(2, 1, 1, 1) X(2, 2, 1, 1)          \
    X(2, 3, 1, 1) X(2, 4, 1, 1) X(4, 1, 1, 1) X(4, 2, 1, 1) X(4, 3, 1, 1) X(4, 4, 1, 1)
// ... and with run tiles (a subset: those one-band layers take)
#define FS_CONV_TILES_RUN_VEC(X)                                                                \
    X(2, 2, 1, 1) X(2, 4, 1, 1) X(2, 7, 1, 1) X(2, 13, 1, 1) X(4, 2, 1, 1) X(4, 3, 1, 2)         \
    X(4, 4, 1, 1) X(4, 7, 2, 1)
#define FS_CONV_TILES_RUN_GATHER(X) \
    X(2, 1, 1, 1) X(2, 2, 1, 1) X(2, 3, 1, 1) X(2, 4, 1, 1) X(4, 1, 1, 1) X(4, 2, 1, 1)

// Workgroups of one tile shape that fit on a CU with `lds` dynamic LDS bytes
// (0 if unknown or the shape has no instance): a 256-thread workgroup
// puts one wave on each of the 4 SIMDs, each SIMD holds 512 VGPRs per lane
// (allocated in granules of 8), and the CU has kMaxLdsBytes of LDS.
template <bool BF, bool IN_F32, bool VEC>
int tile_blocks_per_cu(int mb, int nb, int wn, int wk, bool run, int lds)
{
    const void *kern = nullptr;
#define FS_CONV_OCC(M, N, W, K) \
    if (mb == M && nb == N && wn == W && wk == K) kern = reinterpret_cast<const void *>(conv_frag_mfma<M, N, W, K, BF, IN_F32, VEC, false>);
#define FS_CONV_OCC_RUN(M, N, W, K) \
    if (mb == M && nb == N && wn == W && wk == K) kern = reinterpret_cast<const void *>(conv_frag_mfma<M, N, W, K, BF, IN_F32, VEC, true>);
    if (run) {
        if constexpr (VEC) {
            FS_CONV_TILES_RUN_VEC(FS_CONV_OCC_RUN)
        } else {
            FS_CONV_TILES_RUN_GATHER(FS_CONV_OCC_RUN)
        }
    } else {
        if constexpr (VEC) {
            FS_CONV_TILES_VEC(FS_CONV_OCC)
        } else {
            FS_CONV_TILES_GATHER(FS_CONV_OCC)
        }
    }
#undef FS_CONV_OCC
#undef FS_CONV_OCC_RUN
    if (!kern) return 0;
    hipFuncAttributes fa{};
    if (hipFuncGetAttributes(&fa, kern) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    const int regs = (fa.numRegs + 7) / 8 * 8;
    int n = regs > 0 ? 512 / regs : 8;
    if (lds > 0) n = std::min(n, (int)(kMaxLdsBytes / (size_t)lds));
    return std::min(n, 8);
}

template <bool BF, bool IN_F32, bool VEC>
hipError_t dispatch_tile(const ConvArgs &a, int mb, int nb, int wn, int wk, int gx, int gy, hipStream_t s)
{
#define FS_CONV_CASE(M, N, W, K) \
    if (mb == M && nb == N && wn == W && wk == K) return launch_one<M, N, W, K, BF, IN_F32, VEC, false>(a, gx, gy, s);
#define FS_CONV_CASE_RUN(M, N, W, K) \
    if (mb == M && nb == N && wn == W && wk == K) return launch_one<M, N, W, K, BF, IN_F32, VEC, true>(a, gx, gy, s);
    if (a.run) {
        if constexpr (VEC) {
            FS_CONV_TILES_RUN_VEC(FS_CONV_CASE_RUN)
        } else {
            FS_CONV_TILES_RUN_GATHER(FS_CONV_CASE_RUN)
        }
    } else {
        if constexpr (VEC) {
            FS_CONV_TILES_VEC(FS_CONV_CASE)
        } else {
            FS_CONV_TILES_GATHER(FS_CONV_CASE)
        }
    }
#undef FS_CONV_CASE
#undef FS_CONV_CASE_RUN
    return hipErrorInvalidValue;
}

}  // namespace conv
}  // namespace fs
