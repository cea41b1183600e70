// Fragment-batched convolution on the CDNA4 matrix cores (implicit GEMM).
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
//     pixels (64 * MB: four waves, MB blocks of 16 pixels each).  So tiles
//     follow the fragment's true size with waste only at a band's end.
//   - The workgroup stages the input window its tile needs (all rows the
//     tile's pixels touch, band + k - 1 columns, all c_in channels) in LDS
//     once, zero-filled outside the fragment's true size.
//   - Each wave computes MB x NB blocks of 16 pixels x 16 output channels with
//     v_mfma_f32_16x16x4_f32 (float32) or v_mfma_f32_16x16x32_bf16 (bfloat16,
//     float32 accumulate).  A lane (lm = lane % 16, g = lane / 16) feeds pixel
//     lm of each block and 16 bytes of consecutive K values starting at
//     g * (KSTEP / 4); the weight operand is pre-arranged on the host so every
//     (K step, channel block) is one contiguous 1 KB run that a wave reads in
//     a single coalesced load.
//   - Vector path (c_in a multiple of KSTEP): K is walked tap by tap, KSTEP
//     channels at a time, and the A operand is one 16-byte LDS read.  Gather
//     path (small c_in, e.g. the first layer): K = (tap, channel) flattened
//     and padded to KSTEP, operands gathered through an LDS offset table.
//   - Epilogue: bias, activation (tanh) in float32, store (bf16: round to
//     nearest even) only inside the fragment's true size.
#include "fs_internal.h"

#include <type_traits>

namespace fs {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint16_t f2bf(float f)
{
    // round to nearest even; inputs here are finite
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
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

template <int MB, int NB, bool BF, bool IN_F32, bool VEC>
__global__ __launch_bounds__(256) void conv_frag_mfma(ConvArgs a)
{
    using TC = typename Elem<BF>::T;               // LDS / operand element
    using TI = typename std::conditional<IN_F32, float, TC>::type;  // global input element
    constexpr int KSTEP = Elem<BF>::KSTEP;
    constexpr int LPE = KSTEP / 4;                 // elements per lane per K step (16 bytes)

    extern __shared__ __align__(16) unsigned char smem[];

    int bid = blockIdx.x;
    const int t = bid % a.tiles_per_band;
    bid /= a.tiles_per_band;
    const int band = bid % a.nbands;
    const int q = bid / a.nbands;
    const int nb0 = blockIdx.y * NB;

    const int rem = q % a.F;
    const int fy = rem / a.Q, fx = rem - (rem / a.Q) * a.Q;
    const int hin = a.ext.y[fy], win = a.ext.x[fx];
    const int hout = hin - a.k + 1, wout = win - a.k + 1;
    if (hout <= 0 || wout <= 0) return;
    const int c0 = band * a.band_w;
    const int twb = min(a.band_w, wout - c0);
    if (twb <= 0) return;
    const int npix = hout * twb;
    const int l0 = t * a.mt;
    if (l0 >= npix) return;
    const int lend = min(l0 + a.mt, npix);
    const int yfirst = l0 / twb;
    const int ylast = (lend - 1) / twb;
    const int R = ylast - yfirst + a.k;   // window rows
    const int Cc = twb + a.k - 1;         // window columns
    const int CS = a.lds_cs;
    const int kk_total = a.ksteps * KSTEP;

    int *offtab = reinterpret_cast<int *>(smem);
    TC *win_lds = reinterpret_cast<TC *>(smem + (VEC ? 0 : ((kk_total * 4 + 15) & ~15)));

    // ---- stage the input window --------------------------------------------
    const TI *inp = reinterpret_cast<const TI *>(a.in) + (size_t)q * a.in_h * a.in_w * a.in_c;
    if constexpr (VEC && !IN_F32) {
        const int nvec = a.cin / LPE;
        const int total = R * Cc * nvec;
        for (int idx = threadIdx.x; idx < total; idx += 256) {
            const int v = idx % nvec;
            const int p = idx / nvec;
            const int c = p % Cc, r = p / Cc;
            const int gy = yfirst + r, gx = c0 + c;
            u4 val = {0u, 0u, 0u, 0u};
            if (gy < hin && gx < win)
                val = *reinterpret_cast<const u4 *>(inp + ((size_t)gy * a.in_w + gx) * a.in_c + v * LPE);
            *reinterpret_cast<u4 *>(win_lds + (r * Cc + c) * CS + v * LPE) = val;
        }
    } else {
        const int total = R * Cc * a.cin;
        for (int idx = threadIdx.x; idx < total; idx += 256) {
            const int ci = idx % a.cin;
            const int p = idx / a.cin;
            const int c = p % Cc, r = p / Cc;
            const int gy = yfirst + r, gx = c0 + c;
            TC val = 0;
            if (gy < hin && gx < win) {
                TI x = inp[((size_t)gy * a.in_w + gx) * a.in_c + ci];
                if constexpr (BF && IN_F32)
                    val = f2bf(x);
                else
                    val = x;
            }
            win_lds[(r * Cc + c) * CS + ci] = val;
        }
    }
    if constexpr (!VEC) {
        for (int kk = threadIdx.x; kk < kk_total; kk += 256) {
            const int tap = kk / a.cin, ci = kk - (kk / a.cin) * a.cin;
            int off = -1;
            if (tap < a.k * a.k) {
                const int dy = tap / a.k, dx = tap - (tap / a.k) * a.k;
                off = (dy * Cc + dx) * CS + ci;
            }
            offtab[kk] = off;
        }
    }
    __syncthreads();

    // ---- matrix-core main loop ----------------------------------------------
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int lm = lane & 15, g = lane >> 4;

    int abase[MB];
#pragma unroll
    for (int i = 0; i < MB; ++i) {
        const int l = l0 + (wv * MB + i) * 16 + lm;
        if (l < lend) {
            const int y = l / twb - yfirst, x = l - (l / twb) * twb;
            abase[i] = (y * Cc + x) * CS;
        } else {
            abase[i] = 0;  // any in-window address; the result is not stored
        }
    }

    f4 acc[MB][NB];
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    const u4 *wp = reinterpret_cast<const u4 *>(a.w) + (size_t)nb0 * 64 + lane;

    auto mma = [&](const u4 (&av)[MB], const u4 (&bv)[NB]) {
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

    if constexpr (VEC) {
        const int ncc = a.cin / KSTEP;
        int s = 0;
        for (int dy = 0; dy < a.k; ++dy) {
            for (int dx = 0; dx < a.k; ++dx) {
                const TC *tp = win_lds + (dy * Cc + dx) * CS + g * LPE;
                for (int cc = 0; cc < ncc; ++cc, ++s) {
                    u4 bv[NB];
#pragma unroll
                    for (int j = 0; j < NB; ++j) bv[j] = wp[((size_t)s * a.nbt + j) * 64];
                    u4 av[MB];
#pragma unroll
                    for (int i = 0; i < MB; ++i)
                        av[i] = *reinterpret_cast<const u4 *>(tp + abase[i] + cc * KSTEP);
                    mma(av, bv);
                }
            }
        }
    } else {
        for (int s = 0; s < a.ksteps; ++s) {
            u4 bv[NB];
#pragma unroll
            for (int j = 0; j < NB; ++j) bv[j] = wp[((size_t)s * a.nbt + j) * 64];
            int offs[LPE];
#pragma unroll
            for (int e = 0; e < LPE; ++e) offs[e] = offtab[s * KSTEP + g * LPE + e];
            u4 av[MB];
#pragma unroll
            for (int i = 0; i < MB; ++i) {
                TC v[LPE];
#pragma unroll
                for (int e = 0; e < LPE; ++e) v[e] = offs[e] >= 0 ? win_lds[abase[i] + offs[e]] : TC(0);
                __builtin_memcpy(&av[i], v, 16);
            }
            mma(av, bv);
        }
    }

    // ---- epilogue -------------------------------------------------------------
    TC *outp = reinterpret_cast<TC *>(a.out) + (size_t)q * a.out_h * a.out_w * a.cout;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int co = (nb0 + j) * 16 + lm;
        if (co >= a.cout) continue;
        const float bv = a.bias[co];
#pragma unroll
        for (int i = 0; i < MB; ++i) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int l = l0 + (wv * MB + i) * 16 + 4 * g + e;
                if (l >= lend) continue;
                const int y = l / twb, x = c0 + (l - (l / twb) * twb);
                float v = acc[i][j][e] + bv;
                if (a.act == ACT_TANH) v = tanhf(v);
                TC *dst = outp + ((size_t)y * a.out_w + x) * a.cout + co;
                if constexpr (BF)
                    *dst = f2bf(v);
                else
                    *dst = v;
            }
        }
    }
}

template <int MB, int NB, bool BF, bool IN_F32, bool VEC>
hipError_t launch_one(const ConvArgs &a, int gx, int gy, hipStream_t s)
{
    auto kern = conv_frag_mfma<MB, NB, BF, IN_F32, VEC>;
    if (a.lds_bytes > 65536) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, a.lds_bytes);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3(gx, gy), dim3(256), a.lds_bytes, s, a);
    return hipGetLastError();
}

template <bool BF, bool IN_F32, bool VEC>
hipError_t dispatch_tile(const ConvArgs &a, int mb, int nb, int gx, int gy, hipStream_t s)
{
#define FS_CONV_CASE(M, N) \
    if (mb == M && nb == N) return launch_one<M, N, BF, IN_F32, VEC>(a, gx, gy, s);
    FS_CONV_CASE(1, 1) FS_CONV_CASE(1, 2) FS_CONV_CASE(1, 3) FS_CONV_CASE(1, 4)
    FS_CONV_CASE(2, 1) FS_CONV_CASE(2, 2) FS_CONV_CASE(2, 3) FS_CONV_CASE(2, 4)
    FS_CONV_CASE(4, 1) FS_CONV_CASE(4, 2) FS_CONV_CASE(4, 3) FS_CONV_CASE(4, 4)
    if constexpr (VEC) {
        FS_CONV_CASE(1, 7) FS_CONV_CASE(1, 8) FS_CONV_CASE(1, 13)
        FS_CONV_CASE(2, 7) FS_CONV_CASE(2, 8) FS_CONV_CASE(2, 13)
    }
#undef FS_CONV_CASE
    return hipErrorInvalidValue;
}

}  // namespace

bool conv_tile_supported(int mb, int nb)
{
    if (mb != 1 && mb != 2 && mb != 4) return false;
    if (nb >= 1 && nb <= 4) return true;
    return mb <= 2 && (nb == 7 || nb == 8 || nb == 13);
}

hipError_t launch_conv(const ConvArgs &a, int dtype, bool in_f32, int mb, int nb, bool vec,
                       int grid_x, int grid_y, hipStream_t s)
{
    if (dtype == DT_F32) {
        return vec ? dispatch_tile<false, false, true>(a, mb, nb, grid_x, grid_y, s)
                   : dispatch_tile<false, false, false>(a, mb, nb, grid_x, grid_y, s);
    }
    if (in_f32) {
        if (vec) return hipErrorInvalidValue;
        return dispatch_tile<true, true, false>(a, mb, nb, grid_x, grid_y, s);
    }
    return vec ? dispatch_tile<true, false, true>(a, mb, nb, grid_x, grid_y, s)
               : dispatch_tile<true, false, false>(a, mb, nb, grid_x, grid_y, s);
}

const char *conv_kernel_name(int dtype, bool in_f32, int mb, int nb, bool vec)
{
    static thread_local char buf[64];
    snprintf(buf, sizeof buf, "conv_frag_mfma<%d,%d,%s%s,%s>", mb, nb, dtype == DT_BF16 ? "bf16" : "f32",
             in_f32 && dtype == DT_BF16 ? "<-f32" : "", vec ? "vec" : "gather");
    return buf;
}

}  // namespace fs
