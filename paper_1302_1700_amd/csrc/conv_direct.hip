// Direct (vector-ALU) convolution for layers with very few input channels,
// typically the first layer reading the image: K = c_in * k * k is so small
// (12 .. 64) that a matrix-core tile would spend its time gathering operands,
// while the layer's cost is writing its c_out-channel output.  Same arithmetic
// as the fragment-batched convolution (Section 2.2.1: valid cross-correlation
// of every fragment, sizes shrinking by k - 1):
//   out[q, y, x, co] = act(bias[co] + sum_{dy, dx, ci} W[co, ci, dy, dx] * in[q, y+dy, x+dx, ci]).
// One thread per output pixel: it loads its K inputs once, then walks the
// output channels four (f32) or eight (bf16) at a time and writes each group
// with one 16-byte store; neighbouring threads own neighbouring pixels, so the
// output rows are written contiguously.  The weights, repacked on the host as
// [c_out][KP] (zero padded), are read at wave-uniform addresses, so they
// arrive through scalar loads and feed the multiply-adds as scalar operands.
// bf16: the image and weights are rounded to bf16 first (products exact in
// f32), accumulation in f32, the result rounded to bf16.
#include "fs_internal.h"

#include <type_traits>

namespace fs {
namespace {

typedef uint32_t u4 __attribute__((ext_vector_type(4)));
constexpr int kMaxK = 64;

__device__ __forceinline__ uint16_t f2bf(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bfround(float f) { return __uint_as_float((uint32_t)f2bf(f) << 16); }

__device__ __forceinline__ float tanh_fast(float x)
{
    const float t = __builtin_amdgcn_exp2f(x * 2.8853900817779268f);
    return 1.0f - 2.0f * __builtin_amdgcn_rcpf(t + 1.0f);
}

template <bool BF, bool IN_F32, int KP>  // KP: K rounded up, a multiple of 4
__global__ __launch_bounds__(256) void conv_direct(ConvArgs a, const float *__restrict__ wpk)
{
    using TO = typename std::conditional<BF, uint16_t, float>::type;
    using TI = typename std::conditional<IN_F32 || !BF, float, uint16_t>::type;
    constexpr int G = BF ? 8 : 4;  // channels per 16-byte store
    __shared__ int offs[KP];
    __shared__ float bl[64];
    // output staging (dynamic): 4 waves x 64 pixels x (c_out + 16 bytes)
    extern __shared__ __align__(16) unsigned char ostage[];

    const int K = a.cin * a.ky * a.kx;
    for (int kk = threadIdx.x; kk < KP; kk += 256) {
        int o = 0;  // padding taps read pixel (0, 0) and have zero weight
        if (kk < K) {
            const int tap = kk / a.cin, ci = kk - (kk / a.cin) * a.cin;
            const int dy = tap / a.kx, dx = tap - (tap / a.kx) * a.kx;
            o = (dy * a.in_w + dx) * a.in_c + ci;
        }
        offs[kk] = o;
    }
    const int rows = (a.cout + 7) / 8 * 8;  // weight rows (zero past c_out), then the bias
    if (threadIdx.x < 64) bl[threadIdx.x] = threadIdx.x < a.cout ? wpk[(size_t)rows * KP + threadIdx.x] : 0.f;
    __syncthreads();

    // blockIdx.x -> (fragment q, chunk of 256 pixels of the padded output box)
    const int per_frag = (a.out_h * a.out_w + 255) / 256;
    const int q = blockIdx.x / per_frag;
    const int pix0 = (blockIdx.x - q * per_frag) * 256;
    const int pix = pix0 + threadIdx.x;
    const int y = pix / a.out_w, x = pix - (pix / a.out_w) * a.out_w;
    const int rem = q % a.F;
    const int fy = rem / a.Qx, fx = rem - (rem / a.Qx) * a.Qx;
    const int hout = a.ext.y[fy] - a.ky + 1, wout = a.ext.x[fx] - a.kx + 1;
    const bool valid = pix < a.out_h * a.out_w && y < hout && x < wout;

    const TI *inp = reinterpret_cast<const TI *>(a.in) + (size_t)q * a.in_h * a.in_w * a.in_c +
                    (valid ? ((size_t)y * a.in_w + x) * a.in_c : 0);
    // a valid pixel's window lies inside its fragment's true size; the others
    // read the window at (0, 0), inside the storage
    [[maybe_unused]] const int ry = (valid ? y : 0) + a.ky - 1, rx = (valid ? x : 0) + a.kx - 1;
    const bool rd = FS_DBG_OK(a.dbg,
                              q < a.nfrag && ry < a.in_h && rx < a.in_w &&
                                  (!valid || (ry < a.ext.y[fy] - a.dbg_shrink && rx < a.ext.x[fx] - a.dbg_shrink)),
                              DBG_CONV_READ);
    float xin[KP];
#pragma unroll
    for (int kk = 0; kk < KP; ++kk) {
        const TI raw = rd ? inp[offs[kk]] : TI(0);
        float v;
        if constexpr (BF && !IN_F32) v = __uint_as_float((uint32_t)raw << 16);
        else v = raw;
        if constexpr (BF && IN_F32) v = bfround(v);
        xin[kk] = v;
    }
    // Each wave's 64 pixels are 64 consecutive positions of the padded output
    // box: one contiguous run of 64 * cout elements.  Results go to LDS
    // [pixel][channel] first and leave with consecutive lanes storing
    // consecutive 16-byte chunks.
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int cpad = (a.cout + G - 1) / G * G;
    const int rs = cpad + G;  // row stride (elements): +16 bytes against bank conflicts
    TO *stage = reinterpret_cast<TO *>(ostage) + wv * 64 * rs;
    for (int c0 = 0; c0 < cpad; c0 += G) {
        float z[G];
#pragma unroll
        for (int gg = 0; gg < G; ++gg) {
            float acc = bl[c0 + gg];
            const float *wr = wpk + (size_t)(c0 + gg) * KP;
#pragma unroll
            for (int kk = 0; kk < KP; ++kk) acc = fmaf(wr[kk], xin[kk], acc);
            if (a.act == ACT_TANH) acc = tanh_fast(acc);
            z[gg] = acc;
        }
        u4 pk;
        if constexpr (BF) {
#pragma unroll
            for (int e = 0; e < 4; ++e) pk[e] = (uint32_t)f2bf(z[2 * e]) | ((uint32_t)f2bf(z[2 * e + 1]) << 16);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) pk[e] = __float_as_uint(z[e]);
        }
        *reinterpret_cast<u4 *>(stage + lane * rs + c0) = pk;
    }
    __syncthreads();
    TO *out = reinterpret_cast<TO *>(a.out) + ((size_t)q * a.out_h * a.out_w + pix0 + wv * 64) * a.cout;
    const int wpix0 = pix0 + wv * 64;
    auto write_ok = [&](int py, int px) {
        return FS_DBG_OK(a.dbg, q < a.nfrag && py < hout - a.dbg_shrink && px < wout - a.dbg_shrink, DBG_CONV_WRITE);
    };
    if ((a.cout % G) == 0) {
        const int ng = a.cout / G;
        for (int ch = lane; ch < 64 * ng; ch += 64) {
            const int p = ch / ng, grp = ch - (ch / ng) * ng;
            const int pp = wpix0 + p;
            const int py = pp / a.out_w, px = pp - (pp / a.out_w) * a.out_w;
            if (pp < a.out_h * a.out_w && py < hout && px < wout && write_ok(py, px))
                *reinterpret_cast<u4 *>(out + (size_t)ch * G) = *reinterpret_cast<const u4 *>(stage + p * rs + grp * G);
        }
    } else {
        for (int e = lane; e < 64 * a.cout; e += 64) {
            const int p = e / a.cout, c = e - (e / a.cout) * a.cout;
            const int pp = wpix0 + p;
            const int py = pp / a.out_w, px = pp - (pp / a.out_w) * a.out_w;
            if (pp < a.out_h * a.out_w && py < hout && px < wout && write_ok(py, px)) out[e] = stage[p * rs + c];
        }
    }
}

template <bool BF, bool IN_F32>
hipError_t go(const ConvArgs &a, const float *wpk, int grid, hipStream_t s)
{
    const int K = a.cin * a.ky * a.kx;
    constexpr int G = BF ? 8 : 4;
    const int cpad = (a.cout + G - 1) / G * G;
    const size_t lds = (size_t)4 * 64 * (cpad + G) * (BF ? 2 : 4);
    if (K <= 16) hipLaunchKernelGGL((conv_direct<BF, IN_F32, 16>), dim3(grid), dim3(256), lds, s, a, wpk);
    else if (K <= 32) hipLaunchKernelGGL((conv_direct<BF, IN_F32, 32>), dim3(grid), dim3(256), lds, s, a, wpk);
    else if (K <= 64) hipLaunchKernelGGL((conv_direct<BF, IN_F32, 64>), dim3(grid), dim3(256), lds, s, a, wpk);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace

bool conv_direct_supported(int cin, int taps, int cout) { return cin * taps <= kMaxK && cout <= 48; }

int conv_direct_kp(int cin, int taps)
{
    const int K = cin * taps;
    return K <= 16 ? 16 : K <= 32 ? 32 : 64;
}

hipError_t launch_conv_direct(const ConvArgs &a, const float *wpk, int dtype, bool in_f32, int grid, hipStream_t s)
{
    if (dtype == DT_F32) return go<false, true>(a, wpk, grid, s);
    if (in_f32) return go<true, true>(a, wpk, grid, s);
    return go<true, false>(a, wpk, grid, s);
}

std::string conv_direct_kernel_name(int dtype, bool in_f32, int cin, int taps)
{
    const int K = cin * taps;
    const int kp = K <= 16 ? 16 : K <= 32 ? 32 : 64;
    const bool bf = dtype == DT_BF16;
    return std::string("conv_direct<") + (bf ? "true" : "false") + ", " + (bf && !in_f32 ? "false" : "true") +
           ", " + std::to_string(kp) + ">";
}

}  // namespace fs
