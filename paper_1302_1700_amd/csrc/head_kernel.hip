// Last stage of the scan: the last 1 x 1 layer (when it is one), its
// activation, and the reassembly of the final fragments into the dense map.
//
// Output semantics: the net returns class posterior probabilities (Section 1),
// so a last layer marked softmax gives exp(z - max z) / sum exp(z - max z) over
// its classes, computed in float32.
//
// Reassembly: the window with top-left corner (Y, X) is held by one final
// fragment (Section 3: the fragments together cover every window).  With pool
// sizes k_1..k_P and S = k_1 * ... * k_P, the offsets a window's corner
// selects at the successive pools are the mixed-radix digits of Y mod S (least
// significant first: o_1 = Y mod k_1, then (Y div k_1) mod k_2, ...), and its
// position inside the fragment is Y div S; the same holds for X, with the
// pools' column sizes.  The host turns "Y mod S_y -> row index of the
// fragment grid" (and the same for X) into small tables.
//
// Mapping: LPP = kHeadLanesPerPixel lanes per output pixel, consecutive groups
// take consecutive output pixels, so the dense output is written contiguously
// while each group reads its fragment pixel's channel vector contiguously
// (16-byte loads); the dot products over the channels are finished with
// cross-lane xor shuffles.  A workgroup's 256 / LPP groups take
// kHeadPixelsPerGroup runs of 256 / LPP consecutive pixels, one run after the
// other, so the weights it stages in LDS serve that many more pixels.  The
// per-pixel work every lane of a group repeats (coordinates, softmax) is why
// the groups are narrow: with 16 lanes per pixel, one run per workgroup and
// the coordinates divided out per pixel the kernel moved 2.0 TB/s on N4
// 8 x 1024^2; with 4 lanes, 4 runs and incremental coordinates 3.9 TB/s
// (2, 8 or 1 lanes and 1, 2 or 8 runs measured slower).
#include "fs_internal.h"

namespace fs {
namespace {

typedef uint32_t u4 __attribute__((ext_vector_type(4)));

template <bool BF, bool IN_F32, bool HAS_FC, int V>
__global__ __launch_bounds__(256) void head_softmax_reassemble(HeadArgs a)
{
    using TI = typename std::conditional<BF && !IN_F32, uint16_t, float>::type;
    __shared__ float wl[HAS_FC ? kMaxHeadWeights : 1];
    __shared__ float bl[kMaxHeadClasses];

    const int ncls = a.ncls;
    if constexpr (HAS_FC) {
        for (int i = threadIdx.x; i < ncls * a.C; i += 256) wl[i] = a.w[i];
    }
    if (threadIdx.x < kMaxHeadClasses) bl[threadIdx.x] = threadIdx.x < ncls ? a.bias[threadIdx.x] : 0.f;
    __syncthreads();

    constexpr int LPP = kHeadLanesPerPixel, GPW = 256 / LPP;  // lanes per pixel, groups per workgroup
    const int sub = threadIdx.x & (LPP - 1);
    const long long npix = (long long)a.B * a.ny * a.nx;
    // The group's pixel: image b, window (Y, X) = (yf * Sy + ym, xf * Sx + xm).
    // Divided out once; each later run moves GPW pixels on, which advances the
    // coordinates by additions (a column digit wraps, a row ends, an image
    // ends), since per-pixel integer divisions had dominated the kernel.
    long long gp = (long long)blockIdx.x * kHeadPixelsPerGroup * GPW + threadIdx.x / LPP;
    if (gp >= npix) return;
    const long long plane = (long long)a.ny * a.nx;
    int b = (int)(gp / plane);
    const int r0 = (int)(gp - (long long)b * plane);
    int Y = r0 / a.nx, X = r0 - Y * a.nx;
    int yf = Y / a.Sy, ym = Y - yf * a.Sy;
    int xf = X / a.Sx, xm = X - xf * a.Sx;
    for (int run = 0; run < kHeadPixelsPerGroup; ++run) {
        if (run > 0) {
            gp += GPW;
            if (gp >= npix) return;
            X += GPW;
            xm += GPW;
            while (xm >= a.Sx) {
                xm -= a.Sx;
                ++xf;
            }
            if (X >= a.nx) {
                do {  // past the row's end: the next row, or the next image
                    X -= a.nx;
                    ++Y;
                    if (++ym == a.Sy) {
                        ym = 0;
                        ++yf;
                    }
                    if (Y == a.ny) {
                        Y = 0;
                        ym = 0;
                        yf = 0;
                        ++b;
                    }
                } while (X >= a.nx);
                xf = X / a.Sx;
                xm = X - xf * a.Sx;
            }
        }
        const int fy = a.digit_y[ym], fx = a.digit_x[xm];
        const size_t q = (size_t)b * a.F + (size_t)fy * a.Qx + fx;
        // the fragment pixel lies inside its final fragment, the window inside the map
        if (!FS_DBG_OK(a.dbg,
                       b < a.B && yf < a.ext.y[fy] - a.dbg_shrink && xf < a.ext.x[fx] - a.dbg_shrink && yf < a.in_h &&
                           xf < a.in_w,
                       DBG_HEAD_READ))
            continue;
        if (!FS_DBG_OK(a.dbg, Y < a.ny && X < a.nx && Y < a.out_ny && X < a.out_nx, DBG_HEAD_WRITE)) continue;
        const TI *src = reinterpret_cast<const TI *>(a.in) + ((q * a.in_h + yf) * a.in_w + xf) * a.C;

        float z[kMaxHeadClasses];
#pragma unroll
        for (int c = 0; c < kMaxHeadClasses; ++c) z[c] = 0.f;

        if constexpr (HAS_FC) {
            const int nv = a.C / V;
            for (int cv = sub; cv < nv; cv += LPP) {
                float v[V];
                if constexpr (V == 1) {
                    if constexpr (BF && !IN_F32) v[0] = __uint_as_float((uint32_t)src[cv] << 16);
                    else v[0] = src[cv];
                } else {
                    u4 raw = *reinterpret_cast<const u4 *>(src + cv * V);
                    if constexpr (BF && !IN_F32) {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            v[2 * e] = __uint_as_float(raw[e] << 16);
                            v[2 * e + 1] = __uint_as_float(raw[e] & 0xffff0000u);
                        }
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e) v[e] = __uint_as_float(raw[e]);
                    }
                }
#pragma unroll
                for (int c = 0; c < kMaxHeadClasses; ++c) {
                    if (c < ncls) {
                        const float *wr = wl + c * a.C + cv * V;
#pragma unroll
                        for (int e = 0; e < V; ++e) z[c] = fmaf(wr[e], v[e], z[c]);
                    }
                }
            }
#pragma unroll
            for (int c = 0; c < kMaxHeadClasses; ++c) {
                if (c < ncls) {
                    float t = z[c];
#pragma unroll
                    for (int d = LPP / 2; d >= 1; d /= 2) t += __shfl_xor(t, d);
                    z[c] = t + bl[c];
                }
            }
        } else {
#pragma unroll
            for (int c = 0; c < kMaxHeadClasses; ++c) {
                if (c < ncls) {
                    if constexpr (BF && !IN_F32) z[c] = __uint_as_float((uint32_t)src[c] << 16);
                    else z[c] = src[c];
                }
            }
        }

        if (a.act == ACT_SOFTMAX) {
            float m = z[0];
#pragma unroll
            for (int c = 1; c < kMaxHeadClasses; ++c)
                if (c < ncls) m = fmaxf(m, z[c]);
            float s = 0.f;
#pragma unroll
            for (int c = 0; c < kMaxHeadClasses; ++c) {
                if (c < ncls) {
                    z[c] = __expf(z[c] - m);  // z - m <= 0: the hardware exp2, a few ulp
                    s += z[c];
                }
            }
            const float inv = 1.0f / s;
#pragma unroll
            for (int c = 0; c < kMaxHeadClasses; ++c) z[c] *= inv;
        } else if (a.act == ACT_TANH) {
#pragma unroll
            for (int c = 0; c < kMaxHeadClasses; ++c) z[c] = tanhf(z[c]);
        }

        // lane sub writes classes sub, sub + LPP, ...
#pragma unroll
        for (int c0 = 0; c0 < kMaxHeadClasses; c0 += LPP) {
            float mine = 0.f;
#pragma unroll
            for (int c = c0; c < c0 + LPP && c < kMaxHeadClasses; ++c)
                if (c - c0 == sub) mine = z[c];
            if (c0 + sub < ncls) a.out[(((size_t)b * a.out_ny + Y) * a.out_nx + X) * ncls + c0 + sub] = mine;
        }
    }
}

template <bool BF, bool IN_F32, bool HAS_FC, int V>
hipError_t go(const HeadArgs &a, int grid, hipStream_t s)
{
    hipLaunchKernelGGL((head_softmax_reassemble<BF, IN_F32, HAS_FC, V>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_head(const HeadArgs &a, int dtype, bool in_f32, bool has_fc, int grid, hipStream_t s)
{
    const bool bf_in = dtype == DT_BF16 && !in_f32;
    if (!has_fc) {
        if (bf_in) return go<true, false, false, 1>(a, grid, s);
        return go<false, true, false, 1>(a, grid, s);
    }
    if (bf_in) return (a.C % 8 == 0) ? go<true, false, true, 8>(a, grid, s) : go<true, false, true, 1>(a, grid, s);
    return (a.C % 4 == 0) ? go<false, true, true, 4>(a, grid, s) : go<false, true, true, 1>(a, grid, s);
}

const char *head_kernel_name(int dtype, bool in_f32, bool has_fc)
{
    const bool bf_in = dtype == DT_BF16 && !in_f32;
    if (!has_fc) return bf_in ? "head_softmax_reassemble<bf16,nofc>" : "head_softmax_reassemble<f32,nofc>";
    return bf_in ? "head_softmax_reassemble<bf16,fc>" : "head_softmax_reassemble<f32,fc>";
}

}  // namespace fs
