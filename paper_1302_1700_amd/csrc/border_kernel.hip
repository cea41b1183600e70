// Mirrored borders (Section 3.2: the image's edges are mirrored so that the
// net can be applied at every position): builds the extended image
// [B][H + h_0 - 1][W + w_0 - 1][C] the scan then reads, p0 rows / columns
// before the image and (window side) - 1 - p0 after it, per axis.  One thread per extended
// element, so the writes are contiguous; the reads follow the mirrored
// index, contiguous inside the image and reversed in the borders.
#include "fs_internal.h"

namespace fs {
namespace {

// Image index for extended index i (may be negative or >= n), period 2(n - 1)
// mirrored about the edge pixels (reflect) or period 2n with the edge pixels
// repeated (symmetric).
__device__ __forceinline__ int mirror_index(int i, int n, int mode)
{
    if (mode == BORDER_REFLECT) {
        if (n == 1) return 0;
        const int p = 2 * (n - 1);
        i %= p;
        if (i < 0) i += p;
        return i >= n ? p - i : i;
    }
    const int p = 2 * n;
    i %= p;
    if (i < 0) i += p;
    return i >= n ? p - 1 - i : i;
}

__global__ __launch_bounds__(256) void mirror_pad(const float *__restrict__ in, float *__restrict__ out, int B, int H,
                                                  int W, int C, int p0y, int p0x, int He, int We, int mode,
                                                  long long total, unsigned *dbg, int dbg_shrink)
{
    for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < total; e += (long long)gridDim.x * 256) {
        const int c = (int)(e % C);
        long long p = e / C;
        const int x = (int)(p % We);
        p /= We;
        const int y = (int)(p % He);
        const long long b = p / He;
        const int sy = mirror_index(y - p0y, H, mode), sx = mirror_index(x - p0x, W, mode);
        if (!FS_DBG_OK(dbg, b < B && sy >= 0 && sx >= 0 && sy < H - dbg_shrink && sx < W - dbg_shrink, DBG_PAD_READ))
            continue;
        out[e] = in[((b * H + sy) * W + sx) * C + c];
    }
}

}  // namespace

hipError_t launch_mirror_pad(const float *in, float *out, int B, int H, int W, int C, int p0y, int p0x, int He,
                             int We, int mode, unsigned *dbg, int dbg_shrink, hipStream_t s)
{
    const long long total = (long long)B * He * We * C;
    const long long blocks = (total + 255) / 256;
    const int grid = (int)(blocks < 65536 ? blocks : 65536);
    hipLaunchKernelGGL(mirror_pad, dim3(grid), dim3(256), 0, s, in, out, B, H, W, C, p0y, p0x, He, We, mode, total,
                       dbg, dbg_shrink);
    return hipGetLastError();
}

}  // namespace fs
