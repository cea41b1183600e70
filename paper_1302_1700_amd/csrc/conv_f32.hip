// float32 instances of the fragment-batched convolution (conv_impl.h) and the
// convolution launcher.
#include "conv_ws.h"

#include <cstdio>

namespace fs {

hipError_t launch_conv_bf16(const ConvArgs &a, bool in_f32, int mb, int nb, int wn, int wk, bool vec, int gx,
                            int gy, hipStream_t s);
hipError_t launch_conv_ws_bf16(const ConvArgs &a, int mb, int nb, int wn, int gx, int gy, hipStream_t s);

bool conv_ws_supported(int mb, int nb, int wn)
{
#define FS_WS_HAS(M, N, W) \
    if (mb == M && nb == N && wn == W) return true;
    FS_CONV_TILES_WS(FS_WS_HAS)
#undef FS_WS_HAS
    return false;
}

hipError_t launch_conv_ws(const ConvArgs &a, int dtype, int mb, int nb, int wn, int gx, int gy, hipStream_t s)
{
    if (dtype == DT_BF16) return launch_conv_ws_bf16(a, mb, nb, wn, gx, gy, s);
    return conv::dispatch_ws<false>(a, mb, nb, wn, gx, gy, s);
}

int conv_ws_occupancy(int dtype, int mb, int nb, int wn, int lds_bytes)
{
    int n = 0;
#define FS_WS_OCC(M, N, W)                                                                               \
    if (mb == M && nb == N && wn == W) {                                                                 \
        const void *k = dtype == DT_BF16 ? reinterpret_cast<const void *>(conv::conv_frag_ws<M, N, W, true>) \
                                         : reinterpret_cast<const void *>(conv::conv_frag_ws<M, N, W, false>); \
        if (lds_bytes > 65536 &&                                                                         \
            hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes) != hipSuccess) \
            return 0;                                                                                    \
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k, 512, lds_bytes) != hipSuccess) return 0; \
        return n;                                                                                        \
    }
    FS_CONV_TILES_WS(FS_WS_OCC)
#undef FS_WS_OCC
    return 0;
}

std::string conv_ws_kernel_name(int dtype, int mb, int nb, int wn)
{
    char buf[96];
    snprintf(buf, sizeof buf, "conv_frag_ws<%d, %d, %d, %s>", mb, nb, wn, dtype == DT_BF16 ? "true" : "false");
    return buf;
}

bool conv_tile_supported(int mb, int nb, int wn, int wk, bool vec)
{
#define FS_CONV_HAS(M, N, W, K) \
    if (mb == M && nb == N && wn == W && wk == K) return true;
    if (vec) {
        FS_CONV_TILES_VEC(FS_CONV_HAS)
    } else {
        FS_CONV_TILES_GATHER(FS_CONV_HAS)
    }
#undef FS_CONV_HAS
    return false;
}

hipError_t launch_conv(const ConvArgs &a, int dtype, bool in_f32, int mb, int nb, int wn, int wk, bool vec,
                       int gx, int gy, hipStream_t s)
{
    if (dtype == DT_BF16) return launch_conv_bf16(a, in_f32, mb, nb, wn, wk, vec, gx, gy, s);
    return vec ? conv::dispatch_tile<false, false, true>(a, mb, nb, wn, wk, gx, gy, s)
               : conv::dispatch_tile<false, false, false>(a, mb, nb, wn, wk, gx, gy, s);
}

std::string conv_kernel_name(int dtype, bool in_f32, int mb, int nb, int wn, int wk, bool vec)
{
    char buf[96];
    const bool bf = dtype == DT_BF16;
    snprintf(buf, sizeof buf, "conv_frag_mfma<%d, %d, %d, %d, %s, %s, %s>", mb, nb, wn, wk, bf ? "true" : "false",
             bf && in_f32 ? "true" : "false", vec ? "true" : "false");
    return buf;
}

}  // namespace fs
