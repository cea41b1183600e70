// float32 instances of the fragment-batched convolution (conv_impl.h) and the
// convolution launcher.
#include "conv_impl.h"

#include <array>
#include <cstdio>
#include <map>
#include <mutex>

namespace fs {

hipError_t launch_conv_bf16(const ConvArgs &a, bool in_f32, int mb, int nb, int wn, int wk, bool vec, int gx,
                            int gy, hipStream_t s);
int conv_blocks_per_cu_bf16(bool in_f32, int mb, int nb, int wn, int wk, bool vec, bool run, int lds);

int conv_blocks_per_cu(int dtype, bool in_f32, int mb, int nb, int wn, int wk, bool vec, bool run, int lds)
{
    // memoised per device and kernel shape (plans are rebuilt on every scan)
    static std::mutex mu;
    static std::map<std::array<int, 10>, int> memo;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    const std::array<int, 10> key{dev, dtype, in_f32, mb, nb, wn, wk, vec, lds, run};
    {
        std::lock_guard<std::mutex> g(mu);
        auto it = memo.find(key);
        if (it != memo.end()) return it->second;
    }
    int n;
    if (dtype != DT_BF16 && vec && !run && mb == 4 && nb == 13 && wn == 1 && wk == 1)
        n = lds > 0 && (size_t)lds <= kMaxLdsBytes ? 1 : 0;  // 464 registers per lane: one wave per SIMD
    else if (dtype == DT_BF16)
        n = conv_blocks_per_cu_bf16(in_f32, mb, nb, wn, wk, vec, run, lds);
    else
        n = vec ? conv::tile_blocks_per_cu<false, false, true>(mb, nb, wn, wk, run, lds)
                : conv::tile_blocks_per_cu<false, false, false>(mb, nb, wn, wk, run, lds);
    std::lock_guard<std::mutex> g(mu);
    memo[key] = n;
    return n;
}

bool conv_tile_supported(int mb, int nb, int wn, int wk, bool vec, bool run)
{
#define FS_CONV_HAS(M, N, W, K) \
    if (mb == M && nb == N && wn == W && wk == K) return true;
    if (run) {
        if (vec) {
            FS_CONV_TILES_RUN_VEC(FS_CONV_HAS)
        } else {
            FS_CONV_TILES_RUN_GATHER(FS_CONV_HAS)
        }
    } else if (vec) {
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
    if (vec && !a.run && mb == 4 && nb == 13 && wn == 1 && wk == 1) return launch_conv_f32_wide(a, gx, gy, s);
    return vec ? conv::dispatch_tile<false, false, true>(a, mb, nb, wn, wk, gx, gy, s)
               : conv::dispatch_tile<false, false, false>(a, mb, nb, wn, wk, gx, gy, s);
}

std::string conv_kernel_name(int dtype, bool in_f32, int mb, int nb, int wn, int wk, bool vec, bool run)
{
    char buf[96];
    const bool bf = dtype == DT_BF16;
    snprintf(buf, sizeof buf, "conv_frag_mfma<%d, %d, %d, %d, %s, %s, %s, %s>", mb, nb, wn, wk, bf ? "true" : "false",
             bf && in_f32 ? "true" : "false", vec ? "true" : "false", run ? "true" : "false");
    return buf;
}

}  // namespace fs
