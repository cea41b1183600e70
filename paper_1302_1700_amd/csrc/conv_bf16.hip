// bfloat16 instances of the fragment-batched convolution (conv_impl.h).
#include "conv_impl.h"

namespace fs {

hipError_t launch_conv_bf16(const ConvArgs &a, bool in_f32, int mb, int nb, int wn, int wk, bool vec, int gx,
                            int gy, hipStream_t s)
{
    if (in_f32) {
        if (vec) return hipErrorInvalidValue;
        return conv::dispatch_tile<true, true, false>(a, mb, nb, wn, wk, gx, gy, s);
    }
    return vec ? conv::dispatch_tile<true, false, true>(a, mb, nb, wn, wk, gx, gy, s)
               : conv::dispatch_tile<true, false, false>(a, mb, nb, wn, wk, gx, gy, s);
}

int conv_blocks_per_cu_bf16(bool in_f32, int mb, int nb, int wn, int wk, bool vec, bool run, int lds)
{
    if (in_f32) return vec ? 0 : conv::tile_blocks_per_cu<true, true, false>(mb, nb, wn, wk, run, lds);
    return vec ? conv::tile_blocks_per_cu<true, false, true>(mb, nb, wn, wk, run, lds)
               : conv::tile_blocks_per_cu<true, false, false>(mb, nb, wn, wk, run, lds);
}

}  // namespace fs
