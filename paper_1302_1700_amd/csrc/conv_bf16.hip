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

}  // namespace fs
