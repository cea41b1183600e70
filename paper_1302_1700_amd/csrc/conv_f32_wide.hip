// The float32 4 x 13 register tile of the fragment-batched convolution
// (conv_impl.h): four pixel blocks by thirteen 16-channel blocks per wave,
// four waves across the pixels, so one workgroup covers 256 pixels by 208
// channels (a 200-output fully connected layer without a padding block).
// Its 208 accumulator registers per lane only fit beside the operands in the
// accumulation register file, so this file is compiled without the
// ordinary-register accumulation form the other instances use (build.py);
// at 464 registers per lane it runs one wave per SIMD.
#include "conv_impl.h"

namespace fs {

hipError_t launch_conv_f32_wide(const ConvArgs &a, int gx, int gy, hipStream_t s)
{
    return conv::launch_one<4, 13, 1, 1, false, false, true, false>(a, gx, gy, s);
}

}  // namespace fs
