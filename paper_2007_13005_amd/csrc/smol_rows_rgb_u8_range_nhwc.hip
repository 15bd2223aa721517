// smol_rows_rgb_u8_range_nhwc.hip -- RGB row-streaming kernels, uint8 output (rounded resized values), contiguous row ranges, NHWC output.
#include "smol_rows_rgb.h"

namespace smol {

// uint8 output is not normalised: the exact and the default normalisation are the same kernel
const void *rows_rgb_u8_range_nhwc(const BatchArgs &a)
{
    return rgb_rows_f<2, 0, 0, 1>(a);
}

}  // namespace smol
