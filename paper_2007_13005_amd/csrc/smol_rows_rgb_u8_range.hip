// smol_rows_rgb_u8_range.hip -- RGB row-streaming kernels, uint8 output (rounded resized values), contiguous row ranges.
#include "smol_rows_rgb.h"

namespace smol {

// uint8 output is not normalised: the exact and the default normalisation are the same kernel
const void *rows_rgb_u8_range(const BatchArgs &a)
{
    return rgb_rows_f<2, 0, 0, 0>(a);
}

}  // namespace smol
