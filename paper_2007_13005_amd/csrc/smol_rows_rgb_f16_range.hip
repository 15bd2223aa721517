// smol_rows_rgb_f16_range.hip -- RGB row-streaming kernels, fp16 output, contiguous row ranges, NCHW output.
#include "smol_rows_rgb.h"

namespace smol {

const void *rows_rgb_f16_range(const BatchArgs &a) { return rgb_rows_table<1, 0, 0>(a); }

}  // namespace smol
