// smol_rows_rgb_f32_range_nhwc.hip -- RGB row-streaming kernels, fp32 output, contiguous row ranges, NHWC output.
#include "smol_rows_rgb.h"

namespace smol {

const void *rows_rgb_f32_range_nhwc(const BatchArgs &a) { return rgb_rows_table<0, 0, 1>(a); }

}  // namespace smol
