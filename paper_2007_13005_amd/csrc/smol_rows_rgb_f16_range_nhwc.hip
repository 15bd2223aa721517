// smol_rows_rgb_f16_range_nhwc.hip -- RGB row-streaming kernels, fp16 output, contiguous row ranges, NHWC output.
#include "smol_rows_rgb.h"

namespace smol {

const void *rows_rgb_f16_range_nhwc(const BatchArgs &a) { return rgb_rows_table<1, 0, 1>(a); }

}  // namespace smol
