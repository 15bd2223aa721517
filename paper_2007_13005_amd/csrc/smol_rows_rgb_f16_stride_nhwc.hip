// smol_rows_rgb_f16_stride_nhwc.hip -- RGB row-streaming kernels, fp16 output, rows strided across waves, NHWC output.
#include "smol_rows_rgb.h"

namespace smol {

const void *rows_rgb_f16_stride_nhwc(const BatchArgs &a) { return rgb_rows_table<1, 1, 1>(a); }

}  // namespace smol
