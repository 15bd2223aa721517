// smol_rows_rgb_f32_stride.hip -- RGB row-streaming kernels, fp32 output, rows strided across waves, NCHW output.
#include "smol_rows_rgb.h"

namespace smol {

const void *rows_rgb_f32_stride(const BatchArgs &a) { return rgb_rows_table<0, 1, 0>(a); }

}  // namespace smol
