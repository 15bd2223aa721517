// smol_rows_rgb_f16_stride.hip -- RGB row-streaming kernels, fp16 output, rows strided across waves, NCHW output.
#include "smol_rows_rgb.h"

namespace smol {

const void *rows_rgb_f16_stride(const BatchArgs &a) { return rgb_rows_table<1, 1, 0>(a); }

}  // namespace smol
