// smol_rows_yuv_stride.hip -- I420 row-streaming kernels, rows strided across waves, NCHW output.
#include "smol_rows_yuv.h"

namespace smol {

const void *rows_yuv_stride(const BatchArgs &a, int f16) { return yuv_rows_table<1, 0>(a, f16); }

}  // namespace smol
