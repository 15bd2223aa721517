// smol_rows_yuv_stride_nhwc.hip -- I420 row-streaming kernels, rows strided across waves, NHWC output.
#include "smol_rows_yuv.h"

namespace smol {

const void *rows_yuv_stride_nhwc(const BatchArgs &a, int f16) { return yuv_rows_table<1, 1>(a, f16); }

}  // namespace smol
