// smol_rows_yuv_range_nhwc.hip -- I420 row-streaming kernels, contiguous row ranges, NHWC output.
#include "smol_rows_yuv.h"

namespace smol {

const void *rows_yuv_range_nhwc(const BatchArgs &a, int f16) { return yuv_rows_table<0, 1>(a, f16); }

}  // namespace smol
