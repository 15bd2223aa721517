// smol_rows_yuv_range.hip -- I420 row-streaming kernels, contiguous row ranges, NCHW output.
#include "smol_rows_yuv.h"

namespace smol {

const void *rows_yuv_range(const BatchArgs &a, int f16) { return yuv_rows_table<0, 0>(a, f16); }

}  // namespace smol
