// santa_rows_fp8.hip -- scheduled sampled and flash kernels instantiated for FP8 E4M3 caches (bfloat16 queries and outputs).
#include "santa_rows.h"

namespace santa {

template hipError_t launch_rows_e<uint8_t>(const Plan &, const KvView &, const void *, float, int, const float *, int32_t *, void *, char *, hipStream_t);
template hipError_t launch_row_flash_e<uint8_t>(const Plan &, const KvView &, const void *, float, int, int, const float *, int32_t *, void *, char *, hipStream_t);

}  // namespace santa
