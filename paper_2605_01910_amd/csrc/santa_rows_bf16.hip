// santa_rows_bf16.hip -- scheduled sampled and flash kernels instantiated for bfloat16 elements.
#include "santa_rows.h"

namespace santa {

template hipError_t launch_rows_e<uint16_t>(const Plan &, const KvView &, const void *, float, int, const float *, int32_t *, void *, char *, hipStream_t);
template hipError_t launch_row_flash_e<uint16_t>(const Plan &, const KvView &, const void *, float, int, int, const float *, int32_t *, void *, char *, hipStream_t);

}  // namespace santa
