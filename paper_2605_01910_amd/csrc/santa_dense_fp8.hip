// santa_dense_fp8.hip -- dense kernels instantiated for FP8 E4M3 caches (bfloat16 queries and outputs).
#include "santa_dense.h"

namespace santa {

template hipError_t launch_dense_e<uint8_t>(const Plan &, const KvView &, const void *, float, void *, char *, hipStream_t);
template hipError_t launch_flash_e<uint8_t>(const Plan &, const KvView &, const void *, float, int, int, const float *, int32_t *, void *, char *, hipStream_t);

}  // namespace santa
