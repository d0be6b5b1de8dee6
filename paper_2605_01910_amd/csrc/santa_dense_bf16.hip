// santa_dense_bf16.hip -- dense kernels instantiated for bfloat16 elements.
#include "santa_dense.h"

namespace santa {

template hipError_t launch_dense_e<uint16_t>(const Plan &, const KvView &, const void *, float, void *, char *, hipStream_t);
template hipError_t launch_flash_e<uint16_t>(const Plan &, const KvView &, const void *, float, int, int, const float *, int32_t *, void *, char *, hipStream_t);

}  // namespace santa
