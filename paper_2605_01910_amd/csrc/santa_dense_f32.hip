// santa_dense_f32.hip -- dense kernels instantiated for float32 elements.
#include "santa_dense.h"

namespace santa {

template hipError_t launch_dense_e<float>(const Plan &, const KvView &, const void *, float, void *, char *, hipStream_t);
template hipError_t launch_flash_e<float>(const Plan &, const KvView &, const void *, float, int, int, const float *, int32_t *, void *, char *, hipStream_t);

}  // namespace santa
