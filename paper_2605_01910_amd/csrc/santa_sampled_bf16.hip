// santa_sampled_bf16.hip -- sampled kernels instantiated for bfloat16 elements.
#include "santa_sampled.h"

namespace santa {

template hipError_t launch_one_launch_e<uint16_t>(const Plan &, const KvView &, const void *, float, int, const float *, int32_t *, void *, char *, hipStream_t);

}  // namespace santa
