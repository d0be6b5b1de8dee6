// santa_sampled_fp8.hip -- sampled kernels instantiated for FP8 E4M3 caches (bfloat16 queries and outputs).
#include "santa_sampled.h"

namespace santa {

template hipError_t launch_one_launch_e<uint8_t>(const Plan &, const KvView &, const void *, float, int, const float *, int32_t *, void *, char *, hipStream_t);

}  // namespace santa
