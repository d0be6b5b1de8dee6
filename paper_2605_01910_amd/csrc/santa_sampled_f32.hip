// santa_sampled_f32.hip -- sampled kernels instantiated for float32 elements.
#include "santa_sampled.h"

namespace santa {

template hipError_t launch_one_launch_e<float>(const Plan &, const KvView &, const void *, float, int, const float *, int32_t *, void *, char *, hipStream_t);

}  // namespace santa
