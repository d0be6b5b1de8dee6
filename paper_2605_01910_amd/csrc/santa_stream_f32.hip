// santa_stream_f32.hip -- stream kernels instantiated for float32 elements.
#include "santa_stream.h"

namespace santa {

template hipError_t launch_two_launch_e<float>(const Plan &, const KvView &, const void *, float, int, const float *, int32_t *, void *, char *, hipStream_t);
template hipError_t launch_bernoulli_e<float>(const Plan &, const KvView &, const KtView &, const void *, float, int, int, const float *, const float *, int32_t *, uint8_t *, void *, char *, hipStream_t);

}  // namespace santa
