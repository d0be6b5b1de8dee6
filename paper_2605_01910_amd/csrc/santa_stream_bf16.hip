// santa_stream_bf16.hip -- stream kernels instantiated for bfloat16 elements.
#include "santa_stream.h"

namespace santa {

template hipError_t launch_two_launch_e<uint16_t>(const Plan &, const KvView &, const void *, float, int, const float *, int32_t *, void *, char *, hipStream_t);
template hipError_t launch_bernoulli_e<uint16_t>(const Plan &, const KvView &, const KtView &, const void *, float, int, int, const float *, const float *, int32_t *, uint8_t *, void *, char *, hipStream_t);

}  // namespace santa
