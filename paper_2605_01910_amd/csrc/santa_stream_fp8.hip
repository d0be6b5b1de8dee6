// santa_stream_fp8.hip -- stream kernels instantiated for FP8 E4M3 caches (bfloat16 queries and outputs).
#include "santa_stream.h"

namespace santa {

template hipError_t launch_two_launch_e<uint8_t>(const Plan &, const KvView &, const void *, float, int, const float *, int32_t *, void *, char *, hipStream_t);

}  // namespace santa
