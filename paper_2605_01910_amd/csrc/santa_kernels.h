// santa_kernels.h -- host-side launchers of the decode kernels (internal).
#pragma once

#include <hip/hip_runtime.h>

#include "santa_plan.h"

namespace santa {

hipError_t launch_dense(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                        void *out, char *ws, hipStream_t st);

hipError_t launch_sampled(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                          bool strat, const float *u, int32_t *idx_out, void *out, char *ws,
                          hipStream_t st);

hipError_t launch_bernoulli(const Plan &p, const KvView &kv, const KtView &kt, const void *q,
                            float scale_log2, int Bd, int mode, const float *u_q, const float *u,
                            int32_t *idx_out, uint8_t *mask_out, void *out, char *ws,
                            hipStream_t st);

hipError_t launch_zero(void *ws, size_t bytes, hipStream_t st);

}  // namespace santa
