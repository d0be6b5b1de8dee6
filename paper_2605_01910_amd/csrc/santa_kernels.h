// santa_kernels.h -- host-side launchers of the decode kernels (internal).
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

#include "santa_plan.h"

namespace santa {

// Events the GPU records around the kernels of one call (santa_time_next_call):
// `start` when the call's first kernel is dispatched, `stop` when its last
// kernel completes.  Null events launch normally.  Thread-local, consumed by
// the next santa_decode_* or santa_stream_read call on the thread.
struct CallTimer {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};
CallTimer &call_timer();

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

// Streaming-read calibration (santa_stream_read): at most `max_groups`
// workgroups read `bytes` (a multiple of 16) from buf; sink[w] gets workgroup
// w's XOR fold (words past the grid are left as they were).
hipError_t launch_stream_read(const void *buf, size_t bytes, uint32_t *sink, int max_groups,
                              hipStream_t st);

// Bernoulli query weights, selected-feature lists and the feature mask of
// every GQA group (k_bern_prep); `start` (nullable) is recorded at dispatch.
hipError_t launch_bern_prep(const Plan &p, const void *q, int Bd, int mode, const float *u_q,
                            float *bw, int *blist, int *bn, uint8_t *mask_out, hipStream_t st,
                            hipEvent_t start);

hipError_t launch_fused_bernoulli(const Plan &p, const KvView &kv, const KtView &kt,
                                 const void *q, float scale_log2, int Bd, int mode,
                                 const float *u_q, const float *u, int32_t *idx_out,
                                 uint8_t *mask_out, void *out, char *ws, hipStream_t st);

hipError_t launch_fused_dense(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                              void *out, char *ws, hipStream_t st);

// rows: the scheduled flash kernel (k_row_flash) in place of k_fused_dense's flash mode
hipError_t launch_fused_flash(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                              int tile_log2, int S_tile, const float *u, int32_t *idx_out,
                              void *out, char *ws, hipStream_t st, bool rows);

// mode: 0 systematic, 1 stratified, 2 i.i.d. (thresholds by exponential spacings)
hipError_t launch_fused_sampled(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                                int mode, const float *u, int32_t *idx_out, void *out, char *ws,
                                hipStream_t st);

// Compile-time dispatch over the GQA group size, element type and cache kind.
template <typename F>
inline hipError_t with_g(int G, F &&f) {
  switch (G) {
    case 1: return f(std::integral_constant<int, 1>{});
    case 2: return f(std::integral_constant<int, 2>{});
    case 4: return f(std::integral_constant<int, 4>{});
    case 8: return f(std::integral_constant<int, 8>{});
  }
  return hipErrorInvalidValue;
}

template <typename F>
inline hipError_t with_types(const Plan &p, bool paged, F &&f) {
  return with_g(p.G, [&](auto gc) -> hipError_t {
    if (p.dtype == 0) {
      if (paged) return f((uint16_t *)nullptr, gc, std::true_type{});
      return f((uint16_t *)nullptr, gc, std::false_type{});
    }
    if (paged) return f((float *)nullptr, gc, std::true_type{});
    return f((float *)nullptr, gc, std::false_type{});
  });
}

}  // namespace santa
