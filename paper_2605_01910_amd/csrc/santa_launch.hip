// santa_launch.hip -- host side of the default kernels: occupancy, the
// resident launch, the kernel argument block, and dispatch over the element
// type to the per-type launchers of santa_sampled.h, santa_stream.h and
// santa_dense.h.
#include <mutex>

#include "santa_fused.h"

namespace santa {

namespace {
struct OccKey {
  const void *fn;
  int dev;
  size_t lds;
};
}  // namespace

int capacity_of(const void *fn, size_t lds) {
  static OccKey keys[256];
  static int vals[256];
  static int n = 0;
  static std::mutex mu;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  std::lock_guard<std::mutex> lock(mu);
  for (int i = 0; i < n; ++i)
    if (keys[i].fn == fn && keys[i].dev == dev && keys[i].lds == lds) return vals[i];
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kThreads, lds) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  const int cap = per_cu * cus;
  if (n < 256) {
    keys[n] = OccKey{fn, dev, lds};
    vals[n] = cap;
    ++n;
  }
  return cap;
}

hipError_t launch_resident(const void *fn, const Plan &p, FusedArgs &args, size_t lds,
                           hipStream_t st) {
  const int nrk = p.B * p.Hkv;
  const int cap = capacity_of(fn, lds);
  if (cap < p.T) return hipErrorInvalidConfiguration;
  const int R = std::min(nrk, cap / p.T);
  void *params[] = {&args};
  const CallTimer tm = call_timer();
  return hipExtLaunchKernel(fn, dim3(R * p.T), dim3(kThreads), params, lds, st, tm.start, tm.stop,
                            0);
}

FusedArgs make_args(const Plan &p, const KvView &kv, const void *q, void *out, float scale_log2,
                    char *ws) {
  FusedArgs a{};
  a.kv = kv;
  a.q = q;
  a.out = out;
  a.stats = reinterpret_cast<float2 *>(ws + p.off_stats);
  a.part = p.off_part ? reinterpret_cast<float *>(ws + p.off_part) : nullptr;
  a.qstash = p.off_stash ? reinterpret_cast<uint16_t *>(ws + p.off_stash) : nullptr;
  a.coarse = p.off_coarse ? reinterpret_cast<float *>(ws + p.off_coarse) : nullptr;
  a.sync = p.off_sync ? reinterpret_cast<unsigned long long *>(ws + p.off_sync) : nullptr;
  a.err = reinterpret_cast<int *>(ws + p.off_err);
  a.B = p.B;
  a.Hq = p.Hq;
  a.Hkv = p.Hkv;
  a.T = p.T;
  a.Ls = p.Ls;
  a.S = p.S;
  a.npitch = p.npitch;
  a.invS = p.S ? 1.0f / (float)p.S : 0.0f;
  a.scale_log2 = scale_log2;
  return a;
}

// Element type of the cache: bf16 (uint16_t bit patterns), float, or FP8
// E4M3 codes (uint8_t; q and out bf16).
template <typename F>
static hipError_t with_elem(const Plan &p, F &&f) {
  if (p.elem == 2) return f((uint8_t *)nullptr);
  if (p.elem == 0) return f((uint16_t *)nullptr);
  return f((float *)nullptr);
}

hipError_t launch_fused_sampled(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                                int mode, const float *u, int32_t *idx_out, void *out, char *ws,
                                hipStream_t st) {
  return with_elem(p, [&](auto eptr) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    if (p.rows) return launch_rows_e<E>(p, kv, q, scale_log2, mode, u, idx_out, out, ws, st);
    return p.split2 ? launch_two_launch_e<E>(p, kv, q, scale_log2, mode, u, idx_out, out, ws, st)
                    : launch_one_launch_e<E>(p, kv, q, scale_log2, mode, u, idx_out, out, ws, st);
  });
}

hipError_t launch_fused_dense(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                              void *out, char *ws, hipStream_t st) {
  return with_elem(p, [&](auto eptr) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    return launch_dense_e<E>(p, kv, q, scale_log2, out, ws, st);
  });
}

hipError_t launch_fused_flash(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                              int tile_log2, int S_tile, const float *u, int32_t *idx_out,
                              void *out, char *ws, hipStream_t st, bool rows) {
  return with_elem(p, [&](auto eptr) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    if (rows)
      return launch_row_flash_e<E>(p, kv, q, scale_log2, tile_log2, S_tile, u, idx_out, out, ws, st);
    return launch_flash_e<E>(p, kv, q, scale_log2, tile_log2, S_tile, u, idx_out, out, ws, st);
  });
}

hipError_t launch_fused_bernoulli(const Plan &p, const KvView &kv, const KtView &kt,
                                 const void *q, float scale_log2, int Bd, int mode,
                                 const float *u_q, const float *u, int32_t *idx_out,
                                 uint8_t *mask_out, void *out, char *ws, hipStream_t st) {
  return with_elem(p, [&](auto eptr) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    if constexpr (sizeof(E) == 1) {
      return hipErrorInvalidValue;  // the API accepts no FP8 cache here
    } else {
      return launch_bernoulli_e<E>(p, kv, kt, q, scale_log2, Bd, mode, u_q, u, idx_out, mask_out,
                                   out, ws, st);
    }
  });
}

}  // namespace santa
