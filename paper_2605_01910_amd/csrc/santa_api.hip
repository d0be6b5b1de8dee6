// santa_api.hip -- C ABI of libsanta (declared in include/santa.h): argument
// validation, launch plan, workspace carve-up and kernel dispatch.  Nothing
// here allocates device memory or synchronises.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <mutex>
#include <string>

#include "santa.h"
#include "santa_kernels.h"
#include "santa_plan.h"

namespace {

thread_local std::string g_last_error;
thread_local santa::CallTimer g_timer;

// Consumes the pending call timer when a decode entry point returns.
struct TimerScope {
  ~TimerScope() { g_timer = santa::CallTimer{}; }
};

santa_status_t fail(santa_status_t s, const std::string &msg) {
  g_last_error = msg;
  return s;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

int ilog2(int64_t x) {
  int r = 0;
  while ((int64_t(1) << (r + 1)) <= x) ++r;
  return r;
}

// Split length: enough workgroups to cover the chip several times over (256 CUs),
// at most kSplitMax keys (the LDS tile), at least 256.
int choose_split(int64_t rows, int64_t n_k) {
  const int64_t target_wg = 2048;
  int64_t ls = (n_k * rows) / target_wg;
  int p = 256;
  while (p < santa::kSplitMax && p * 2 <= ls) p *= 2;
  return p;
}

// The calling thread's launch options (santa_set_options).  They select a
// launch path for tuning and for tests of every path; a workspace must be
// sized under the options of the calls that use it.
thread_local santa_options_t g_opts{SANTA_PATH_AUTO, 0};

// Splits per row of the fused path: enough that the whole batch of rows fills
// about `target` workgroups, at least ceil(n_k / kSplitMax).  Sampled steps
// with budgets up to S = 1024 take 256 (one per CU): at batch 1 and 32k keys
// the stratified S = 256 step runs in 27.5 us against 28.3 us with 512,
// systematic S = 512 in 27.7 against 29.1 us, S = 1024 in 29.4 against
// 29.7 us, the i.i.d. S = 256 step in 29.4 against 29.8 us.  Larger budgets
// put more claims in each split and take 512 (systematic S = 2048: 32.7 us
// against 34.2 us), and so do the dense and flash steps (level either way).
int fused_splits(int64_t rows_kv, int64_t n_k, int64_t target) {
  const int tmin = (int)((n_k + santa::kSplitMax - 1) / santa::kSplitMax);
  int fill = 128;
  while (fill > 1 && (int64_t)fill * rows_kv > target) fill >>= 1;
  int T = std::max(tmin, fill);
  if (g_opts.splits > 0) T = std::max(tmin, (int)g_opts.splits);
  return T;
}

santa_status_t check_shape(const santa_shape_t *sh) {
  if (!sh) return fail(SANTA_ERR_INVALID_ARG, "shape is NULL");
  if (sh->batch < 1 || sh->num_q_heads < 1 || sh->num_kv_heads < 1)
    return fail(SANTA_ERR_INVALID_ARG, "batch and head counts must be >= 1");
  if (sh->num_q_heads % sh->num_kv_heads)
    return fail(SANTA_ERR_INVALID_ARG, "num_q_heads must be a multiple of num_kv_heads");
  const int G = sh->num_q_heads / sh->num_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(SANTA_ERR_UNSUPPORTED, "GQA group size must be 1, 2, 4 or 8");
  if (sh->head_dim != santa::kHeadDim) return fail(SANTA_ERR_UNSUPPORTED, "head_dim must be 128");
  if (sh->dtype != SANTA_BF16 && sh->dtype != SANTA_F32)
    return fail(SANTA_ERR_INVALID_ARG, "dtype must be SANTA_BF16 or SANTA_F32");
  return SANTA_OK;
}

santa_status_t check_kv(const santa_kv_t *kv, const santa_shape_t *sh, bool need_k) {
  if (!kv) return fail(SANTA_ERR_INVALID_ARG, "kv is NULL");
  if ((need_k && !kv->k) || !kv->v) return fail(SANTA_ERR_INVALID_ARG, "kv->k or kv->v is NULL");
  if (kv->n_k < 1) return fail(SANTA_ERR_INVALID_ARG, "n_k must be >= 1");
  if (kv->kv_dtype != SANTA_KV_AS_Q && kv->kv_dtype != SANTA_KV_FP8_E4M3)
    return fail(SANTA_ERR_INVALID_ARG, "kv_dtype must be SANTA_KV_AS_Q or SANTA_KV_FP8_E4M3");
  const bool fp8 = kv->kv_dtype == SANTA_KV_FP8_E4M3;
  if (fp8) {
    if (sh->dtype != SANTA_BF16)
      return fail(SANTA_ERR_UNSUPPORTED, "an FP8 cache needs bfloat16 queries (shape->dtype)");
    if (!kv->k_scale || !kv->v_scale)
      return fail(SANTA_ERR_INVALID_ARG, "an FP8 cache needs k_scale and v_scale");
    if (kv->k_new || kv->v_new)
      return fail(SANTA_ERR_UNSUPPORTED, "the fused append is not available with an FP8 cache");
    if (g_opts.path == SANTA_PATH_MULTI)
      return fail(SANTA_ERR_UNSUPPORTED, "an FP8 cache needs the fused launch layout");
  }
  const int64_t esz = fp8 ? 1 : sh->dtype == SANTA_BF16 ? 2 : 4;
  const int64_t a = 16 / esz;  // elements per 16 bytes
  if (kv->stride_b < 0 || kv->stride_n < 0 || kv->stride_h < 0)
    return fail(SANTA_ERR_INVALID_ARG, "strides must be non-negative");
  if (kv->stride_b % a || kv->stride_n % a || kv->stride_h % a)
    return fail(SANTA_ERR_UNSUPPORTED, "strides must keep every row 16-byte aligned");
  // a lane's byte offset inside a 16-row batch of keys is 32 bits
  if ((15 * kv->stride_n + santa::kHeadDim) * esz >= (int64_t(1) << 31))
    return fail(SANTA_ERR_UNSUPPORTED, "stride_n too large");
  if ((need_k && (reinterpret_cast<uintptr_t>(kv->k) & 15)) ||
      (reinterpret_cast<uintptr_t>(kv->v) & 15))
    return fail(SANTA_ERR_UNSUPPORTED, "k and v must be 16-byte aligned");
  if (!kv->k_new != !kv->v_new) return fail(SANTA_ERR_INVALID_ARG, "k_new and v_new go together");
  if ((reinterpret_cast<uintptr_t>(kv->k_new) & 15) || (reinterpret_cast<uintptr_t>(kv->v_new) & 15))
    return fail(SANTA_ERR_UNSUPPORTED, "k_new and v_new must be 16-byte aligned");
  if (kv->block_table) {
    if (!is_pow2(kv->page_size)) return fail(SANTA_ERR_UNSUPPORTED, "page_size must be a power of two");
    if (kv->max_pages < 1) return fail(SANTA_ERR_INVALID_ARG, "max_pages must be >= 1");
    if ((int64_t)kv->max_pages * kv->page_size < kv->n_k)
      return fail(SANTA_ERR_INVALID_ARG, "max_pages * page_size < n_k");
  }
  return SANTA_OK;
}

// The flash step takes the scheduled kernel (k_row_flash: no barrier before
// the value stage, one arrival per split) under the automatic and scheduled
// paths for G <= 4 and at most kRowTMax splits per row; k_fused_dense's flash
// mode otherwise.
static bool flash_rows(const santa::Plan &p) {
  return p.fused && (g_opts.path == SANTA_PATH_AUTO || g_opts.path == SANTA_PATH_SCHEDULED) &&
         p.G <= 4 && p.T <= santa::kRowTMax;
}

santa::Plan make_plan(const santa_shape_t *sh, const santa_kv_t *kv, int S, int kind) {
  santa::Plan p{};
  p.B = sh->batch;
  p.Hq = sh->num_q_heads;
  p.Hkv = sh->num_kv_heads;
  p.G = p.Hq / p.Hkv;
  p.dtype = sh->dtype;
  p.elem = kv->kv_dtype == SANTA_KV_FP8_E4M3 ? 2 : sh->dtype == SANTA_BF16 ? 0 : 1;
  p.n_k = kv->n_k;
  p.Ls = choose_split((int64_t)p.B * p.Hkv, p.n_k);
  p.T = (int)((p.n_k + p.Ls - 1) / p.Ls);
  p.S = kind == SANTA_KIND_DENSE ? 0 : S;
  p.kind = kind;
  const size_t rows = (size_t)p.B * p.Hq;
  const size_t D = santa::kHeadDim;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  // Every layout, fused or not, starts with the error flag and the fused
  // paths' counter area, at the same offsets
  // and of the same size, so that calls of any kind and shape can share one
  // workspace in any order: no layout puts data where another keeps counters.
  // The counters must start at zero (santa_workspace_init).
  p.off_err = take(santa::kErrBytes);
  p.off_sync = take((size_t)santa::kSyncRowsMax * santa::kSyncStride * 4);
  const bool fused = g_opts.path != SANTA_PATH_MULTI;
  // (kind FLASH: the scheduled flash kernel's plan, the dense layout with the
  // small budget's split count, which is never more than the dense step's)
  const bool small_budget = ((kind == SANTA_KIND_SYSTEMATIC || kind == SANTA_KIND_STRATIFIED ||
                              kind == SANTA_KIND_IID) && S <= 1024) || kind == SANTA_KIND_FLASH;
  const int Tf = fused_splits((int64_t)p.B * p.Hkv, p.n_k, small_budget ? 256 : 512);
  if (kind != SANTA_KIND_BERNOULLI && fused && Tf <= santa::kMaxSplits &&
      (int64_t)p.B * p.Hkv <= santa::kSyncRowsMax) {
    p.fused = 1;
    p.T = Tf;
    // rows use ceil(L_b / T) keys per split rounded up to 64; Ls is the longest
    p.Ls = (int)(((p.n_k + p.T - 1) / p.T + 63) & ~63);
    // only splits that hold keys (short caches: fewer than T splits of 64 keys)
    p.T = (int)((p.n_k + p.Ls - 1) / p.Ls);
    const bool sampled = kind != SANTA_KIND_DENSE && kind != SANTA_KIND_FLASH;
    const bool big = (int64_t)p.B * p.Hkv * p.T > 1024;  // workgroups beyond one resident round
    // systematic and stratified steps, and i.i.d. steps at G <= 4 whose sorted
    // thresholds fit registers or LDS (iid_rows), take the scheduled path
    // (its row offsets live in LDS, so at most kRowTMax splits per row) when
    // asked for, and by default where it measured faster than both other
    // paths: budgets up to 1024; paged caches up to 8192 workgroups and FP8
    // caches up to 2048 (beyond those the two-launch path was faster)
    const int64_t grid = (int64_t)p.B * p.Hkv * p.T;
    // i.i.d. thresholds: in registers up to 256 per head, in LDS up to 2048
    // on grids of at most kDirectPollMax workgroups
    const bool iid_rows = p.G <= 4 && (S <= 256 || (S <= 2048 && grid <= santa::kDirectPollMax));
    const bool rows_ok = (kind == SANTA_KIND_SYSTEMATIC || kind == SANTA_KIND_STRATIFIED ||
                          (kind == SANTA_KIND_IID && iid_rows)) &&
                         p.T <= santa::kRowTMax;
    const bool rows_auto = rows_ok && S <= 1024 && (!kv->block_table || grid <= 8192) &&
                           (p.elem != 2 || grid <= 2048);
    p.rows = g_opts.path == SANTA_PATH_SCHEDULED ? rows_ok
                                                 : (g_opts.path == SANTA_PATH_AUTO && rows_auto);
    // other sampled steps whose rows do not fit in one resident round of about
    // 1024 workgroups take the two-launch path
    p.split2 = sampled && !p.rows &&
               (g_opts.path == SANTA_PATH_TWO_LAUNCH ||
                ((g_opts.path == SANTA_PATH_AUTO || g_opts.path == SANTA_PATH_SCHEDULED) && big));
    if (p.split2) {
      p.npitch = ((int64_t)p.n_k + 63) & ~int64_t(63);
      p.off_stats = take(rows * p.T * 8);
      p.off_stash = take(rows * (size_t)p.npitch * 2);   // 16-bit in-block CDF
      p.off_coarse = take(rows * (size_t)(p.npitch / 32) * 4);
    } else {
      p.off_stats = take(rows * p.T * 8);
      p.off_part = take((size_t)p.B * p.Hkv * p.T * p.G * D * 4);
    }
    p.total = off;
    return p;
  }
  if (kind == SANTA_KIND_BERNOULLI && fused && Tf <= santa::kMaxSplits) {
    // Bernoulli scores from the feature-major cache, then the value stage of
    // the two-launch path (one workgroup per query head)
    p.fused = 1;
    p.split2 = 1;
    // splits of at most 512 keys by default: the feature-row stream of a
    // split is short, so more workgroups keep more of it in flight; a split
    // count set in the options applies as given (at least n_k / 1024)
    p.T = g_opts.splits > 0 ? Tf
                            : std::min(santa::kMaxSplits, std::max(Tf, (int)((p.n_k + 511) / 512)));
    p.Ls = (int)(((p.n_k + p.T - 1) / p.T + 63) & ~63);
    p.npitch = ((int64_t)p.n_k + 63) & ~int64_t(63);
    p.off_stats = take(rows * p.T * 8);
    p.off_stash = take(rows * (size_t)p.npitch * 2);
    p.off_coarse = take(rows * (size_t)(p.npitch / 32) * 4);
    p.total = off;
    return p;
  }
  p.off_stats = take(rows * p.T * 8);
  p.off_part = take((size_t)p.B * p.Hkv * p.T * p.G * D * 4);
  if (kind != SANTA_KIND_DENSE) {
    p.off_stash = take(rows * (size_t)p.T * p.Ls * 4);
    p.off_offs = take(rows * (size_t)(p.T + 1) * 4);
    p.off_alpha = take(rows * (size_t)p.T * 4);
    p.off_rowst = take(rows * 8);
    p.off_flag = take((size_t)p.B * p.Hkv * p.T * 4);
  }
  if (kind == SANTA_KIND_BERNOULLI) {
    p.off_bw = take(rows * D * 4);
    p.off_blist = take((size_t)p.B * p.Hkv * D * 4);
    p.off_bn = take((size_t)p.B * p.Hkv * 4);
  }
  p.total = off;
  return p;
}

santa_status_t check_ws(const santa::Plan &p, void *ws, size_t ws_bytes) {
  if (!ws) return fail(SANTA_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) & 255) return fail(SANTA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < p.total)
    return fail(SANTA_ERR_WORKSPACE, "workspace too small: need " + std::to_string(p.total) +
                                         " bytes, got " + std::to_string(ws_bytes));
  return SANTA_OK;
}

santa::KvView make_view(const santa_kv_t *kv) {
  santa::KvView v{};
  v.k = kv->k;
  v.v = kv->v;
  v.sb = kv->stride_b;
  v.sn = kv->stride_n;
  v.sh = kv->stride_h;
  v.ctx = kv->ctx_len;
  v.bt = kv->block_table;
  v.ps_log2 = kv->block_table ? ilog2(kv->page_size) : 0;
  v.max_pages = kv->max_pages;
  v.n_k = kv->n_k;
  v.k_new = kv->k_new;
  v.v_new = kv->v_new;
  v.ks = kv->kv_dtype == SANTA_KV_FP8_E4M3 ? kv->k_scale : nullptr;
  v.vs = kv->kv_dtype == SANTA_KV_FP8_E4M3 ? kv->v_scale : nullptr;
  return v;
}

santa_status_t hip_status(hipError_t e) {
  if (e != hipSuccess) return fail(SANTA_ERR_HIP, std::string("HIP: ") + hipGetErrorString(e));
  return SANTA_OK;
}

float log2_scale(float scale) { return scale * 1.44269504088896340736f; }

santa_status_t common_checks(const void *q, const santa_kv_t *kv, const santa_shape_t *sh,
                             float scale, void *out, bool need_k) {
  g_last_error.clear();
  santa_status_t s = check_shape(sh);
  if (s != SANTA_OK) return s;
  s = check_kv(kv, sh, need_k);
  if (s != SANTA_OK) return s;
  if (!q || !out) return fail(SANTA_ERR_INVALID_ARG, "q or out is NULL");
  if ((reinterpret_cast<uintptr_t>(q) & 15)) return fail(SANTA_ERR_UNSUPPORTED, "q must be 16-byte aligned");
  if (!std::isfinite(scale)) return fail(SANTA_ERR_INVALID_ARG, "scale must be finite");
  return SANTA_OK;
}

santa_status_t sampled(const void *q, const santa_kv_t *kv, const santa_shape_t *sh, float scale,
                       int32_t S, const float *u, int32_t *idx_out, void *out, void *ws,
                       size_t ws_bytes, void *stream, bool strat) {
  TimerScope timer_scope;
  santa_status_t s = common_checks(q, kv, sh, scale, out, true);
  if (s != SANTA_OK) return s;
  if (S < 1 || S > (1 << 24)) return fail(SANTA_ERR_INVALID_ARG, "S must be in [1, 2^24]");
  if (!u) return fail(SANTA_ERR_INVALID_ARG, "u is NULL");
  const santa::Plan p = make_plan(sh, kv, S, strat ? SANTA_KIND_STRATIFIED : SANTA_KIND_SYSTEMATIC);
  s = check_ws(p, ws, ws_bytes);
  if (s == SANTA_OK && kv->k_new && !p.fused)
    s = fail(SANTA_ERR_UNSUPPORTED, "the fused append (k_new, v_new) needs the fused path");
  if (s == SANTA_OK && kv->kv_dtype != SANTA_KV_AS_Q && !p.fused)
    s = fail(SANTA_ERR_UNSUPPORTED, "an FP8 cache needs the fused launch layout");
  if (s != SANTA_OK) return s;
  if (p.fused)
    return hip_status(santa::launch_fused_sampled(p, make_view(kv), q, log2_scale(scale),
                                                  strat ? 1 : 0, u, idx_out, out,
                                                  static_cast<char *>(ws),
                                                  static_cast<hipStream_t>(stream)));
  return hip_status(santa::launch_sampled(p, make_view(kv), q, log2_scale(scale), strat, u, idx_out,
                                          out, static_cast<char *>(ws),
                                          static_cast<hipStream_t>(stream)));
}

// Scratch of the no-allocation entry point: the workspace of its calls, one
// array per GPU in the library's own device memory (a code-object global, so
// the loader places it and nothing is allocated at call time).  In host code
// `scratch` names a host-side stand-in, never a device address: its device
// address on each GPU comes from hipGetSymbolAddress, taken once per device
// with that device current, and only that address is passed to kernels.
static __device__ __align__(256) unsigned char scratch[SANTA_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each GPU (null: not yet)

// The calling thread's current device, which must also own `stream`, and the
// device address of its scratch array (set up on the device's first call).
santa_status_t scratch_for(hipStream_t stream, void **ptr) {
  int dev = -1, sdev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return fail(SANTA_ERR_HIP, "no usable current device");
  if (stream && (hipStreamGetDevice(stream, &sdev) != hipSuccess || sdev != dev))
    return fail(SANTA_ERR_INVALID_ARG, "stream must belong to the current device");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return fail(SANTA_ERR_HIP, "hipGetSymbolAddress(scratch) failed");
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return SANTA_OK;
}

}  // namespace

santa::CallTimer &santa::call_timer() { return g_timer; }

extern "C" {

size_t santa_workspace_size(const santa_shape_t *shape, const santa_kv_t *kv, int32_t S,
                            int32_t kind) {
  if (check_shape(shape) != SANTA_OK || !kv || kv->n_k < 1) return 0;
  if (kind < SANTA_KIND_DENSE || kind > SANTA_KIND_IID) return 0;
  if (kind == SANTA_KIND_FLASH) kind = SANTA_KIND_DENSE;  // the same launch layout
  if (kind != SANTA_KIND_DENSE && (S < 1 || S > (1 << 24))) return 0;
  return make_plan(shape, kv, S, kind).total;
}

santa_status_t santa_workspace_init(void *ws, size_t ws_bytes, void *stream) {
  g_last_error.clear();
  if (!ws) return fail(SANTA_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) & 255) return fail(SANTA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  return hip_status(santa::launch_zero(ws, ws_bytes & ~size_t(15), static_cast<hipStream_t>(stream)));
}

santa_status_t santa_decode_dense(const void *q, const santa_kv_t *kv, const santa_shape_t *shape,
                                  float scale, void *out, void *ws, size_t ws_bytes,
                                  void *stream) {
  TimerScope timer_scope;
  santa_status_t s = common_checks(q, kv, shape, scale, out, true);
  if (s != SANTA_OK) return s;
  const santa::Plan p = make_plan(shape, kv, 0, SANTA_KIND_DENSE);
  s = check_ws(p, ws, ws_bytes);
  if (s == SANTA_OK && kv->k_new && !p.fused)
    s = fail(SANTA_ERR_UNSUPPORTED, "the fused append (k_new, v_new) needs the fused path");
  if (s == SANTA_OK && kv->kv_dtype != SANTA_KV_AS_Q && !p.fused)
    s = fail(SANTA_ERR_UNSUPPORTED, "an FP8 cache needs the fused launch layout");
  if (s != SANTA_OK) return s;
  if (p.fused)
    return hip_status(santa::launch_fused_dense(p, make_view(kv), q, log2_scale(scale), out,
                                                static_cast<char *>(ws),
                                                static_cast<hipStream_t>(stream)));
  return hip_status(santa::launch_dense(p, make_view(kv), q, log2_scale(scale), out,
                                        static_cast<char *>(ws), static_cast<hipStream_t>(stream)));
}

santa_status_t santa_decode_systematic(const void *q, const santa_kv_t *kv,
                                       const santa_shape_t *shape, float scale, int32_t S,
                                       const float *u, int32_t *idx_out, void *out, void *ws,
                                       size_t ws_bytes, void *stream) {
  return sampled(q, kv, shape, scale, S, u, idx_out, out, ws, ws_bytes, stream, false);
}

santa_status_t santa_decode_stratified(const void *q, const santa_kv_t *kv,
                                       const santa_shape_t *shape, float scale, int32_t S,
                                       const float *u, int32_t *idx_out, void *out, void *ws,
                                       size_t ws_bytes, void *stream) {
  return sampled(q, kv, shape, scale, S, u, idx_out, out, ws, ws_bytes, stream, true);
}

santa_status_t santa_decode_stratified_noalloc(const void *q, const santa_kv_t *kv,
                                               const santa_shape_t *shape, float scale, int32_t S,
                                               const float *u, int32_t *idx_out, void *out,
                                               void *stream) {
  TimerScope timer_scope;
  santa_status_t s = common_checks(q, kv, shape, scale, out, true);
  if (s != SANTA_OK) return s;
  if (S < 1 || S > (1 << 24)) return fail(SANTA_ERR_INVALID_ARG, "S must be in [1, 2^24]");
  if (!u) return fail(SANTA_ERR_INVALID_ARG, "u is NULL");
  const santa::Plan p = make_plan(shape, kv, S, SANTA_KIND_STRATIFIED);
  if (p.total > SANTA_STATIC_SCRATCH_BYTES)
    return fail(SANTA_ERR_WORKSPACE, "the call needs more workspace than the static scratch array "
                                     "holds (SANTA_STATIC_SCRATCH_BYTES)");
  if (!p.fused) return fail(SANTA_ERR_UNSUPPORTED, "the no-allocation call needs the fused launch layout");
  const hipStream_t st = static_cast<hipStream_t>(stream);
  void *ws = nullptr;
  s = scratch_for(st, &ws);
  if (s != SANTA_OK) return s;
  // The array keeps the previous call's contents.  Clear what must start at
  // zero: the wait flag and the row counters this call uses (a fill kernel,
  // not a memset, so that the call can be captured in a graph).  Everything
  // else the call reads it writes first.
  const size_t head = p.off_sync + (size_t)p.B * p.Hkv * santa::kSyncStride * 4;
  hipError_t e = santa::launch_zero(ws, head, st);
  if (e != hipSuccess) return hip_status(e);
  return hip_status(santa::launch_fused_sampled(p, make_view(kv), q, log2_scale(scale), 1, u,
                                                idx_out, out, static_cast<char *>(ws), st));
}

santa_status_t santa_decode_bernoulli_qk(const void *q, const santa_kt_t *kt,
                                         const santa_kv_t *kv, const santa_shape_t *shape,
                                         float scale, int32_t B_draws, int32_t mode,
                                         const float *u_q, int32_t S, const float *u,
                                         int32_t *idx_out, uint8_t *feat_mask_out, void *out,
                                         void *ws, size_t ws_bytes, void *stream) {
  TimerScope timer_scope;
  santa_status_t s = common_checks(q, kv, shape, scale, out, false);
  if (s != SANTA_OK) return s;
  if (kv->block_table) return fail(SANTA_ERR_UNSUPPORTED, "Bernoulli scores need a contiguous cache");
  if (kv->kv_dtype != SANTA_KV_AS_Q)
    return fail(SANTA_ERR_UNSUPPORTED, "Bernoulli scores need a cache in the query's dtype");
  if (!kt || !kt->k_t) return fail(SANTA_ERR_INVALID_ARG, "kt or kt->k_t is NULL");
  const int64_t a = shape->dtype == SANTA_BF16 ? 8 : 4;
  if (kt->stride_b < 0 || kt->stride_h < 0 || kt->stride_d < kv->n_k)
    return fail(SANTA_ERR_INVALID_ARG, "kt strides must be >= 0 and stride_d >= n_k");
  if (kt->stride_b % a || kt->stride_h % a || kt->stride_d % a ||
      (reinterpret_cast<uintptr_t>(kt->k_t) & 15))
    return fail(SANTA_ERR_UNSUPPORTED, "kt rows must be 16-byte aligned");
  if (mode != 0 && mode != 1) return fail(SANTA_ERR_INVALID_ARG, "mode must be 0 or 1");
  if (B_draws < 1 || B_draws > 64) return fail(SANTA_ERR_INVALID_ARG, "B_draws must be in [1, 64]");
  if (!u_q || !u) return fail(SANTA_ERR_INVALID_ARG, "u_q or u is NULL");
  if (S < 1 || S > (1 << 24)) return fail(SANTA_ERR_INVALID_ARG, "S must be in [1, 2^24]");
  const santa::Plan p = make_plan(shape, kv, S, SANTA_KIND_BERNOULLI);
  s = check_ws(p, ws, ws_bytes);
  if (s == SANTA_OK && kv->k_new)
    s = fail(SANTA_ERR_UNSUPPORTED, "the fused append (k_new, v_new) is not available with Bernoulli scores");
  if (s != SANTA_OK) return s;
  santa::KtView ktv{kt->k_t, kt->stride_b, kt->stride_h, kt->stride_d};
  if (p.fused)
    return hip_status(santa::launch_fused_bernoulli(
        p, make_view(kv), ktv, q, log2_scale(scale), B_draws, mode, u_q, u, idx_out,
        feat_mask_out, out, static_cast<char *>(ws), static_cast<hipStream_t>(stream)));
  return hip_status(santa::launch_bernoulli(p, make_view(kv), ktv, q, log2_scale(scale), B_draws,
                                            mode, u_q, u, idx_out, feat_mask_out, out,
                                            static_cast<char *>(ws),
                                            static_cast<hipStream_t>(stream)));
}

santa_status_t santa_decode_iid(const void *q, const santa_kv_t *kv, const santa_shape_t *shape,
                                float scale, int32_t S, const float *u, int32_t *idx_out,
                                void *out, void *ws, size_t ws_bytes, void *stream) {
  TimerScope timer_scope;
  santa_status_t s = common_checks(q, kv, shape, scale, out, true);
  if (s != SANTA_OK) return s;
  const int G = shape->num_q_heads / shape->num_kv_heads;
  if (S < 1 || (int64_t)G * (2 * S + 1) > 4096)
    return fail(SANTA_ERR_INVALID_ARG, "S must satisfy 1 <= S and G*(2S+1) <= 4096 for the i.i.d. step");
  if (!u) return fail(SANTA_ERR_INVALID_ARG, "u is NULL");
  const santa::Plan p = make_plan(shape, kv, S, SANTA_KIND_IID);
  s = check_ws(p, ws, ws_bytes);
  if (s == SANTA_OK && kv->k_new && !p.fused)
    s = fail(SANTA_ERR_UNSUPPORTED, "the fused append (k_new, v_new) needs the fused path");
  if (s == SANTA_OK && kv->kv_dtype != SANTA_KV_AS_Q && !p.fused)
    s = fail(SANTA_ERR_UNSUPPORTED, "an FP8 cache needs the fused launch layout");
  if (s != SANTA_OK) return s;
  if (!p.fused) return fail(SANTA_ERR_UNSUPPORTED, "the i.i.d. step needs the fused launch layout");
  return hip_status(santa::launch_fused_sampled(p, make_view(kv), q, log2_scale(scale), 2, u,
                                                idx_out, out, static_cast<char *>(ws),
                                                static_cast<hipStream_t>(stream)));
}

santa_status_t santa_decode_flash(const void *q, const santa_kv_t *kv, const santa_shape_t *shape,
                                  float scale, int32_t tile, int32_t S_tile, const float *u,
                                  int32_t *idx_out, void *out, void *ws, size_t ws_bytes,
                                  void *stream) {
  TimerScope timer_scope;
  santa_status_t s = common_checks(q, kv, shape, scale, out, true);
  if (s != SANTA_OK) return s;
  if (!is_pow2(tile) || tile < 16 || tile > santa::kSplitMax)
    return fail(SANTA_ERR_INVALID_ARG, "tile must be a power of two in [16, 1024]");
  if (S_tile < 1 || S_tile > 4096) return fail(SANTA_ERR_INVALID_ARG, "S_tile must be in [1, 4096]");
  if (!u) return fail(SANTA_ERR_INVALID_ARG, "u is NULL");
  santa::Plan p = make_plan(shape, kv, 0, SANTA_KIND_DENSE);
  const bool rows = flash_rows(p);
  if (rows) p = make_plan(shape, kv, 0, SANTA_KIND_FLASH);
  s = check_ws(p, ws, ws_bytes);
  if (s == SANTA_OK && kv->k_new && !p.fused)
    s = fail(SANTA_ERR_UNSUPPORTED, "the fused append (k_new, v_new) needs the fused path");
  if (s == SANTA_OK && kv->kv_dtype != SANTA_KV_AS_Q && !p.fused)
    s = fail(SANTA_ERR_UNSUPPORTED, "an FP8 cache needs the fused launch layout");
  if (s != SANTA_OK) return s;
  if (!p.fused) return fail(SANTA_ERR_UNSUPPORTED, "the flash step needs the fused launch layout");
  return hip_status(santa::launch_fused_flash(p, make_view(kv), q, log2_scale(scale), ilog2(tile),
                                              S_tile, u, idx_out, out, static_cast<char *>(ws),
                                              static_cast<hipStream_t>(stream), rows));
}

santa_status_t santa_stream_read(const void *buf, size_t bytes, uint32_t *sink, void *stream) {
  TimerScope timer_scope;
  g_last_error.clear();
  if (!buf || !sink) return fail(SANTA_ERR_INVALID_ARG, "buf or sink is NULL");
  if (bytes == 0 || bytes % 16) return fail(SANTA_ERR_INVALID_ARG, "bytes must be a positive multiple of 16");
  if (bytes / 16 / SANTA_STREAM_READ_GROUPS >= (size_t(1) << 30))
    return fail(SANTA_ERR_INVALID_ARG, "bytes too large");
  if (reinterpret_cast<uintptr_t>(buf) & 15) return fail(SANTA_ERR_INVALID_ARG, "buf must be 16-byte aligned");
  return hip_status(santa::launch_stream_read(buf, bytes, sink, SANTA_STREAM_READ_GROUPS,
                                              static_cast<hipStream_t>(stream)));
}

santa_status_t santa_set_options(const santa_options_t *opts) {
  g_last_error.clear();
  if (!opts) {
    g_opts = santa_options_t{SANTA_PATH_AUTO, 0};
    return SANTA_OK;
  }
  if (opts->path < SANTA_PATH_AUTO || opts->path > SANTA_PATH_SCHEDULED)
    return fail(SANTA_ERR_INVALID_ARG, "path must be a santa_path_t");
  if (opts->splits < 0 || opts->splits > santa::kMaxSplits)
    return fail(SANTA_ERR_INVALID_ARG, "splits must be in [0, 256]");
  g_opts = *opts;
  return SANTA_OK;
}

santa_status_t santa_get_options(santa_options_t *opts) {
  g_last_error.clear();
  if (!opts) return fail(SANTA_ERR_INVALID_ARG, "opts is NULL");
  *opts = g_opts;
  return SANTA_OK;
}

santa_status_t santa_plan_info(const santa_shape_t *shape, const santa_kv_t *kv, int32_t S,
                               int32_t kind, santa_plan_info_t *info) {
  g_last_error.clear();
  if (!info) return fail(SANTA_ERR_INVALID_ARG, "info is NULL");
  santa_status_t s = check_shape(shape);
  if (s != SANTA_OK) return s;
  if (!kv || kv->n_k < 1) return fail(SANTA_ERR_INVALID_ARG, "kv is NULL or n_k < 1");
  if (kind < SANTA_KIND_DENSE || kind > SANTA_KIND_IID) return fail(SANTA_ERR_INVALID_ARG, "bad kind");
  const int32_t plan_kind = kind == SANTA_KIND_FLASH ? SANTA_KIND_DENSE : kind;
  if (plan_kind != SANTA_KIND_DENSE && (S < 1 || S > (1 << 24)))
    return fail(SANTA_ERR_INVALID_ARG, "S must be in [1, 2^24]");
  santa::Plan p = make_plan(shape, kv, S, plan_kind);
  const bool frows = kind == SANTA_KIND_FLASH && flash_rows(p);
  if (frows) p = make_plan(shape, kv, S, SANTA_KIND_FLASH);
  info->splits = p.T;
  info->split_len = p.Ls;
  info->workspace = p.total;
  if (!p.fused) {
    info->path = SANTA_PATH_MULTI;
    info->kernels = "multi-kernel variant (k_score_cdf / k_dense_split / k_bern_score, k_offsets, "
                    "k_sample, k_merge_*)";
  } else if (kind == SANTA_KIND_BERNOULLI) {
    info->path = SANTA_PATH_TWO_LAUNCH;
    info->kernels = "k_bern_stream + k_value_heads";
  } else if (frows) {
    info->path = SANTA_PATH_SCHEDULED;
    info->kernels = "k_row_flash";
  } else if (kind == SANTA_KIND_DENSE || kind == SANTA_KIND_FLASH) {
    info->path = SANTA_PATH_ONE_LAUNCH;
    info->kernels = kind == SANTA_KIND_DENSE ? "k_fused_dense" : "k_fused_dense (flash mode)";
  } else if (p.rows) {
    info->path = SANTA_PATH_SCHEDULED;
    info->kernels = "k_row_sampled";
  } else if (p.split2) {
    info->path = SANTA_PATH_TWO_LAUNCH;
    info->kernels = "k_stream_cdf + k_value_heads";
  } else {
    info->path = SANTA_PATH_ONE_LAUNCH;
    info->kernels = "k_fused_sampled";
  }
  return SANTA_OK;
}

santa_status_t santa_time_next_call(void *start_event, void *stop_event) {
  g_last_error.clear();
  if ((start_event == nullptr) != (stop_event == nullptr))
    return fail(SANTA_ERR_INVALID_ARG, "start_event and stop_event must both be set or both NULL");
  g_timer.start = static_cast<hipEvent_t>(start_event);
  g_timer.stop = static_cast<hipEvent_t>(stop_event);
  return SANTA_OK;
}

const char *santa_status_string(santa_status_t status) {
  switch (status) {
    case SANTA_OK: return "SANTA_OK";
    case SANTA_ERR_INVALID_ARG: return "SANTA_ERR_INVALID_ARG";
    case SANTA_ERR_UNSUPPORTED: return "SANTA_ERR_UNSUPPORTED";
    case SANTA_ERR_WORKSPACE: return "SANTA_ERR_WORKSPACE";
    case SANTA_ERR_HIP: return "SANTA_ERR_HIP";
  }
  return "SANTA_ERR_UNKNOWN";
}

const char *santa_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
