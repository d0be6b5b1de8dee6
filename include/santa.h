/*
 * santa.h -- C ABI of libsanta: one decode step of SANTA / S2ANTA attention on
 * an AMD Instinct MI355X (gfx950).
 *
 * Method: "Stochastic Sparse Attention for Memory-Bound Inference" (arXiv
 * 2605.01910).  A decode step computes, for every query row (batch b, query
 * head h) with context length L = ctx_len[b] and KV head k = h / (Hq / Hkv):
 *
 *   scores   s_j = scale * <q_h, K_{b,j,k}>,  j < L             (Sec. 2, SDPA equation)
 *   softmax  p = softmax(s)                                      (Sec. 2, SDPA equation)
 *   dense    out = sum_j p_j V_{b,j,k}                           (Sec. 2, SDPA equation)
 *   sampled  out = (1/S) sum_m V_{b,J_m,k},  J_m = F^{-1}(T_m)   (Sec. 2, Eq. "stochastic-add-only-attn";
 *            F = CDF of p; T_m systematic or stratified          Sec. 2.1, "Construction")
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every pointer argument except `stream` and the `shape`/`kv`/`kt` structs is
 *   a DEVICE pointer owned by the caller.  The library never allocates, frees
 *   or synchronises; all kernels are enqueued on `stream` (a hipStream_t,
 *   NULL = the null stream) and the call returns before they finish.
 * - Element type: `shape->dtype` (SANTA_BF16 or SANTA_F32) is the type of q, K,
 *   V and out.  Accumulation is float32.
 * - q is [batch, num_q_heads, head_dim] contiguous; out is the same shape and
 *   type; idx_out (optional, NULL to skip) is int32 [batch, num_q_heads, S].
 * - head_dim must be 128; num_q_heads / num_kv_heads must be 1, 2, 4 or 8.
 * - Errors: arguments are validated on the host before any launch; on error
 *   nothing is enqueued and a status code is returned (santa_last_error() gives
 *   a message).  A launch failure returns SANTA_ERR_HIP.  No C++ exception
 *   crosses this interface.
 * - Not checked on the device (preconditions): u values in [0, 1),
 *   0 <= ctx_len[b] <= n_k, block-table entries naming valid pages.  A row with
 *   ctx_len 0 yields a zero output and idx -1.
 * - Workspace: `ws` must be at least santa_workspace_size(...) bytes, 256-byte
 *   aligned, and initialised once by santa_workspace_init() (or zero-filled)
 *   before its first use.  Every call leaves it ready for the next call, of
 *   any kind and shape, provided the workspace is large enough for that call.
 *   Calls that share one workspace must be ordered (same stream or
 *   synchronised).
 * - Bounded waits: the single-launch paths wait on other workgroups of the
 *   same launch with a spin limit.  A wait that gives up sets the int32 at
 *   byte 0 of the workspace to nonzero; that call's outputs are then not
 *   valid and the workspace needs santa_workspace_init() again.  The library
 *   never reads the flag back (it does not synchronise); callers may.
 * - Per-thread state: the last error message, a pending call timer
 *   (santa_time_next_call) and the launch options (santa_set_options).
 *   Nothing else persists between calls outside the caller's workspace.
 */
#ifndef SANTA_H
#define SANTA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SANTA_OK = 0,
  SANTA_ERR_INVALID_ARG = 1, /* null pointer, bad size, inconsistent shape   */
  SANTA_ERR_UNSUPPORTED = 2, /* valid but not implemented (head_dim, G, ...) */
  SANTA_ERR_WORKSPACE = 3,   /* workspace missing, too small or misaligned   */
  SANTA_ERR_HIP = 4          /* a HIP runtime call or kernel launch failed    */
} santa_status_t;

typedef enum { SANTA_BF16 = 0, SANTA_F32 = 1 } santa_dtype_t;

typedef enum {
  SANTA_KIND_DENSE = 0,
  SANTA_KIND_SYSTEMATIC = 1,
  SANTA_KIND_STRATIFIED = 2,
  SANTA_KIND_BERNOULLI = 3,
  SANTA_KIND_FLASH = 4,
  SANTA_KIND_IID = 5
} santa_kind_t;

/* Problem shape.  dtype is a santa_dtype_t. */
typedef struct {
  int32_t batch;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t dtype;
} santa_shape_t;

/* KV cache descriptor (device pointers, caller-owned).  The feature dimension
 * is always contiguous (stride 1); strides are in ELEMENTS and must keep every
 * 128-feature row 16-byte aligned.
 *
 * Contiguous cache (block_table == NULL): element (b, j, k, i) of K or V is at
 *   base + b*stride_b + j*stride_n + k*stride_h + i,
 * so the sequence-major layout [B, n, Hkv, d] of the paper's microbenchmark and
 * the head-major layout [B, Hkv, n, d] are both expressible.
 *
 * Paged cache (block_table != NULL, int32 [batch, max_pages]): token j of
 * sequence b lives in page P = block_table[b*max_pages + j/page_size]; its
 * element (k, i) is at
 *   base + P*stride_b + (j % page_size)*stride_n + k*stride_h + i,
 * e.g. stride_b = Hkv*page_size*d, stride_h = page_size*d, stride_n = d for a
 * [pages, Hkv, page_size, d] pool.  page_size must be a power of two.
 *
 * ctx_len: int32 [batch] per-sequence lengths, or NULL for "every sequence has
 * n_k keys".  n_k (host value) is the maximum length; it sizes the launch. */
typedef struct {
  const void *k;
  const void *v;
  int64_t stride_b, stride_n, stride_h;
  const int32_t *ctx_len;
  const int32_t *block_table;
  int32_t page_size;
  int32_t max_pages;
  int32_t n_k;
  /* Fused current-token append (nullable, both or neither; 16-byte aligned,
   * [batch, num_kv_heads, head_dim] in the cache's dtype).  A decode step
   * first stores the new token's key and value in the cache, then attends
   * over it; FlashAttention-2's decode call fuses that store, the paper's
   * kernels take a cache that already holds the token (App. Decode-Step
   * Kernel Microbenchmark Details, note on KV-cache appends).  When set, the
   * call writes k_new / v_new into row ctx_len[b] - 1 (n_k - 1 without
   * ctx_len) of every (b, kv head), through the block table for paged
   * caches, inside the attention launch, and attends over the cache with
   * those rows: the cache memory must be writable and ctx_len[b] >= 1.
   * Supported by the dense, flash and sampled calls on their fused paths;
   * the Bernoulli call and the multi-kernel path return
   * SANTA_ERR_UNSUPPORTED. */
  const void *k_new;
  const void *v_new;
  /* Element type of K and V (a santa_kv_dtype_t).  SANTA_KV_AS_Q (0, the
   * default): shape->dtype.  SANTA_KV_FP8_E4M3 (1): one byte per element, an
   * OCP FP8 E4M3 code (1 sign bit, 4 exponent bits with bias 7, 3 mantissa
   * bits; exponent field 0 encodes the subnormals m/8 * 2^-6; S.1111.111 is
   * NaN; no infinities), scaled per (batch, KV head): element (b, j, k, i) of
   * K is k_scale[b*num_kv_heads + k] * e4m3(code), and likewise for V with
   * v_scale (device float32 arrays [batch, num_kv_heads]).  Quantising the
   * cache is complementary to SANTA (Sec. 1; Related Work on KV-cache
   * compression): keys and values are read at one byte each.  Needs
   * shape->dtype == SANTA_BF16 (q and out stay bfloat16); strides are in
   * elements (= bytes) and must keep rows 16-byte aligned.  Supported by the
   * dense, flash, systematic, stratified and i.i.d. calls on their fused
   * paths; the Bernoulli call, the multi-kernel path and the fused append
   * return SANTA_ERR_UNSUPPORTED. */
  int32_t kv_dtype;
  const float *k_scale;
  const float *v_scale;
} santa_kv_t;

typedef enum { SANTA_KV_AS_Q = 0, SANTA_KV_FP8_E4M3 = 1 } santa_kv_dtype_t;

/* Feature-major key cache for the Bernoulli score stage: element (b, k, i, j)
 * (feature i of key j) at k_t + b*stride_b + k*stride_h + i*stride_d + j; keys
 * are contiguous so that skipping a feature skips a contiguous row of K^T
 * (Sec. 5: features whose query sample is zero need not be read). */
typedef struct {
  const void *k_t;
  int64_t stride_b, stride_h, stride_d;
} santa_kt_t;

/* Bytes of workspace the given call needs (kind: santa_kind_t; S ignored for
 * SANTA_KIND_DENSE and SANTA_KIND_FLASH).  Returns 0 if the arguments are invalid. */
size_t santa_workspace_size(const santa_shape_t *shape, const santa_kv_t *kv, int32_t S,
                            int32_t kind);

/* Prepare a workspace for first use (zero-fills it on `stream`). */
santa_status_t santa_workspace_init(void *ws, size_t ws_bytes, void *stream);

/* Exact decode attention (Sec. 2, SDPA equation): out = softmax(scale q K^T) V,
 * computed split-K with a max/sum-exp merge.  The like-for-like dense baseline
 * of the sampled entry points below. */
santa_status_t santa_decode_dense(const void *q, const santa_kv_t *kv, const santa_shape_t *shape,
                                  float scale, void *out, void *ws, size_t ws_bytes,
                                  void *stream);

/* S2ANTA-sys (Sec. 2.1, "Construction", systematic): one uniform u per row
 * (u: float32 [batch, num_q_heads], in [0,1)); thresholds T_m = (m + u)/S for
 * m = 0..S-1; J_m = F^{-1}(T_m) is the key whose CDF interval [F(j-1), F(j))
 * contains T_m (App. A, "Unbiasedness of S2ANTA"); out = (1/S) sum_m V_{J_m}.
 * Samples are assigned to KV splits by the exact global CDF, so the estimator
 * is the paper's systematic one for any split size.  1 <= S <= 2^24. */
santa_status_t santa_decode_systematic(const void *q, const santa_kv_t *kv,
                                       const santa_shape_t *shape, float scale, int32_t S,
                                       const float *u, int32_t *idx_out, void *out, void *ws,
                                       size_t ws_bytes, void *stream);

/* S2ANTA-strat (Sec. 2.1, "Construction", independent stratified): S uniforms
 * per row (u: float32 [batch, num_q_heads, S]); T_m = (m + u_m)/S lies in
 * stratum [m/S, (m+1)/S); otherwise as santa_decode_systematic. */
santa_status_t santa_decode_stratified(const void *q, const santa_kv_t *kv,
                                       const santa_shape_t *shape, float scale, int32_t S,
                                       const float *u, int32_t *idx_out, void *out, void *ws,
                                       size_t ws_bytes, void *stream);

/* SANTA with i.i.d. draws (Sec. 2, Eq. "stochastic-add-only-attn": S indices
 * drawn independently from the attention distribution, with replacement).
 * The draws are the inverse CDF (as above) of S sorted independent uniforms,
 * built without a sort from S + 1 uniforms per row (u: float32 [batch,
 * num_q_heads, S + 1], in [0,1)): E_i = -ln(1 - u_i), T_m = C_m / C_S with
 * C_m = sum_{i<=m} E_i (the normalised partial sums of S + 1 unit
 * exponentials are the order statistics of S uniforms); out = (1/S)
 * sum_m V_{J_m}.  Requires G*(2S + 1) <= 4096 (G = num_q_heads /
 * num_kv_heads; S <= 511 at G = 4); workspace as SANTA_KIND_IID.  Needs the
 * fused launch layout: returns SANTA_ERR_UNSUPPORTED under SANTA_PATH_MULTI
 * and when batch * num_kv_heads exceeds 4096. */
santa_status_t santa_decode_iid(const void *q, const santa_kv_t *kv, const santa_shape_t *shape,
                                float scale, int32_t S, const float *u, int32_t *idx_out,
                                void *out, void *ws, size_t ws_bytes, void *stream);

/* No-allocation form of santa_decode_stratified, for callers that cannot
 * allocate device memory at call time: code under HIP graph capture, serving
 * loops and harnesses that forbid it.  Same arguments, computation and
 * outputs as santa_decode_stratified, without the workspace: the call uses a
 * scratch array of SANTA_STATIC_SCRATCH_BYTES (64 MiB) in the library's own
 * device memory, one per GPU, placed when the library's code is loaded on that
 * GPU and held until the process ends.  The first call on a device looks up
 * the array's address there.  Every call first clears the part of the array
 * that must start at zero (a fill kernel on `stream`), so it does not depend
 * on what earlier calls left; calls on one GPU share the array, so calls that
 * overlap in time on one GPU (on different streams, or from different
 * threads without ordering) race and give invalid outputs.  `stream` must
 * belong to the calling thread's current device.  Errors: as
 * santa_decode_stratified; SANTA_ERR_WORKSPACE when the call needs more than
 * SANTA_STATIC_SCRATCH_BYTES of workspace (santa_workspace_size with
 * SANTA_KIND_STRATIFIED gives the need); SANTA_ERR_UNSUPPORTED under
 * SANTA_PATH_MULTI.  It never calls hipMalloc or hipFree. */
#define SANTA_STATIC_SCRATCH_BYTES (64u << 20)
santa_status_t santa_decode_stratified_noalloc(const void *q, const santa_kv_t *kv,
                                               const santa_shape_t *shape, float scale, int32_t S,
                                               const float *u, int32_t *idx_out, void *out,
                                               void *stream);

/* Bernoulli qK^T score sampling (Sec. 5, Eq. "qk_estimator"; App. C) followed
 * by the systematic value stage.
 *   mode 0, per-head ternary query: norm = max_i |q_i|, pi_i = |q_i|/norm,
 *           w_i = (norm/B) * sign(q_i) * c_i;
 *   mode 1, mean group query (Sec. 5, Eq. "mean_group_query"; App. C, GQA):
 *           m_i = mean over the group of |q_{g,i}|, norm = max_i m_i,
 *           pi_i = m_i/norm, w_{g,i} = (norm/B) c_i q_{g,i} / m_i (0 if m_i = 0);
 *   with B = B_draws and the stratified count c_i = #{n < B : (n + u_i)/B < pi_i}
 *   (for B = 1 this is one Bernoulli(pi_i) draw).  The decision is taken in
 *   float32.  Scores s_j = scale * <w, k_j> read only the features in the
 *   union over the GQA group of nonzero weights, from the feature-major cache kt.
 * u_q: float32 [batch, num_q_heads, head_dim] (mode 0) or
 *      [batch, num_kv_heads, head_dim] (mode 1).
 * kv:  supplies V (kv->k is ignored), ctx_len and n_k; contiguous only.
 * u:   systematic uniforms [batch, num_q_heads].
 * feat_mask_out: optional uint8 [batch, num_kv_heads, head_dim], 1 where the
 *      feature row of K^T was read.  1 <= B_draws <= 64. */
santa_status_t santa_decode_bernoulli_qk(const void *q, const santa_kt_t *kt,
                                         const santa_kv_t *kv, const santa_shape_t *shape,
                                         float scale, int32_t B_draws, int32_t mode,
                                         const float *u_q, int32_t S, const float *u,
                                         int32_t *idx_out, uint8_t *feat_mask_out, void *out,
                                         void *ws, size_t ws_bytes, void *stream);

/* S2ANTA-flash (Sec. 3.3, "Speculative Sampling with Deferred Normalization";
 * App. "S2ANTA-Flash Pseudocode", Kernels 1 and 2).  Each row's keys are cut
 * into tiles of `tile` keys (tile t = [t*tile, min((t+1)*tile, L))); every
 * tile draws S_tile samples by systematic sampling on its own distribution
 * e_j / l_t, e_j = exp(s_j - m_t), m_t = max_t s, l_t = sum e_j (thresholds
 * (i + a)/S_tile with the tile's uniform a, inverse CDF as above, clamped to
 * the tile), giving the tile estimate O_t = (1/S_tile) sum_i V_{J_{t,i}}; the
 * tiles are merged by their softmax mass: out = sum_t W_t O_t / sum_t W_t,
 * W_t = exp(m_t - max_t m_t) l_t.  The paper's budget is S_tile ~ S/T for a
 * total of S draws over T tiles; the caller passes S_tile.
 * tile:    keys per tile, a power of two in [16, 1024].
 * S_tile:  draws per tile and query head, 1 <= S_tile <= 4096.
 * u:       float32 [batch, num_q_heads, T_max], T_max = ceil(n_k / tile): the
 *          uniform in [0,1) of each (row, tile).
 * idx_out: optional int32 [batch, num_q_heads, T_max, S_tile]: the drawn keys
 *          (logical positions) tile by tile, -1 for tiles at or past the row's
 *          length.
 * The workspace is sized by santa_workspace_size(..., SANTA_KIND_FLASH) (the
 * dense step's workspace).  Contiguous and paged caches.  Needs the fused
 * launch layout: returns SANTA_ERR_UNSUPPORTED under SANTA_PATH_MULTI and
 * when batch * num_kv_heads exceeds 4096. */
santa_status_t santa_decode_flash(const void *q, const santa_kv_t *kv, const santa_shape_t *shape,
                                  float scale, int32_t tile, int32_t S_tile, const float *u,
                                  int32_t *idx_out, void *out, void *ws, size_t ws_bytes,
                                  void *stream);

/* Profiling hook (not part of the method).  start_event and stop_event are
 * hipEvent_t handles created by the caller with timing enabled.  The next
 * santa_decode_* (or santa_stream_read) call made on the calling thread
 * attaches them to its own kernels: the GPU records start_event when the
 * call's first kernel is
 * dispatched and stop_event when its last kernel completes, so
 * hipEventElapsedTime(start, stop) is the call's execution time on the device
 * without host launch latency.  One-shot: that call consumes the request even
 * if it fails validation.  (NULL, NULL) cancels a pending request; exactly one
 * NULL is SANTA_ERR_INVALID_ARG.  The events stay owned by the caller and must
 * outlive the call's kernels. */
santa_status_t santa_time_next_call(void *start_event, void *stop_event);

/* Measurement helper (not part of the method): the attainable HBM read rate.
 * Streams `bytes` from the device buffer buf with the load the decode kernels
 * use for keys (16 bytes per lane, non-temporal, up to 16 loads in flight per
 * lane) over at most SANTA_STREAM_READ_GROUPS workgroups, each reading one
 * contiguous share, and writes to sink[w] (device,
 * caller-owned, SANTA_STREAM_READ_GROUPS uint32) the XOR of all 32-bit words
 * workgroup w read; words past the grid keep their contents, so with sink
 * zeroed first the XOR over sink is the XOR over the buffer.  buf must be
 * 16-byte aligned and bytes a positive multiple of 16 below
 * 2^34 * SANTA_STREAM_READ_GROUPS (else SANTA_ERR_INVALID_ARG).  Asynchronous
 * on `stream`; santa_time_next_call applies to it as to a decode call.  Timed
 * on a buffer the size of a step's algorithmic bytes, it is the ceiling those
 * bytes can be read at. */
#define SANTA_STREAM_READ_GROUPS 4096
santa_status_t santa_stream_read(const void *buf, size_t bytes, uint32_t *sink, void *stream);

/* Launch options (not part of the method): which kernels a call runs.  They
 * exist for tuning sweeps and for tests that cover every path; the defaults
 * choose by problem size.
 *   SANTA_PATH_AUTO        by measured speed: systematic and stratified steps
 *                          with at most 64 splits per row take the scheduled
 *                          path for S <= 1024 (paged caches up to 8192
 *                          workgroups, KV rows x splits, FP8 caches up to
 *                          2048), i.i.d. steps too at num_q_heads /
 *                          num_kv_heads <= 4 for S <= 256, or larger S on
 *                          grids of at most 256 workgroups; other sampled
 *                          steps whose rows fit one
 *                          resident round of about 1024 workgroups take one
 *                          persistent launch, larger ones the two-launch path;
 *   SANTA_PATH_ONE_LAUNCH  sampled steps: one persistent launch (k_fused_sampled);
 *   SANTA_PATH_TWO_LAUNCH  sampled steps: key stream with a CDF stash, then one
 *                          workgroup per query head (k_stream_cdf, k_value_heads);
 *   SANTA_PATH_MULTI       every step: the multi-kernel variant (score/CDF,
 *                          offsets, sampling and merge kernels);
 *   SANTA_PATH_SCHEDULED   systematic and stratified steps with at most 64
 *                          splits per row, and i.i.d. steps among them at
 *                          num_q_heads / num_kv_heads <= 4 (S <= 256, or
 *                          larger S on grids of at most 256 workgroups): one
 *                          hardware-scheduled launch, a
 *                          workgroup per split that keeps its CDF in LDS across
 *                          a row barrier (k_row_sampled); other sampled steps
 *                          as under AUTO.
 * splits: KV splits per row of the fused paths (0 = by size; at least
 * ceil(n_k / 1024)).  The options apply to every later call made on the
 * calling thread (santa_workspace_size and santa_plan_info included) until
 * they are set again; opts = NULL restores the defaults {AUTO, 0}.  A
 * workspace must be sized under the options of the calls that use it.
 * Returns SANTA_ERR_INVALID_ARG for an unknown path or splits outside
 * [0, 256]. */
typedef enum {
  SANTA_PATH_AUTO = 0,
  SANTA_PATH_ONE_LAUNCH = 1,
  SANTA_PATH_TWO_LAUNCH = 2,
  SANTA_PATH_MULTI = 3,
  SANTA_PATH_SCHEDULED = 4
} santa_path_t;

typedef struct {
  int32_t path;   /* santa_path_t */
  int32_t splits; /* 0 = by size */
} santa_options_t;

santa_status_t santa_set_options(const santa_options_t *opts);

/* The calling thread's current options (written to *opts). */
santa_status_t santa_get_options(santa_options_t *opts);

/* What a call with these arguments would launch under the calling thread's
 * options, without launching anything: the path taken (a santa_path_t other
 * than AUTO), the KV splits per row, the longest split in keys, the
 * workspace bytes (as santa_workspace_size) and the names of the kernels.
 * kernels points to a static string.  Same argument rules as
 * santa_workspace_size (S is ignored for dense and flash). */
typedef struct {
  int32_t path;
  int32_t splits;
  int32_t split_len;
  size_t workspace;
  const char *kernels;
} santa_plan_info_t;

santa_status_t santa_plan_info(const santa_shape_t *shape, const santa_kv_t *kv, int32_t S,
                               int32_t kind, santa_plan_info_t *info);

/* Human-readable name of a status code. */
const char *santa_status_string(santa_status_t status);

/* Message describing the last error returned on the calling thread ("" if none). */
const char *santa_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SANTA_H */
