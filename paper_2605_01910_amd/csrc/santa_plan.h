// santa_plan.h -- internal definitions shared by the host dispatcher and the
// kernels of libsanta: the launch plan (split length, workspace carve-up) and
// the by-value views the kernels receive.  Not part of the public ABI.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace santa {

constexpr int kHeadDim = 128;   // supported head dimension
constexpr int kThreads = 256;   // threads per workgroup (4 waves of 64)
constexpr int kSplitMax = 1024; // largest KV split (keys) handled by one workgroup
constexpr int kMaxSplits = 256; // largest number of splits per row in the fused kernels
constexpr int kRowTMax = 64;    // largest number of splits per row of the scheduled sampled path
// Scheduled path: grids of at most this many workgroups (one per CU of the
// MI355X) wait at the row barrier by polling the statistics directly and
// may hold large threshold sets in LDS.
constexpr int kDirectPollMax = 256;
// Per KV row, the fused paths keep a sync block of kSyncStride ints: the
// counters in the first 256 bytes, then (at u64 index kMailOffset) the
// scheduled sampled path's statistics mailbox, one u64 per (head < 8, split <
// kRowTMax), zero whenever no call is running.
constexpr int kMailOffset = 32;
constexpr int kSyncStride = 2 * kMailOffset + 2 * 8 * kRowTMax;
constexpr int kSyncRowsMax = 4096; // KV rows (batch * kv heads) of the fused paths' counter area
constexpr int kErrBytes = 128;    // the error flag's section

// Per-call launch plan.  The KV sequence of every (batch, kv head) row is cut
// into T splits of Ls keys; each split is one workgroup.  All sizes below are
// a pure function of (shape, n_k, S, kind), so santa_workspace_size() and the
// decode calls agree on the layout.
struct Plan {
  int B, Hq, Hkv, G, dtype;
  int elem;     // element type of K and V: 0 bfloat16, 1 float32, 2 FP8 E4M3 (q, out bfloat16)
  int n_k;      // max context length
  int Ls;       // keys per split (multi-kernel: multiple of 16; fused: longest split of
                // any row, multiple of 64; <= kSplitMax)
  int T;        // splits per row for n_k keys
  int S;        // samples per row (0 for dense)
  int kind;     // santa_kind_t
  int fused;    // 1: single persistent launch (per-row split lengths), 0: multi-kernel
  int rows;     // fused systematic / stratified: 1 = one hardware-scheduled launch, a
                // workgroup per split with row barriers (k_row_sampled)
  int split2;   // fused sampled: 1 = stream + CDF stash, then one workgroup per
                // query head; 0 = one persistent launch
  int64_t npitch;  // two-launch sampled: stash entries per query head (n_k rounded up to 64)
  // workspace carve-up (byte offsets, 256-aligned)
  size_t off_stats;  // float2 [B*Hq*T]     per-split (max, sum) in log2 units
  size_t off_stash;  // float  [B*Hq*T*Ls] split-local CDF of each row (multi-kernel);
                     // uint16 [B*Hq*npitch] in-block CDF fraction of each key (two launches)
  size_t off_coarse; // float  [B*Hq*npitch/32] fused: CDF at every 32-key block end
  size_t off_offs;   // float  [B*Hq*(T+1)] global split offsets of the CDF
  size_t off_alpha;  // float  [B*Hq*T]     per-split rescale exp2(m_t - m*)
  size_t off_rowst;  // float2 [B*Hq]       (m*, Z) per row
  size_t off_part;   // float  [B*Hkv*T*G*128] per-split partial outputs
  size_t off_flag;   // int    [B*Hkv*T]    1 if the split holds samples
  size_t off_bw;     // float  [B*Hq*128]   Bernoulli query weights
  size_t off_blist;  // int    [B*Hkv*128]  Bernoulli feature list
  size_t off_bn;     // int    [B*Hkv]      Bernoulli feature count
  size_t off_err;    // int    [1]          fused: a wait gave up
  size_t off_sync;   // u64    [kSyncRowsMax*kSyncStride/2] fused: per-row sync blocks
                     // (counters, mailbox); the area has the same offset and size in every
                     // layout, so calls of any kind and shape find their counters where
                     // earlier calls left them
  size_t total;
};

// KV cache as the kernels see it (see santa_kv_t for the addressing rules).
struct KvView {
  const void *k, *v;
  int64_t sb, sn, sh;
  const int32_t *ctx;   // nullable
  const int32_t *bt;    // nullable (contiguous)
  int32_t ps_log2;      // log2(page_size)
  int32_t max_pages;
  int32_t n_k;
  const void *k_new, *v_new;  // nullable: the current token's rows [B, Hkv, 128], appended in-launch
  const float *ks, *vs;       // FP8 cache: dequantisation scales [B*Hkv] of K and V (else null)
};

struct KtView {
  const void *kt;
  int64_t sb, sh, sd;
};

}  // namespace santa
