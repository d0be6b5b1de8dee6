// santa_fused.hip -- the default decode kernels.
//
// Every (batch b, KV head k) row is cut into Tb <= T splits of Ls keys (Ls =
// ceil(L_b / T) rounded up to 64); split t of a row is one work item of one
// 256-thread workgroup.  The persistent kernels hold R whole rows per round
// (R*T workgroups, all resident) and loop over rounds; a row's splits run on
// one XCD when R is a multiple of 8 (map_item).
//
// Sampled step, small batches (one launch, k_fused_sampled).  Per work item:
//   1. stream the split's keys (double-buffered 16-byte loads); the scores of
//      the G heads go to LDS and each lane keeps its running max;
//   2. the split-local CDF P_j = sum_{i<=j} exp2(s_i - m_t) is built in LDS
//      (Sec. 2.1: F is the running sum of the attention weights) and the split
//      publishes (m_t, l_t = P_last); then it arrives on the row counter and
//      waits until every split of the row has published (the last arrival does
//      not wait);
//   3. global offsets Off_t = sum_{t'<t} a_t' l_t' with a_t = exp2(m_t - m*)
//      and the total Z, identical in every split; threshold tau_r = ((r + u)/S) Z
//      (u per row, or u_r) is claimed by the split with Off_t <= tau_r <
//      Off_{t+1}; each claimed tau_r maps to the key #{j : a_t P_j <= tau_r -
//      Off_t} (the CDF interval holding it, App. A), clamped to the split; the
//      union of chosen keys over the group's heads is gathered once per key and
//      the G x 128 partial sums are published;
//   4. take an arrival rank; the last G arrivals each merge one head:
//      O_h = (1/S) sum_t o_t in split order.
// Sampled step, large batches (two launches): k_stream_cdf streams every work
// item and writes the split-local CDF at every 32-key block end (fp32), each
// key's CDF within its block as a 16-bit fraction of the block's mass (the
// stash) and the split statistics; then k_value_heads, one workgroup per
// query head, finds each threshold's split from the offsets, its 32-key block
// from the block ends and the key inside the block from the stash, and
// gathers the chosen V rows once per distinct key.
// Dense step (k_fused_dense): the split's exact softmax-weighted V sum o_t with
// (m_t, l_t); the last G arrivals merge O = sum_t a_t o_t / sum_t a_t l_t.
// Batches that need more than one resident round launch one workgroup per
// split instead, and the last arrival of a row merges all of its heads.
//
// Inside one launch, cross-workgroup data (statistics, partial sums,
// counters) is written and read with relaxed agent-scope atomics, which are
// coherent per access across the XCDs' L2s; a writer waits for its stores to
// complete before it arrives.  No cache-wide write-back or invalidation is
// issued.  Between the two launches of the two-launch path the kernel
// boundary orders the accesses and plain loads and stores are used.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "santa_kernels.h"
#include "santa_tiles.h"

namespace santa {

struct FusedArgs {
  KvView kv;
  const void *q;
  void *out;
  const float *u;
  int32_t *idx_out;
  float2 *stats;  // [B*Hq][T]          (m_t, l_t) per head and split
  float *part;    // [B*Hkv][T][G*128]  split partial outputs
  uint16_t *qstash;  // [B*Hq][npitch]  two-launch path: every key's CDF within its
                     //                 32-key block, in units of 2^-16 of the block's mass
  float *coarse;  // [B*Hq][npitch/32]  two-launch path: the CDF at every 32-key block end
  unsigned long long *sync;  // [B*Hkv][kSyncStride/2] arrival counter, counter base
  int *err;       // [1]                set if a wait gave up
  unsigned *tickets;  // [8]            one-launch large-batch path: next ticket of each XCD queue
  int B, Hq, Hkv, T, S;
  int ustage;     // the group's uniforms (G*S stratified, G systematic) staged in LDS if 1
  int64_t npitch; // stash floats per head row (n_k rounded up to 64)
  float invS, scale_log2;
  int tile_log2;  // flash: log2 of the tile length (16 .. kSplitMax keys)
  int S_tile;     // flash: samples per tile and head
  int Tmax;       // flash: tiles of the longest row, ceil(n_k / tile)
};

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kSpinLimit = 1 << 22;
constexpr int kAlign = 64;         // split lengths and stash rows are multiples of this many keys
constexpr int kBlock = 32;         // keys per block of the two-level CDF search
constexpr int kGatherUnroll = 8;   // V rows in flight per row slot in k_value_heads
constexpr int kUReg = 4;           // uniforms per thread fetched into registers before the stream
constexpr int kUStageMax = 4096;   // largest uniform set (floats per KV group) staged in LDS

// ---------------------------------------------------------------------------
// LDS sizes (dynamic shared memory), in floats
// ---------------------------------------------------------------------------
// LDS arrays of a split have a row pitch of kSplitMax keys (a compile-time
// constant, so per-key LDS offsets are immediates).
// k_fused_sampled: P [G][Lsmax] (scores, CDF; then the slot reduction and the
// merge scratch), cnt [G][Lsmax], list [max(Lsmax, 2G(T+1))] (offsets and
// split factors before the claims, the union list after), ul [G*S or G] if staged.
__host__ __device__ constexpr int imax(int x, int y) { return x > y ? x : y; }
__host__ __device__ constexpr int fused_p_floats(int G, int Lsmax, int T) {
  return imax(imax(G * Lsmax, 4 * G * kHeadDim), T + kThreads);
}
__host__ __device__ constexpr int fused_list_ints(int G, int Lsmax, int T) {
  return imax(Lsmax, 2 * G * (T + 1));
}
__host__ __device__ constexpr int fused_sampled_floats(int G, int Lsmax, int T, int ustaged) {
  return fused_p_floats(G, Lsmax, T) + G * Lsmax + fused_list_ints(G, Lsmax, T) + ustaged;
}
// k_fused_dense: s [G][Lsmax], red [4][G*128] (also the merge scratch).
// (Lsmax = kSplitMax in every launch.)
__host__ __device__ constexpr int fused_dense_floats(int G, int Lsmax, int T) {
  return G * Lsmax + imax(4 * G * kHeadDim, T + kThreads);
}
// flash mode of k_fused_dense: s [G][Lsmax] (scores, then tile CDFs), cnt
// [G][Lsmax] (counts, then weights; after the gather the slot reduction and
// merge scratch), list [Lsmax], tile statistics [G][2][kSplitMax/16].
__host__ __device__ constexpr int fused_flash_floats(int G, int Lsmax, int T) {
  return G * Lsmax + imax(G * Lsmax, imax(4 * G * kHeadDim, T + kThreads)) + Lsmax +
         2 * G * (kSplitMax / 16);
}
// k_stream_cdf: P [G][kSplitMax].
// k_value_heads: block ends [ncoarse], offsets [T+1], split factors [T], chosen
// keys and run list [2][kThreads], slot reduction [4][128].
__host__ __device__ constexpr int value_heads_floats(int T, int ncoarse) {
  return ncoarse + (T + 1) + T + 2 * kThreads + 4 * kHeadDim;
}

__device__ __forceinline__ void split_geometry(int L, int T, int &Ls, int &Tb, int align = kAlign) {
  if (L <= 0) {
    Ls = align;
    Tb = 0;
    return;
  }
  Ls = (((L + T - 1) / T) + align - 1) & ~(align - 1);
  Tb = (L + Ls - 1) / Ls;
}

// Work item of workgroup w within a round of R rows: row rho, split t.  When R
// is a multiple of 8, the splits of a row all run on one XCD (workgroups are
// dispatched round-robin over the 8 XCDs: w -> XCD w % 8).
__device__ __forceinline__ void map_item(int w, int T, int R, int &rho, int &t) {
  if ((R & 7) == 0) {
    const int x = w & 7, l = w >> 3;
    rho = x + 8 * (l / T);
    t = l % T;
  } else {
    rho = w / T;
    t = w % T;
  }
}

template <bool COHERENT>
__device__ __forceinline__ float2 ld2(const float2 *p) {
  if constexpr (COHERENT) return ld_coherent(p);
  return *p;
}

// ---------------------------------------------------------------------------
// Row counter.  sync[0] counts arrivals and only ever grows; sync[1] holds its
// value when the current call started (the base).  A split reads the base
// when it starts; the counter passes base + Tb once every split has published
// its statistics and base + 2 Tb once every split has published its partial
// sums; the last of those arrivals advances the base by 2 Tb for the next
// call, when every split has read it.  Nothing is reset between calls.
// ---------------------------------------------------------------------------
// All threads: make this workgroup's global stores complete, then take an
// arrival rank relative to `from` (block-uniform).
__device__ __forceinline__ int row_arrive(unsigned long long *sync, unsigned long long from,
                                          int *rank_lds) {
  wait_stores();
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned long long old =
        __hip_atomic_fetch_add(sync, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *rank_lds = (int)(old - from);
  }
  __syncthreads();
  return *rank_lds;
}

// All threads: wait until the counter reaches `target` (bounded spin; on
// giving up the error flag is set and the caller's results are not valid).
__device__ __forceinline__ void row_wait(const unsigned long long *sync, unsigned long long target,
                                         int *err) {
  if (threadIdx.x == 0) {
    int spins = 0;
    while (__hip_atomic_load(const_cast<unsigned long long *>(sync), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT) < target) {
      if (++spins > kSpinLimit) {
        atomicOr(err, 1);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  __syncthreads();
}

// row_wait for a workgroup that has already arrived: thread 0 holds in
// `arrived` the counter value its own arrival produced and skips the poll when
// that value already reaches `target` (the last arrival).
__device__ __forceinline__ void row_wait_unless(const unsigned long long *sync,
                                                unsigned long long target,
                                                unsigned long long arrived, int *err) {
  if (threadIdx.x == 0 && arrived < target) {
    int spins = 0;
    while (__hip_atomic_load(const_cast<unsigned long long *>(sync), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT) < target) {
      if (++spins > kSpinLimit) {
        atomicOr(err, 1);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  __syncthreads();
}

// One wave: global offsets of one head over the row's Tb splits.  off[0..Tb]
// receives Off_0 = 0, Off_{t+1} = Off_t + a_t l_t with a_t = exp2(m_t - m*),
// made exactly non-decreasing; al[t] receives a_t.  Returns m*.  Lane l owns
// splits l*ch .. l*ch+ch-1 (ch <= kMaxSplits / 64).
template <bool COHERENT>
__device__ __forceinline__ float head_offsets_wave(const float2 *st, int Tb, int lane, float *off,
                                                   float *al) {
  constexpr int CHM = kMaxSplits / 64;
  const int ch = (Tb + 63) >> 6;
  const int t0 = lane * ch;
  float2 sv[CHM];
#pragma unroll
  for (int i = 0; i < CHM; ++i)
    sv[i] = (i < ch && t0 + i < Tb) ? ld2<COHERENT>(st + t0 + i) : make_float2(-kInf, 0.0f);
  float m = -kInf;
#pragma unroll
  for (int i = 0; i < CHM; ++i) m = fmaxf(m, sv[i].x);
  m = wave_max(m);
  float a[CHM];
  float tot = 0.0f;
#pragma unroll
  for (int i = 0; i < CHM; ++i) {
    a[i] = (i < ch && t0 + i < Tb) ? fast_exp2(sv[i].x - m) : 0.0f;
    tot = fmaf(a[i], sv[i].y, tot);
  }
  const float base = wave_prev(0.0f, wave_incl_scan(tot));
  float run = base;
#pragma unroll
  for (int i = 0; i < CHM; ++i) run = fmaf(a[i], sv[i].y, run);
  // lane runs are non-decreasing; lift each to the largest end of earlier runs
  const float floor_v = wave_prev(0.0f, wave_incl_max(run));
  run = base;
#pragma unroll
  for (int i = 0; i < CHM; ++i) {
    run = fmaf(a[i], sv[i].y, run);
    if (i < ch && t0 + i < Tb) {
      off[t0 + i + 1] = fmaxf(run, floor_v);
      al[t0 + i] = a[i];
    }
  }
  if (lane == 0) off[0] = 0.0f;
  return m;
}

// out_h = scale * sum_t w_t part[t][h*128 + o] (w_t = 1 if w is null), divided
// by *den if den is not null.  Two interleaved halves of the splits, each
// summed in split order with 32 loads in flight, then added.  scratch holds
// kThreads floats.
template <typename E, int G>
__device__ __forceinline__ void merge_head(const float *part_row, int h, int Tb, const float *w,
                                           const float *den, float scale, float *scratch,
                                           E *out_row) {
  const int tid = threadIdx.x, o = tid & (kHeadDim - 1), g = tid >> 7;
  const float *ph = part_row + h * kHeadDim + o;
  const int nk = (Tb - g + 1) >> 1;  // splits g, g + 2, ...
  float s = 0.0f;
  for (int k0 = 0; k0 < nk; k0 += 32) {
    float v[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const int tt = g + 2 * (k0 + i);
      v[i] = k0 + i < nk ? ld_coherent(ph + (int64_t)tt * G * kHeadDim) : 0.0f;
    }
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const int tt = g + 2 * (k0 + i);
      if (k0 + i < nk) s = w ? fmaf(w[tt], v[i], s) : s + v[i];
    }
  }
  scratch[tid] = s;
  __syncthreads();
  if (tid < kHeadDim) {
    const float r = (scratch[tid] + scratch[tid + kHeadDim]) * scale;
    store_out(out_row + tid, den ? r / *den : r);
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// S2ANTA-flash value stage (Sec. 3.3; App. "S2ANTA-Flash Pseudocode", Kernel 1)
// ---------------------------------------------------------------------------
// Tile-local CDFs of one head's split, computed by one wave in place: the
// split (nrows <= kSplitMax scores in s, log2 units) holds tiles of 2^tl2 keys
// (16 <= tile; the split starts on a tile boundary).  For tile tau: m_tau =
// max s, P_j = sum_{i <= j in tau} exp2(s_i - m_tau), written over s[j];
// tm[tau] = m_tau and tl[tau] = P_last.  Lane l owns keys 16l..16l+15 and a
// tile spans 2^tl2 / 16 aligned lanes, so the tile max is a butterfly and the
// tile prefix a segmented scan over those lanes, made non-decreasing by a
// segmented prefix max (fixed order: equal inputs give equal CDFs).
__device__ __forceinline__ void wave_tile_cdf(float *s, int nrows, int lane, int tl2, float *tm,
                                              float *tl) {
  constexpr int CH = kSplitMax / 64;
  const int j0 = lane * CH;
  const int seg = (1 << tl2) / CH;  // lanes per tile, 1 .. 64
  const int pos = lane & (seg - 1);
  float x[CH];
#pragma unroll
  for (int i = 0; i < CH / 4; ++i) {
    const float4 v = reinterpret_cast<const float4 *>(s + j0)[i];
    x[4 * i] = v.x;
    x[4 * i + 1] = v.y;
    x[4 * i + 2] = v.z;
    x[4 * i + 3] = v.w;
  }
  float m = -kInf;
#pragma unroll
  for (int i = 0; i < CH; ++i) m = (j0 + i < nrows) ? fmaxf(m, x[i]) : m;
  for (int d = 1; d < seg; d <<= 1) m = fmaxf(m, __shfl_xor(m, d));
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    acc += (j0 + i < nrows) ? fast_exp2(x[i] - m) : 0.0f;
    x[i] = acc;
  }
  float incl = acc;
  for (int d = 1; d < seg; d <<= 1) {
    const float y = __shfl_up(incl, d);
    incl += pos >= d ? y : 0.0f;
  }
  for (int d = 1; d < seg; d <<= 1) {
    const float y = __shfl_up(incl, d);
    incl = pos >= d ? fmaxf(incl, y) : incl;
  }
  const float prev = __shfl_up(incl, 1);
  const float base = pos == 0 ? 0.0f : prev;
  if (j0 < nrows) {
#pragma unroll
    for (int i = 0; i < CH / 4; ++i)
      reinterpret_cast<float4 *>(s + j0)[i] =
          make_float4(fminf(base + x[4 * i], incl), fminf(base + x[4 * i + 1], incl),
                      fminf(base + x[4 * i + 2], incl), fminf(base + x[4 * i + 3], incl));
  }
  if (pos == seg - 1 && (lane / seg) * (1 << tl2) < nrows) {
    tm[lane / seg] = m;
    tl[lane / seg] = incl;
  }
}

// #{j < n : P_j <= x} over a non-decreasing LDS CDF (n <= kSplitMax): branch-
// free binary lifting in a rolled loop.
__device__ __forceinline__ int lds_count_le(const float *P, int n, float x) {
  int pos = 0;
#pragma unroll 1
  for (int step = 1 << (31 - __clz(n)); step > 0; step >>= 1) {
    const int np = pos + step;
    const float v = P[min(np, n) - 1];
    pos = (np <= n && v <= x) ? np : pos;
  }
  return pos;
}

// Flash draws of one split (Kernel 1): every tile tau of the split and every
// head h takes S_tile systematic draws on the tile's own distribution: draw i
// is the key whose tile-CDF interval holds ((i + a)/S_tile) l_tau, a = u of
// (head, tile) (App. A's inverse CDF, clamped to the tile).  Counts go to cnt;
// then each drawn key's count becomes the weight count * exp2(m_tau - m_w) *
// l_tau / S_tile (m_w: the split max), so the split's partial sum is
// o_w = sum_tau exp2(m_tau - m_w) l_tau O_tau with O_tau the tile estimate.
// Returns (block-uniform) whether any key was drawn.
template <int G>
__device__ __forceinline__ bool flash_draws(const FusedArgs &a, const float *P, int pitch, int *cnt,
                                            const float *tst, const float *mh, int start,
                                            int nrows, int64_t row0) {
  const int tid = threadIdx.x, tl2 = a.tile_log2, St = a.S_tile;
  const int ntile = (nrows + (1 << tl2) - 1) >> tl2;
  const int per_h = ntile * St;
  const float invSt = 1.0f / (float)St;
  const int gt0 = start >> tl2;  // global index of the split's first tile
  for (int i = tid; i < G * per_h; i += kThreads) {
    const int h = i / per_h, rem = i - h * per_h, tau = rem / St, is = rem - tau * St;
    const int t0 = tau << tl2, n = min(1 << tl2, nrows - t0);
    const float l = tst[(2 * h + 1) * (kSplitMax / 16) + tau];
    const float ua = a.u[(row0 + h) * a.Tmax + gt0 + tau];
    const float x = (((float)is + ua) * invSt) * l;
    const int k = lds_count_le(P + h * pitch + t0, n, x);
    const int j = t0 + (k < n ? k : n - 1);
    atomicAdd(&cnt[h * pitch + j], 1);
    if (a.idx_out) a.idx_out[((row0 + h) * a.Tmax + gt0 + tau) * St + is] = start + j;
  }
  __syncthreads();
  // counts -> weights
  for (int i = tid; i < G * nrows; i += kThreads) {
    const int h = i / nrows, j = i - h * nrows;
    const int c = cnt[h * pitch + j];
    if (c) {
      const int tau = j >> tl2;
      const float m = tst[(2 * h) * (kSplitMax / 16) + tau];
      const float l = tst[(2 * h + 1) * (kSplitMax / 16) + tau];
      cnt[h * pitch + j] = __float_as_int((float)c * (fast_exp2(m - mh[h]) * l * invSt));
    }
  }
  __syncthreads();
  return G * per_h > 0;
}

// ---------------------------------------------------------------------------
// Small-batch sampled step
// ---------------------------------------------------------------------------
// #{j < nrows : a P_j <= x} over a non-decreasing LDS CDF P (nrows <=
// kSplitMax): branch-free binary lifting in a rolled loop (a handful of
// instructions; one LDS read per step).
__device__ __forceinline__ int lds_cdf_count(const float *Ph, int nrows, float a, float x) {
  int pos = 0;
#pragma unroll 1
  for (int step = 1 << (31 - __clz(nrows)); step > 0; step >>= 1) {
    const int np = pos + step;
    const float v = Ph[min(np, nrows) - 1];
    pos = (np <= nrows && a * v <= x) ? np : pos;
  }
  return pos;
}

// Sampling modes of the sampled kernels: the thresholds tau_r of one head
// (Sec. 2.1, "Construction"; Sec. 2 for the i.i.d. draws), in global CDF
// units (Z the row's total):
//   kSys:   ((r + u)/S) Z with one uniform u (uh[0]);
//   kStrat: ((r + u_r)/S) Z (uh[r]);
//   kIid:   T_r Z with T the head's sorted i.i.d. thresholds (uh[r], built by
//           wave_iid_thresholds).
constexpr int kSys = 0, kStrat = 1, kIid = 2;

template <int MODE>
__device__ __forceinline__ float tau_of(const float *uh, int r, float invS, float Z) {
  if constexpr (MODE == kIid) return uh[r] * Z;
  else return threshold(r, MODE == kStrat ? uh[r] : uh[0], invS, Z);
}

// Sorted thresholds of the i.i.d. estimator from S + 1 uniforms u without a
// sort, by one wave: E_i = -log2(1 - u_i) (unit exponentials up to the factor
// ln 2, which the ratio cancels), C_m = sum_{i <= m} E_i in double, T_m = C_m /
// C_S for m < S -- the normalised partial sums of S + 1 exponentials are the
// order statistics of S independent uniforms.  Lane l sums a contiguous chunk
// of the E_i; the chunk totals are joined by a wave scan made non-decreasing
// by a prefix max and every partial sum is capped at its lane's total, so T
// is non-decreasing.  u: S + 1 floats; T: S floats (LDS).
__device__ __forceinline__ void wave_iid_thresholds(const float *u, int S, float *T, int lane) {
  const int n = S + 1, ch = (n + 63) >> 6, i0 = lane * ch;
  double tot = 0.0;
  for (int k = 0; k < ch; ++k)
    if (i0 + k < n) tot -= (double)__builtin_amdgcn_logf(1.0f - u[i0 + k]);
  double incl = tot;
  for (int d = 1; d < 64; d <<= 1) {
    const double y = __shfl_up(incl, d);
    incl += lane >= d ? y : 0.0;
  }
  for (int d = 1; d < 64; d <<= 1) {
    const double y = __shfl_up(incl, d);
    incl = lane >= d ? fmax(incl, y) : incl;
  }
  const double prev = __shfl_up(incl, 1);
  const double total = __shfl(incl, 63);
  const double inv = total > 0.0 ? 1.0 / total : 0.0;
  double run = lane == 0 ? 0.0 : prev;
  for (int k = 0; k < ch; ++k) {
    const int i = i0 + k;
    if (i < n) {
      run -= (double)__builtin_amdgcn_logf(1.0f - u[i]);
      if (i < S) T[i] = (float)(fmin(run, incl) * inv);
    }
  }
}

// Claims and inverse CDF of one split for thresholds held in LDS without a
// closed-form count (the i.i.d. mode's sorted T_r Z; G*S <= kUStageMax): the
// G*S thresholds are numbered n = r*G + h (the G heads of one r on
// neighbouring lanes) and thread i evaluates n = i, i + kThreads, ...; those
// with lo <= tau < hi belong to this split and map to the key #{j : a P_j <=
// tau - lo} (the CDF interval holding tau, App. A), clamped to the split.
// Counts per key go to cnt (LDS), indices to idx_out.  Returns (block-uniform)
// whether the split holds any sample.
template <int G, int MODE>
__device__ __forceinline__ bool claim_scan(const HeadClaim *hc, const float *ul, int S, float invS,
                                           const float *P, int pitch, int start, int nrows,
                                           int64_t row0, int *cnt, int32_t *__restrict__ idx_out) {
  const int tid = threadIdx.x;
  const int h = tid % G;  // the same head on every pass (kThreads is a multiple of G)
  const HeadClaim c = hc[h];
  const float *Ph = P + h * pitch;
  bool any = false;
#pragma unroll 1
  for (int n = tid; n < G * S; n += kThreads) {
    const int r = n / G;
    const float tau = tau_of<MODE>(ul + h * (MODE == kSys ? 1 : S), r, invS, c.Z);
    if ((tau >= c.lo) & (tau < c.hi)) {
      const int pos = lds_cdf_count(Ph, nrows, c.a, tau - c.lo);
      const int j = pos < nrows ? pos : nrows - 1;
      atomicAdd(&cnt[h * pitch + j], 1);
      if (idx_out) idx_out[(row0 + h) * S + r] = start + j;
      any = true;
    }
  }
  return __syncthreads_or(any) != 0;
}

// Number of one head's thresholds below y, N(y) = #{r < S : tau_r < y}, for
// sorted thresholds (kSys, kStrat; uniforms in LDS).  tau_r is non-decreasing
// in r (its fp32 evaluation is monotone), so N is its closed-form estimate --
// kSys: ceil(y S/Z - u); kStrat: floor(y S/Z) + 1, the strata up to y's --
// corrected until tau_{N-1} < y <= tau_N holds for tau as evaluated by the
// claims (tau_of).  The estimate is off by at most one step of fp32 rounding
// for S below 2^23: both neighbours are checked at once, and a loop only runs
// when a check fails.  u0 is the head's uniform (kSys); sZ = S / Z; y = +inf
// gives S.
template <int MODE>
__device__ __forceinline__ int count_below(const float *uh, float u0, int S, float invS, float Z,
                                           float sZ, float y) {
  static_assert(MODE == kSys || MODE == kStrat, "sorted thresholds with a closed form");
  auto tau = [&](int r) {
    return MODE == kSys ? threshold(r, u0, invS, Z) : tau_of<MODE>(uh, r, invS, Z);
  };
  const float q = fminf(y * sZ, (float)S + 2.0f);
  int n = MODE == kSys ? (int)ceilf(q - u0) : (int)floorf(q) + 1;
  n = min(max(n, 0), S);
  const float tm = n > 0 ? tau(n - 1) : -kInf;
  const float tp = n < S ? tau(n) : kInf;
  if (tm >= y) {
    --n;
    while (n > 0 && tau(n - 1) >= y) --n;
  } else if (tp < y) {
    ++n;
    while (n < S && tau(n) < y) ++n;
  }
  return n;
}

// Claimed ranges of one split for sorted thresholds (kSys, kStrat; uniforms
// in LDS): head h claims r in [N(lo), N(hi)) -- exactly the r with lo <= tau_r
// < hi -- found in closed form by threads 2h and 2h + 1 (count_below), so
// claim_keys then inverts only the claimed thresholds.  rng: [G][2] (LDS).
template <int G, int MODE>
__device__ __forceinline__ void claim_ranges_closed(const HeadClaim *hc, const float *ul, int S,
                                                    float invS, int *rng) {
  const int tid = threadIdx.x;
  if (tid < 2 * G) {
    const int h = tid >> 1;
    const HeadClaim c = hc[h];
    const float *uh = ul + h * (MODE == kSys ? 1 : S);
    rng[tid] = count_below<MODE>(uh, MODE == kSys ? uh[0] : 0.0f, S, invS, c.Z, (float)S / c.Z,
                                 (tid & 1) ? c.hi : c.lo);
  }
  __syncthreads();
}

// Threshold r of head h is claimed iff lo <= tau_r < hi.  tau_r is
// non-decreasing in r (fp32 rounding is monotone), so the claimed r form the
// range [#{r : tau_r < lo}, #{r : tau_r < hi}); threads 2h and 2h+1 count the
// two ends by binary search.
template <int G, int MODE>
__device__ __forceinline__ void claim_ranges(const HeadClaim *hc, const float *us, int64_t ustride,
                                             int S, float invS, int *rng /* [G][2] */) {
  const int tid = threadIdx.x;
  if (tid < 2 * G) {
    const int h = tid >> 1;
    const HeadClaim c = hc[h];
    const float bound = (tid & 1) ? c.hi : c.lo;
    const float *uh = us + h * ustride;
    int pos = 0;
    for (int step = 1 << (31 - __clz(S)); step > 0; step >>= 1) {
      const int np = pos + step;
      if (np <= S && tau_of<MODE>(uh, np - 1, invS, c.Z) < bound) pos = np;
    }
    rng[tid] = pos;
  }
  __syncthreads();
}

// Inverse CDF of the claimed thresholds of every head (LDS CDF P of the
// split): key #{j : a P_j <= tau - lo}, clamped to the split.  Counts per key
// go to cnt (LDS), indices to idx_out.  Returns (block-uniform) whether the
// split holds any sample.
template <int G, int MODE>
__device__ __forceinline__ bool claim_keys(const HeadClaim *hc, const int *rng, const float *us,
                                           int64_t ustride, int S, float invS, const float *P,
                                           int pitch, int start, int nrows, int64_t row0, int *cnt,
                                           int32_t *__restrict__ idx_out) {
  const int tid = threadIdx.x;
  int first[G + 1];
  first[0] = 0;
#pragma unroll
  for (int h = 0; h < G; ++h) first[h + 1] = first[h] + max(0, rng[2 * h + 1] - rng[2 * h]);
  const int total = first[G];
  for (int i = tid; i < total; i += kThreads) {
    int h = 0;
#pragma unroll
    for (int k = 1; k < G; ++k) h += (i >= first[k]) ? 1 : 0;
    const int r = rng[2 * h] + (i - first[h]);
    const HeadClaim c = hc[h];
    const float tau = tau_of<MODE>(us + h * ustride, r, invS, c.Z);
    const int pos = lds_cdf_count(P + h * pitch, nrows, c.a, tau - c.lo);
    const int j = pos < nrows ? pos : nrows - 1;
    atomicAdd(&cnt[h * pitch + j], 1);
    if (idx_out) idx_out[(row0 + h) * S + r] = start + j;
  }
  return total > 0;
}

// Value stage of one split with one query head per wave (G >= 4), for a short
// compacted union list (list[0..nlist), the group's chosen keys in key order):
// wave w accumulates heads w, w + 4, ... over the whole list (4 rows per wave
// instruction, 4 rows in flight per row slot), sums its 4 row slots with lane
// swaps and writes the heads' 128 partial sums directly, with no workgroup
// reduction: O_h += c_{h,j} V_j (Sec. 2, the stochastic add-only attention).
// FW: cnt holds float weights (bit patterns) instead of counts.
template <typename E, int G, bool PAGED, bool FW = false>
__device__ __forceinline__ void gather_heads_waves(const KvView &kv, int b, int kvh, int start,
                                                   const int *cnt, int pitch, const int *list,
                                                   int nlist, float *__restrict__ part_out) {
  static_assert(G % 4 == 0, "one head per wave needs G >= 4");
  constexpr int HW = G / 4, U = 4;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, rs = lane >> 4, c = lane & 15;
  const E *V = static_cast<const E *>(kv.v);
  float acc[HW][8];
#pragma unroll
  for (int hw = 0; hw < HW; ++hw)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[hw][i] = 0.0f;
  for (int e0 = rs; e0 < nlist; e0 += 4 * U) {
    Chunk<E> ch[U];
    int jj[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = e0 + 4 * u;
      jj[u] = e < nlist ? list[e] : -1;
      ch[u] = jj[u] >= 0 ? Chunk<E>::load(V + row_offset<PAGED>(kv, b, kvh, start + jj[u]) + c * 8)
                         : Chunk<E>::zero();
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (jj[u] < 0) continue;
      float f[8];
      ch[u].to_float(f);
#pragma unroll
      for (int hw = 0; hw < HW; ++hw) {
        const int cw = cnt[(wave + 4 * hw) * pitch + jj[u]];
        const float w = FW ? __int_as_float(cw) : (float)cw;
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[hw][i] = fmaf(w, f[i], acc[hw][i]);
      }
    }
  }
#pragma unroll
  for (int hw = 0; hw < HW; ++hw)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[hw][i] = xor32_sum(xor16_sum(acc[hw][i]));
  if (lane < 16) {
#pragma unroll
    for (int hw = 0; hw < HW; ++hw) {
      float2 *dst = reinterpret_cast<float2 *>(part_out + (wave + 4 * hw) * kHeadDim + c * 8);
#pragma unroll
      for (int i = 0; i < 4; ++i) st_coherent(dst + i, make_float2(acc[hw][2 * i], acc[hw][2 * i + 1]));
    }
  }
}

// APPEND: the fused current-token append (append_current) is compiled in;
// calls without one run the kernel without that code.
template <typename E, int G, bool PAGED, int MODE, bool APPEND = false>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void k_fused_sampled(FusedArgs a) {
  constexpr bool STRAT = MODE == kStrat;
  extern __shared__ __attribute__((aligned(16))) float dyn[];
  constexpr int pitch = kSplitMax;
  const int T = a.T;
  float *P = dyn;
  int *cnt = reinterpret_cast<int *>(dyn + fused_p_floats(G, pitch, T));
  int *list = cnt + G * pitch;
  float *offl = reinterpret_cast<float *>(list);  // [G][T+1], then al [G][T]
  float *all = offl + G * (T + 1);
  float *ul = reinterpret_cast<float *>(list + fused_list_ints(G, pitch, T));
  __shared__ HeadClaim hc[G];
  __shared__ float mh[G], lh[G], mtmp[8 * G];
  __shared__ int rank_lds, rng[2 * G];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nrk = a.B * a.Hkv;
  const int R = gridDim.x / T;  // rows per round
  int rho, t;
  map_item(blockIdx.x, T, R, rho, t);
  E *out = static_cast<E *>(a.out);

  for (int rbase = 0; rbase < nrk; rbase += R) {
    __builtin_amdgcn_s_setprio(0);
    const int rowkv = rbase + rho;
    if (rowkv >= nrk) break;
    const int b = rowkv / a.Hkv, kvh = rowkv % a.Hkv;
    const int64_t row0 = (int64_t)b * a.Hq + kvh * G;
    const int L = seq_len(a.kv, b);
    int Ls, Tb;
    split_geometry(L, T, Ls, Tb);
    if (t >= Tb) {
      if (Tb == 0 && t == 0) {  // empty sequence: zero output, no samples
        for (int o = tid; o < G * kHeadDim; o += kThreads) store_out(out + row0 * kHeadDim + o, 0.0f);
        if (a.idx_out)
          for (int o = tid; o < G * a.S; o += kThreads) a.idx_out[row0 * a.S + o] = -1;
      }
      continue;
    }
    const int start = t * Ls, nrows = min(Ls, L - start);
    if constexpr (APPEND) append_current<E, PAGED>(a.kv, b, kvh, a.Hkv, start, nrows, L);
    unsigned long long *sync = a.sync + (int64_t)rowkv * (kSyncStride / 2);
    const unsigned long long base =
        __hip_atomic_load(sync + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    float *part_row = a.part + (int64_t)rowkv * T * G * kHeadDim;

    // uniforms of the group: G*S (stratified), G*(S+1) (i.i.d.) or G
    // (systematic) consecutive floats, staged in LDS when there are few of
    // them (always for i.i.d.); the first kUReg*kThreads are fetched into
    // registers before the keys stream
    const int upr = MODE == kIid ? a.S + 1 : (STRAT ? a.S : 1);  // uniforms per head
    const float *us = a.u + row0 * upr;
    const int64_t ustride = upr;
    const int nu = G * upr;
    float ureg[kUReg];
    if (a.ustage) {
#pragma unroll
      for (int k = 0; k < kUReg; ++k) {
        const int i = tid + k * kThreads;
        ureg[k] = i < nu ? us[i] : 0.0f;
      }
    }

    // 1. scores of the G heads into LDS; split max m_t per head
    const QRegs<E, G> qr = load_q<E, G>(static_cast<const E *>(a.q), b, a.Hq, kvh, tid & 15);
    float mx[G];
    score_tile<E, G, PAGED, score_unroll<E, G>()>(a.kv, b, kvh, start, nrows, qr, a.scale_log2, P,
                                                  pitch, mx);
    // from here on the split is on its row's critical path: its waves issue
    // ahead of waves that are still streaming keys
    __builtin_amdgcn_s_setprio(3);
    block_max_heads<G>(mx, mtmp, mh);

    // 2. split-local CDF of head h by wave h; the split's (m_t, l_t = P_last)
    //    is published as soon as its CDF is built, then the workgroup arrives
    for (int h = wave; h < G; h += kThreads / 64) {
      float *Ph = P + h * pitch;
      wave_split_cdf_m(Ph, nrows, lane, mh[h]);
      if (lane == 0) st_coherent(a.stats + (row0 + h) * T + t, make_float2(mh[h], Ph[nrows - 1]));
    }
    wait_stores();
    __syncthreads();
    unsigned long long arrived = 0;
    if (tid == 0)
      arrived = __hip_atomic_fetch_add(sync, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1;

    // zero counts and stage the uniforms while the other splits arrive, then
    // wait until every split of the row has published (the last arrival does
    // not wait)
    for (int i = tid; i < G * pitch; i += kThreads) cnt[i] = 0;
    if (a.ustage) {
#pragma unroll
      for (int k = 0; k < kUReg; ++k) {
        const int i = tid + k * kThreads;
        if (i < nu) ul[i] = ureg[k];
      }
      for (int i = tid + kUReg * kThreads; i < nu; i += kThreads) ul[i] = us[i];
      if constexpr (MODE == kIid) {
        // each head's S + 1 uniforms become its S sorted thresholds, after
        // the raw uniforms in LDS
        __syncthreads();
        for (int h = wave; h < G; h += kThreads / 64)
          wave_iid_thresholds(ul + h * upr, a.S, ul + nu + h * a.S, lane);
      }
    }
    row_wait_unless(sync, base + (unsigned long long)Tb, arrived, a.err);

    // 3. offsets, claims, inverse CDF, union gather, partial sums
    for (int h = wave; h < G; h += kThreads / 64) {
      float *oh = offl + h * (T + 1), *ah = all + h * T;
      head_offsets_wave<true>(a.stats + (row0 + h) * T, Tb, lane, oh, ah);
      if (lane == 0) hc[h] = HeadClaim{oh[t], t == Tb - 1 ? kInf : oh[t + 1], oh[Tb], ah[t]};
    }
    __syncthreads();
    bool has;
    if (a.ustage && MODE != kIid) {
      constexpr int M = MODE == kIid ? kSys : MODE;
      claim_ranges_closed<G, M>(hc, ul, a.S, a.invS, rng);
      has = claim_keys<G, M>(hc, rng, ul, M == kSys ? 1 : a.S, a.S, a.invS, P, pitch, start,
                             nrows, row0, cnt, a.idx_out);
    } else if (a.ustage) {
      has = claim_scan<G, MODE>(hc, ul + nu, a.S, a.invS, P, pitch, start, nrows, row0, cnt,
                                a.idx_out);
    } else {
      claim_ranges<G, MODE>(hc, us, ustride, a.S, a.invS, rng);
      has = claim_keys<G, MODE>(hc, rng, us, ustride, a.S, a.invS, P, pitch, start, nrows, row0,
                                cnt, a.idx_out);
    }
    __syncthreads();  // counts complete; offl/all are no longer needed
    if (has) {
      float *po = part_row + (int64_t)t * G * kHeadDim;
      if constexpr (G >= 4) {
        // a short union (one pass of a wave's 16 rows) goes one head per wave,
        // with no workgroup reduction; a long one (large S) is shared by all
        // 16 row slots of the workgroup, so it takes nlist / (16 UG) dependent
        // passes instead of nlist / 16
        const int nlist = compact_union<G>(cnt, pitch, nrows, list);
        constexpr int UG = (sizeof(E) == 2 && G <= 4) ? 8 : 4;
        if (nlist <= 16)
          gather_heads_waves<E, G, PAGED>(a.kv, b, kvh, start, cnt, pitch, list, nlist, po);
        else
          gather_list<E, G, PAGED, true, false, UG>(a.kv, b, kvh, start, list, nlist, P, pitch,
                                                    cnt, po);
      } else {
        gather_union<E, G, PAGED, true>(a.kv, b, kvh, start, nrows, P, pitch, cnt, list, po);
      }
    } else {  // a split without samples contributes zeros
      float2 *pz = reinterpret_cast<float2 *>(part_row + (int64_t)t * G * kHeadDim);
      for (int o2 = tid; o2 < G * kHeadDim / 2; o2 += kThreads) st_coherent(pz + o2, make_float2(0.f, 0.f));
    }

    // 4. arrive; the last min(G, Tb) arrivals merge one or more heads each
    const int W = min(G, Tb);
    const int rank = row_arrive(sync, base + (unsigned long long)Tb, &rank_lds);
    if (rank < Tb - W) continue;
    if (rank == Tb - 1) {
      if (tid == 0)
        __hip_atomic_store(sync + 1, base + 2ull * Tb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      row_wait(sync, base + 2ull * Tb, a.err);
    }
    for (int h = rank - (Tb - W); h < G; h += W)
      merge_head<E, G>(part_row, h, Tb, nullptr, nullptr, a.invS, P, out + (row0 + h) * kHeadDim);
  }
}

// ---------------------------------------------------------------------------
// Dense step
// ---------------------------------------------------------------------------
// PERSIST: a resident grid of R whole rows per round (small batches; the last
// min(G, Tb) arrivals of a row merge one head each).  Otherwise one work item
// per workgroup, hardware-scheduled (large batches): the row's last arrival
// merges every head and nothing waits, so the grid need not be resident.
// FLASH: the split's value stage is S2ANTA-flash (Sec. 3.3; App. "S2ANTA-Flash
// Pseudocode"): S_tile draws per tile and head on the tile's own distribution
// instead of the exact weighted sum; the split publishes o_w = sum_tau
// exp2(m_tau - m_w) l_tau O_tau with l_w = sum_tau exp2(m_tau - m_w) l_tau, so
// the same merge gives O = sum_tau W_tau O_tau / sum_tau W_tau (Kernel 2).
template <typename E, int G, bool PAGED, bool PERSIST, bool FLASH = false, bool APPEND = false>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(PERSIST ? 2 : 3))) void k_fused_dense(FusedArgs a) {
  // dynamic LDS: s [G][pitch] scores / weights, red [4][G*128] (also the merge scratch);
  // flash: s, cnt [G][pitch] (later red), list [pitch], tile statistics [G][2][kSplitMax/16]
  extern __shared__ __attribute__((aligned(16))) float dyn[];
  constexpr int pitch = kSplitMax;
  float *s = dyn;
  float *red = s + G * pitch;
  int *cnt = reinterpret_cast<int *>(red);
  int *list = cnt + imax(G * pitch, imax(4 * G * kHeadDim, a.T + kThreads));
  float *tst = reinterpret_cast<float *>(list + pitch);
  __shared__ float mh[G], lh[G], mtmp[4 * G], den;
  __shared__ int rank_lds;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, c = tid & 15;
  const int nrk = a.B * a.Hkv, T = a.T;
  const int R = gridDim.x / T;  // rows per round
  int rho, t;
  map_item(blockIdx.x, T, R, rho, t);
  E *out = static_cast<E *>(a.out);
  const int align = FLASH ? imax(kAlign, 1 << a.tile_log2) : kAlign;

  for (int rbase = 0; rbase < nrk; rbase += R) {
    __builtin_amdgcn_s_setprio(0);
    const int rowkv = rbase + rho;
    if (rowkv >= nrk) break;
    const int b = rowkv / a.Hkv, kvh = rowkv % a.Hkv;
    const int64_t row0 = (int64_t)b * a.Hq + kvh * G;
    const int L = seq_len(a.kv, b);
    int Ls, Tb;
    split_geometry(L, T, Ls, Tb, align);
    if constexpr (FLASH) {
      // tiles no split covers (past the row's length) have no draws
      if (a.idx_out && (t == Tb - 1 || (Tb == 0 && t == 0))) {
        const int t_end = (L + (1 << a.tile_log2) - 1) >> a.tile_log2;
        const int nt = (a.Tmax - t_end) * a.S_tile;
        for (int i = tid; i < G * nt; i += kThreads) {
          const int h = i / nt, k = i - h * nt;
          a.idx_out[((row0 + h) * a.Tmax + t_end) * a.S_tile + k] = -1;
        }
      }
    }
    if (t >= Tb) {
      if (Tb == 0 && t == 0)
        for (int o = tid; o < G * kHeadDim; o += kThreads) store_out(out + row0 * kHeadDim + o, 0.0f);
      continue;
    }
    const int start = t * Ls, nrows = min(Ls, L - start);
    if constexpr (APPEND) append_current<E, PAGED>(a.kv, b, kvh, a.Hkv, start, nrows, L);
    unsigned long long *sync = a.sync + (int64_t)rowkv * (kSyncStride / 2);
    const unsigned long long base =
        __hip_atomic_load(sync + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    float *part_row = a.part + (int64_t)rowkv * T * G * kHeadDim;

    const QRegs<E, G> qr = load_q<E, G>(static_cast<const E *>(a.q), b, a.Hq, kvh, c);
    float mx[G];
    constexpr int U = PERSIST ? score_unroll<E, G>() : 4;
    score_tile<E, G, PAGED, U>(a.kv, b, kvh, start, nrows, qr, a.scale_log2, s, pitch, mx);
    block_max_heads<G>(mx, mtmp, mh);
    if constexpr (FLASH) {
      // tile CDFs (wave h: head h), the split normaliser l_w, zeroed counts
      constexpr int TS = kSplitMax / 16;
      for (int h = wave; h < G; h += kThreads / 64) {
        wave_tile_cdf(s + h * pitch, nrows, lane, a.tile_log2, tst + 2 * h * TS, tst + (2 * h + 1) * TS);
        const int ntile = (nrows + (1 << a.tile_log2) - 1) >> a.tile_log2;
        float l = 0.0f;
        for (int tau = lane; tau < ntile; tau += 64)
          l += fast_exp2(tst[2 * h * TS + tau] - mh[h]) * tst[(2 * h + 1) * TS + tau];
        l = wave_sum(l);
        if (lane == 0) lh[h] = l;
      }
      for (int i = tid; i < G * pitch; i += kThreads) cnt[i] = 0;
      __syncthreads();
      __builtin_amdgcn_s_setprio(3);
      const bool has = flash_draws<G>(a, s, pitch, cnt, tst, mh, start, nrows, row0);
      // the draws of a split can reach many distinct rows, so all 16 row slots
      // of the workgroup share the union list (8 rows in flight per slot, 4
      // for the wider accumulators of fp32 rows or G = 8)
      if (has) {
        constexpr int UG = (sizeof(E) == 2 && G <= 4) ? 8 : 4;
        gather_union<E, G, PAGED, true, true, UG>(a.kv, b, kvh, start, nrows, s, pitch, cnt, list,
                                                  part_row + (int64_t)t * G * kHeadDim);
      } else {
        float2 *pz = reinterpret_cast<float2 *>(part_row + (int64_t)t * G * kHeadDim);
        for (int o2 = tid; o2 < G * kHeadDim / 2; o2 += kThreads) st_coherent(pz + o2, make_float2(0.f, 0.f));
      }
    } else {
      for (int h = wave; h < G; h += kThreads / 64) {
        float *sh = s + h * pitch;
        const float m = mh[h];
        float l = 0.0f;
        for (int j = lane; j < nrows; j += 64) {
          const float e = fast_exp2(sh[j] - m);
          sh[j] = e;
          l += e;
        }
        l = wave_sum(l);
        if (lane == 0) lh[h] = l;
      }
      __syncthreads();
      float acc[G][8];
      value_tile<E, G, PAGED, U>(a.kv, b, kvh, start, nrows, s, pitch, acc);
      __builtin_amdgcn_s_setprio(3);  // the merge chain issues ahead of streaming waves
      reduce_slots<G>(acc, red);
      float2 *mypart = reinterpret_cast<float2 *>(part_row + (int64_t)t * G * kHeadDim);
      for (int o2 = tid; o2 < G * kHeadDim / 2; o2 += kThreads) {
        float2 v = make_float2(0.0f, 0.0f);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          v.x += red[w * G * kHeadDim + 2 * o2];
          v.y += red[w * G * kHeadDim + 2 * o2 + 1];
        }
        st_coherent(mypart + o2, v);
      }
    }
    if (tid < G) st_coherent(a.stats + (row0 + tid) * T + t, make_float2(mh[tid], lh[tid]));

    // arrive; the last W arrivals merge one or more heads each
    const int W = PERSIST ? min(G, Tb) : 1;
    const int rank = row_arrive(sync, base, &rank_lds);
    if (rank < Tb - W) continue;
    if (rank == Tb - 1) {
      if (tid == 0)
        __hip_atomic_store(sync + 1, base + (unsigned long long)Tb, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    } else {
      row_wait(sync, base + (unsigned long long)Tb, a.err);
    }
    for (int h = rank - (Tb - W); h < G; h += W) {
      // a_t = exp2(m_t - m*) and the denominator sum_t a_t l_t
      float *al = red + kThreads;
      if (wave == 0) {
        const float2 *st = a.stats + (row0 + h) * T;
        float m = -kInf;
        for (int tt = lane; tt < Tb; tt += 64) m = fmaxf(m, ld_coherent(st + tt).x);
        m = wave_max(m);
        float d = 0.0f;
        for (int tt = lane; tt < Tb; tt += 64) {
          const float2 v = ld_coherent(st + tt);
          const float aa = fast_exp2(v.x - m);
          al[tt] = aa;
          d = fmaf(aa, v.y, d);
        }
        d = wave_sum(d);
        if (lane == 0) den = d;
      }
      __syncthreads();
      merge_head<E, G>(part_row, h, Tb, al, &den, 1.0f, red, out + (row0 + h) * kHeadDim);
    }
  }
}

// ---------------------------------------------------------------------------
// Large-batch sampled step: two launches
// ---------------------------------------------------------------------------
// Split outputs of the two-launch path, after the split's CDF P (pitch kSplitMax,
// nrows keys per head) and maxima mh are in LDS: the statistics (m_t, l_t =
// P_last), each key's CDF within its 32-key block as a 16-bit fraction of the
// block's mass (the stash) and the CDF at every block end.
template <int G>
__device__ __forceinline__ void write_split_stash(const FusedArgs &a, const float *P, const float *mh,
                                                  int nrows, int64_t row0, int t, int start) {
  constexpr int pitch = kSplitMax;
  const int tid = threadIdx.x, T = a.T;
  if (tid < G) a.stats[(row0 + tid) * T + t] = make_float2(mh[tid], P[tid * pitch + nrows - 1]);
  // stash: 8 keys per 16-byte store; key j of 32-key block k holds
  // round(65535 (P_j - P_{32k-1}) / (P_{block end} - P_{32k-1})) (P_{-1} = 0),
  // non-decreasing in j; every block is written whole, keys past the split
  // holding 65535 (the last split of a row ends within the row's stash pitch)
  const int q8 = ((nrows + kBlock - 1) / kBlock) * (kBlock / 8);
  for (int i = tid; i < G * q8; i += kThreads) {
    const int h = i / q8, j = 8 * (i - h * q8);
    const float *ph = P + h * pitch;
    const int k0 = j & ~(kBlock - 1);
    const float lo = k0 ? ph[k0 - 1] : 0.0f;
    const float hi = ph[min(k0 + kBlock - 1, nrows - 1)];
    const float sc = hi > lo ? 65535.0f / (hi - lo) : 0.0f;
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j0 = j + 2 * e, j1 = j0 + 1;
      const uint32_t q0 = j0 < nrows ? (uint32_t)fminf(fmaf(ph[j0] - lo, sc, 0.5f), 65535.0f) : 65535u;
      const uint32_t q1 = j1 < nrows ? (uint32_t)fminf(fmaf(ph[min(j1, nrows - 1)] - lo, sc, 0.5f), 65535.0f) : 65535u;
      w[e] = q0 | (q1 << 16);
    }
    // non-temporal: the stash is read once, by the value kernel
    const u32x4 sv = {w[0], w[1], w[2], w[3]};
    __builtin_nontemporal_store(sv, reinterpret_cast<u32x4 *>(a.qstash + (row0 + h) * a.npitch + start + j));
  }
  // block ends, in pairs (start / 32 is even); an odd last count also writes
  // the (unused) slot after the row's last block
  const int ncoarse = (int)(a.npitch / kBlock);
  const int nbh = ((nrows + kBlock - 1) / kBlock + 1) >> 1;
  for (int i = tid; i < G * nbh; i += kThreads) {
    const int h = i / nbh, k = 2 * (i - h * nbh);
    const float *ph = P + h * pitch;
    const f32x2 cv = {ph[min(k * kBlock + kBlock - 1, nrows - 1)],
                      ph[min(k * kBlock + 2 * kBlock - 1, nrows - 1)]};
    __builtin_nontemporal_store(cv, reinterpret_cast<f32x2 *>(a.coarse + (row0 + h) * ncoarse + start / kBlock + k));
  }
}

// Waves per SIMD of the key-stream kernels: many resident waves keep the
// stream's loads in flight (64 VGPRs for bf16 rows with G <= 4).
template <typename E, int G, bool PAGED>
constexpr int stream_waves() {
  return sizeof(E) == 2 && G <= 4 && !PAGED ? 8 : (G <= 4 ? 4 : 2);
}

// Split t of KV row rowkv (= b * Hkv + kvh): scores, CDF, then the stash, the
// block ends and the statistics.  Splits past the row's last (t >= Tb) write
// nothing.
template <typename E, int G, bool PAGED, bool APPEND = true>
__device__ __forceinline__ void stream_cdf_item(const FusedArgs &a, int rowkv, int t) {
  extern __shared__ __attribute__((aligned(16))) float dyn[];
  constexpr int pitch = kSplitMax;
  const int T = a.T;
  float *P = dyn;
  __shared__ float mh[G], mtmp[4 * G];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = rowkv / a.Hkv, kvh = rowkv % a.Hkv;
  const int64_t row0 = (int64_t)b * a.Hq + kvh * G;
  const int L = seq_len(a.kv, b);
  int Ls, Tb;
  split_geometry(L, T, Ls, Tb);
  if (t >= Tb) return;
  const int start = t * Ls, nrows = min(Ls, L - start);
  if constexpr (APPEND) append_current<E, PAGED>(a.kv, b, kvh, a.Hkv, start, nrows, L);

  const QRegs<E, G> qr = load_q<E, G>(static_cast<const E *>(a.q), b, a.Hq, kvh, tid & 15);
  float mx[G];
  // 4 rows per lane and batch: this kernel relies on many resident waves
  // (64 VGPRs) rather than on deep per-wave buffering
  score_tile<E, G, PAGED, 4>(a.kv, b, kvh, start, nrows, qr, a.scale_log2, P, pitch, mx);
  block_max_heads<G>(mx, mtmp, mh);
  for (int h = wave; h < G; h += kThreads / 64) wave_split_cdf_m(P + h * pitch, nrows, lane, mh[h]);
  __syncthreads();
  write_split_stash<G>(a, P, mh, nrows, row0, t, start);
}

// One work item per workgroup, items row-major; the hardware dispatcher
// balances them.  Writes the stash, the block ends and the statistics.
template <typename E, int G, bool PAGED, bool APPEND = false>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(stream_waves<E, G, PAGED>()))) void k_stream_cdf(FusedArgs a) {
  stream_cdf_item<E, G, PAGED, APPEND>(a, blockIdx.x / a.T, blockIdx.x % a.T);
}

// Query weights of one GQA group for the Bernoulli score stage (Sec. 5, Eq.
// "qk_estimator"; App. C, Eq. "mean_group_query"), one feature per thread of
// the first 128: pi_i = |q_i| / norm (mode 0, per head) or m_i / norm (mode
// 1, m_i the group's mean |q_i|), the stratified count c_i = #{n < B : (n +
// u_i)/B < pi_i} taken in float32, and w = sign(q_i) c_i norm / B (mode 0) or
// c_i (norm / B) q_{g,i} / m_i (mode 1).  Writes wl[g*128 + i], the list fl of
// features with a nonzero weight in some head (in feature order) and, if
// mask is not null, the group's feature mask.  Returns the list length
// (block-uniform).  Every thread of the workgroup calls it.
template <typename E, int G>
__device__ __forceinline__ int bern_group_weights(const E *__restrict__ q, int64_t row0, int64_t grp,
                                                  int Bd, int mode, const float *__restrict__ u_q,
                                                  float *wl, int *fl, uint8_t *mask) {
  __shared__ float tmp[4];
  __shared__ int wc[2];
  const int i = threadIdx.x, lane = i & 63, wave = i >> 6;
  const bool act = i < kHeadDim;
  auto max128 = [&](float v) -> float {  // max over the first 128 threads (values >= 0)
    v = wave_max(act ? v : 0.0f);
    if (lane == 0) tmp[wave] = v;
    __syncthreads();
    const float r = fmaxf(tmp[0], tmp[1]);
    __syncthreads();
    return r;
  };
  float qv[G];
#pragma unroll
  for (int g = 0; g < G; ++g) qv[g] = act ? to_f32(q[(row0 + g) * kHeadDim + i]) : 0.0f;
  float w[G];
  const float fB = (float)Bd;
  if (mode == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float norm = max128(fabsf(qv[g]));
      const float pi = norm > 0.0f ? fabsf(qv[g]) / norm : 0.0f;
      const float ug = act ? u_q[(row0 + g) * kHeadDim + i] : 1.0f;
      int cnt = 0;
      for (int n = 0; n < Bd; ++n) cnt += (((float)n + ug) / fB) < pi;
      const float sgn = qv[g] > 0.0f ? 1.0f : (qv[g] < 0.0f ? -1.0f : 0.0f);
      w[g] = sgn * (float)cnt * (norm / fB);
    }
  } else {
    float m = 0.0f;
#pragma unroll
    for (int g = 0; g < G; ++g) m += fabsf(qv[g]);
    m = m / (float)G;
    const float norm = max128(m);
    const float pi = norm > 0.0f ? m / norm : 0.0f;
    const float ug = act ? u_q[grp * kHeadDim + i] : 1.0f;
    int cnt = 0;
    for (int n = 0; n < Bd; ++n) cnt += (((float)n + ug) / fB) < pi;
    const float mhat = (float)cnt * (norm / fB);
#pragma unroll
    for (int g = 0; g < G; ++g) w[g] = m > 0.0f ? mhat * qv[g] / m : 0.0f;
  }
  bool keep = false;
#pragma unroll
  for (int g = 0; g < G; ++g) keep |= act && w[g] != 0.0f;
  if (act) {
#pragma unroll
    for (int g = 0; g < G; ++g) wl[g * kHeadDim + i] = w[g];
    if (mask) mask[grp * kHeadDim + i] = keep ? 1 : 0;
  }
  const uint64_t bm = __ballot(keep);
  if (lane == 0 && wave < 2) wc[wave] = __popcll(bm);
  __syncthreads();
  if (keep) fl[(wave ? wc[0] : 0) + __popcll(bm & ((1ull << lane) - 1ull))] = i;
  const int nf = wc[0] + wc[1];
  __syncthreads();
  return nf;
}

// Bernoulli score stage of the two-launch path (Sec. 5, Eq. "qk_estimator";
// App. C): every split computes its group's query weights, then s_j = scale *
// sum_{i in F} w_{h,i} K^T_{i,j} over the selected feature rows F of the
// feature-major cache only; then the split's CDF and the same stash, block
// ends and statistics as k_stream_cdf, so that k_value_heads finishes the
// step.  Thread (feature slot fs, key chunk kc) reads 8 consecutive keys of
// one feature row per 128-bit load, four features in flight; the slots'
// partial scores are added in slot order.  Split 0 writes the feature mask.
template <typename E, int G>
__global__ __launch_bounds__(kThreads) void k_bern_stream(FusedArgs a, KtView kt, int Bd, int mode,
                                                           const float *__restrict__ u_q,
                                                           uint8_t *__restrict__ mask_out) {
  extern __shared__ __attribute__((aligned(16))) float dyn[];
  constexpr int pitch = kSplitMax;
  float *P = dyn;  // [G][pitch] scores, then the split CDF
  __shared__ float wl[G * kHeadDim];
  __shared__ int fl[kHeadDim];
  __shared__ float mh[G];
  const int T = a.T, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rowkv = blockIdx.x / T, t = blockIdx.x % T;
  const int b = rowkv / a.Hkv, kvh = rowkv % a.Hkv;
  const int64_t row0 = (int64_t)b * a.Hq + kvh * G;
  const int L = seq_len(a.kv, b);
  int Ls, Tb;
  split_geometry(L, T, Ls, Tb);
  if (t >= max(Tb, 1)) return;
  const int nf = bern_group_weights<E, G>(static_cast<const E *>(a.q), row0, rowkv, Bd, mode, u_q,
                                          wl, fl, t == 0 ? mask_out : nullptr);
  if (t >= Tb) return;  // empty row: split 0 only wrote the mask
  const int start = t * Ls, nrows = min(Ls, L - start);

  const int nchunk = Ls >> 3, FS = kThreads / nchunk;
  const int kc = tid % nchunk, fs = tid / nchunk;
  const E *ktb = static_cast<const E *>(kt.kt) + (int64_t)b * kt.sb + (int64_t)kvh * kt.sh;
  const int p0 = start + kc * 8;
  const bool full = p0 + 8 <= L;
  float acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.0f;
  auto add = [&](const float (&kf)[8], int i) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float wv = wl[h * kHeadDim + i];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(wv, kf[e], acc[h][e]);
    }
  };
  if (fs < FS) {
    constexpr int UF = 4;
    int fi = fs;
    if (full) {
      for (; fi + (UF - 1) * FS < nf; fi += UF * FS) {
        Chunk<E> ch[UF];
#pragma unroll
        for (int u = 0; u < UF; ++u) ch[u] = Chunk<E>::load_nt(ktb + (int64_t)fl[fi + u * FS] * kt.sd + p0);
#pragma unroll
        for (int u = 0; u < UF; ++u) {
          float kf[8];
          ch[u].to_float(kf);
          add(kf, fl[fi + u * FS]);
        }
      }
    }
    for (; fi < nf; fi += FS) {
      const int i = fl[fi];
      const E *rp = ktb + (int64_t)i * kt.sd + p0;
      float kf[8];
      if (full) {
        Chunk<E>::load_nt(rp).to_float(kf);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) kf[e] = p0 + e < L ? to_f32(rp[e]) : 0.0f;
      }
      add(kf, i);
    }
  }
  // slot partials added in slot order: slot 0 stores, slots 1.. add in turn
  for (int r = 0; r < FS; ++r) {
    if (fs == r) {
#pragma unroll
      for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          float *d = P + h * pitch + kc * 8 + e;
          *d = r == 0 ? acc[h][e] : *d + acc[h][e];
        }
    }
    __syncthreads();
  }
  for (int o = tid; o < G * nrows; o += kThreads) {
    const int h = o / nrows, j = o - h * nrows;
    P[h * pitch + j] *= a.scale_log2;
  }
  __syncthreads();
  for (int h = wave; h < G; h += kThreads / 64) {
    const float m = wave_split_cdf(P + h * pitch, nrows, lane);
    if (lane == 0) mh[h] = m;
  }
  __syncthreads();
  write_split_stash<G>(a, P, mh, nrows, row0, t, start);
}

// Inverse CDF of one threshold (global units) for one query head: split
// t = #{t' in [1,Tb) : off[t'] <= tau}; inside it the key #{j : al_t P_j <=
// tau - off[t]} over the split's CDF, clamped to the split.  Two levels: the
// number kb of whole 32-key blocks below the threshold, from the block-end
// values cl[] in LDS (exact), then the count inside block kb from the 16-bit
// stash row Qst: the threshold's fraction f of the block's mass against each
// key's stored fraction.  The second level can differ from the exact count only
// where the threshold lies within 2^-17 of the block's mass of a key boundary.
// Returns the logical key position.
__device__ __forceinline__ int invert_threshold(const uint16_t *Qst, const float *cl,
                                                const float *off, const float *al, int Tb, int Ls,
                                                int L, float tau) {
  int t = 0;
  for (int step = 1 << (31 - __clz(Tb)); step > 0; step >>= 1) {
    const int nt = t + step;
    t = (nt < Tb && off[nt] <= tau) ? nt : t;
  }
  const float x = tau - off[t], a = al[t];
  const int st = t * Ls, nr = min(Ls, L - st);
  const int nb = (nr + kBlock - 1) / kBlock;
  const float *ce = cl + st / kBlock;
  int kb = 0;
#pragma unroll
  for (int step = kSplitMax / kBlock / 2; step > 0; step >>= 1) {
    const int nk = kb + step;
    kb = (nk <= nb && a * ce[nk - 1] <= x) ? nk : kb;
  }
  int pos;
  if (kb >= nb) {
    pos = nr;
  } else {
    const int j0 = kb * kBlock, nin = min(kBlock, nr - j0);
    const float alo = kb ? a * ce[kb - 1] : 0.0f, ahi = a * ce[kb];
    const float fq = (x - alo) / (ahi - alo) * 65535.0f;  // a*lo <= x < a*hi
    const uint4 *Qb = reinterpret_cast<const uint4 *>(Qst + st + j0);
    uint4 v[kBlock / 8];
#pragma unroll
    for (int i = 0; i < kBlock / 8; ++i) v[i] = Qb[i];
    int c = 0;
#pragma unroll
    for (int i = 0; i < kBlock / 8; ++i) {
      const uint32_t w[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        c += (float)(w[e] & 0xffffu) <= fq ? 1 : 0;
        c += (float)(w[e] >> 16) <= fq ? 1 : 0;
      }
    }
    // keys past the split hold 65535 and the block's last key is above the
    // threshold, so at most nin - 1 keys count
    pos = j0 + min(c, nin - 1);
  }
  return st + min(pos, nr - 1);
}

// One workgroup per query head.  Thresholds are taken kThreads at a time; the
// chosen keys of a chunk are non-decreasing, so equal keys form runs, and each
// run's V row is read once and added with its length: O = (1/S) sum_r
// V_{idx_r} (Sec. 2, the stochastic add-only attention).
// COHERENT: the statistics were published by other workgroups of the same
// launch and are read with coherent loads.
template <typename E, bool PAGED, int MODE, bool COHERENT>
__device__ __forceinline__ void value_head_item(const FusedArgs &a, int G, int64_t rowq) {
  constexpr bool STRAT = MODE == kStrat;
  extern __shared__ __attribute__((aligned(16))) float dyn[];
  __shared__ int wave_cnt[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, slot = tid >> 4, c = tid & 15;
  const int b = (int)(rowq / a.Hq), kvh = (int)(rowq % a.Hq) / G;
  E *out = static_cast<E *>(a.out) + rowq * kHeadDim;
  const int L = seq_len(a.kv, b);
  if (L <= 0) {
    if (tid < kHeadDim) store_out(out + tid, 0.0f);
    if (a.idx_out)
      for (int r = tid; r < a.S; r += kThreads) a.idx_out[rowq * a.S + r] = -1;
    return;
  }
  int Ls, Tb;
  split_geometry(L, a.T, Ls, Tb);
  const int ncoarse = (int)(a.npitch / kBlock);
  float *cl = dyn;                   // [ncoarse]
  float *off = cl + ncoarse;         // [T+1]
  float *al = off + (a.T + 1);       // [T]
  int *keys = reinterpret_cast<int *>(al + a.T);            // [kThreads]
  int *runs = keys + kThreads;                               // [kThreads]
  float *red = reinterpret_cast<float *>(runs + kThreads);  // [4][128]
  float *Tq = red + 4 * kHeadDim;                            // [S] i.i.d. thresholds
  {
    // the head's block ends, in pairs (ncoarse is even)
    const float2 *src = reinterpret_cast<const float2 *>(a.coarse + rowq * ncoarse);
    const int nc2 = ((L + kBlock - 1) / kBlock + 1) >> 1;
    for (int i = tid; i < nc2; i += kThreads) reinterpret_cast<float2 *>(cl)[i] = src[i];
  }
  if (wave == 0) head_offsets_wave<COHERENT>(a.stats + rowq * a.T, Tb, lane, off, al);
  if constexpr (MODE == kIid) {
    if (wave == 1) wave_iid_thresholds(a.u + rowq * (a.S + 1), a.S, Tq, lane);
  }
  __syncthreads();
  const float Z = off[Tb];
  const uint16_t *Qst = a.qstash + rowq * a.npitch;
  const E *V = static_cast<const E *>(a.kv.v);

  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.0f;
  const float u0 = MODE == kSys ? a.u[rowq] : 0.0f;
  for (int r0 = 0; r0 < a.S; r0 += kThreads) {
    const int n = min(kThreads, a.S - r0);
    const int r = r0 + tid;
    int key = 0;
    if (tid < n) {
      const float ur = STRAT ? a.u[rowq * a.S + r] : u0;
      const float tau = MODE == kIid ? Tq[r] * Z : threshold(r, ur, a.invS, Z);
      key = invert_threshold(Qst, cl, off, al, Tb, Ls, L, tau);
      keys[tid] = key;
      if (a.idx_out) a.idx_out[rowq * a.S + r] = key;
    }
    __syncthreads();
    // run starts in threshold order (ballot per wave, waves in order)
    const bool start = tid < n && (tid == 0 || keys[tid - 1] != key);
    const unsigned long long mask = __ballot(start);
    if (lane == 0) wave_cnt[wave] = __popcll(mask);
    __syncthreads();
    int before = 0;
    for (int w = 0; w < wave; ++w) before += wave_cnt[w];
    const int nruns = wave_cnt[0] + wave_cnt[1] + wave_cnt[2] + wave_cnt[3];
    if (start) runs[before + __popcll(mask & ((1ull << lane) - 1))] = tid;
    __syncthreads();
    // gather: 16 row slots, U rows in flight per slot
    constexpr int U = kGatherUnroll;
    for (int g0 = 0; g0 < nruns; g0 += 16 * U) {
      Chunk<E> ch[U];
      float w[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = g0 + u * 16 + slot;
        if (i < nruns) {
          const int j = runs[i];
          const int len = (i + 1 < nruns ? runs[i + 1] : n) - j;
          ch[u] = Chunk<E>::load(V + row_offset<PAGED>(a.kv, b, kvh, keys[j]) + c * 8);
          w[u] = (float)len;
        } else {
          ch[u] = Chunk<E>::zero();
          w[u] = 0.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float f[8];
        ch[u].to_float(f);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = fmaf(w[u], f[i], acc[i]);
      }
    }
    __syncthreads();  // keys / runs are rewritten by the next chunk
  }
  // sum the 16 slots (4 per wave, then the 4 waves in order), scale, store
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = xor32_sum(xor16_sum(acc[i]));
  if (lane < 16) {
#pragma unroll
    for (int i = 0; i < 8; ++i) red[wave * kHeadDim + c * 8 + i] = acc[i];
  }
  __syncthreads();
  if (tid < kHeadDim) {
    const float s = ((red[tid] + red[kHeadDim + tid]) + red[2 * kHeadDim + tid]) + red[3 * kHeadDim + tid];
    store_out(out + tid, s * a.invS);
  }
}

template <typename E, bool PAGED, int MODE>
__global__ __launch_bounds__(kThreads) void k_value_heads(FusedArgs a, int G) {
  value_head_item<E, PAGED, MODE, false>(a, G, blockIdx.x);
}

// Both stages of the two-launch path in one launch, as one work queue per XCD.
// Workgroup w serves queue x = w % 8, which holds the KV rows rho = x, x + 8,
// ...: first every split of those rows (the key stream, as k_stream_cdf), then
// one item per query head of those rows (the value stage, as k_value_heads).
// A workgroup takes the next ticket of its queue when it starts, so the value
// item of a head begins as soon as its row's splits have arrived, while other
// rows are still streaming, instead of after the whole grid.  A value item
// waits only for stream items of its own queue, every one of which was taken
// earlier by a running workgroup and waits for nothing, so the waits end.
// When the dispatcher places workgroup w on XCD w % 8, a row's writers and
// readers share one L2.  Counters: tickets[x] (the last taker of a queue
// clears it) and, per KV row, sync[4] (split arrivals) and sync[5] (value
// items done; the last one clears both), so every counter is zero between
// calls.  A wait that gives up sets the error flag; the workspace must then be
// cleared again (santa_workspace_init).  Opt-in (SANTA_QUEUE=1): at batch 16
// and 32k keys it measured 249 us against 205 us for the two launches, since
// a split may arrive only once its stash stores have completed, and under the
// full read stream that wait holds its workgroup slot; the two-launch kernel
// ends without it.
template <typename E, int G, bool PAGED, int MODE>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(stream_waves<E, G, PAGED>()))) void k_stream_value(FusedArgs a) {
  __shared__ int ticket;
  const int x = blockIdx.x & 7, nq = gridDim.x >> 3;
  const int rows = a.B * a.Hkv;
  const int nrx = (rows - x + 7) >> 3;  // rows of this queue
  if (threadIdx.x == 0) {
    const unsigned v = __hip_atomic_fetch_add(a.tickets + x, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((int)v == nq - 1) __hip_atomic_store(a.tickets + x, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    ticket = (int)v;
  }
  __syncthreads();
  const int w = ticket;
  const int ns = nrx * a.T;
  if (w < ns) {
    const int rowkv = x + 8 * (w / a.T);
    stream_cdf_item<E, G, PAGED>(a, rowkv, w % a.T);
    wait_stores();
    __syncthreads();
    if (threadIdx.x == 0)
      __hip_atomic_fetch_add(a.sync + (int64_t)rowkv * (kSyncStride / 2) + 4, 1ull, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
    return;
  }
  const int v = w - ns;
  if (v >= nrx * G) return;
  const int rowkv = x + 8 * (v / G), h = v % G;
  unsigned long long *cnt = a.sync + (int64_t)rowkv * (kSyncStride / 2) + 4;
  row_wait(cnt, (unsigned long long)a.T, a.err);
  const int b = rowkv / a.Hkv, kvh = rowkv % a.Hkv;
  value_head_item<E, PAGED, MODE, true>(a, G, (int64_t)b * a.Hq + kvh * G + h);
  if (threadIdx.x == 0) {
    const unsigned long long d = __hip_atomic_fetch_add(cnt + 1, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (d == (unsigned long long)(G - 1)) {
      __hip_atomic_store(cnt, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(cnt + 1, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
namespace {

struct OccKey {
  const void *fn;
  int dev;
  size_t lds;
};

// Co-resident workgroups of kernel fn on the current device (cached).
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

// Launch R*T workgroups with R whole rows per round, R limited so that every
// workgroup of the grid is resident at once: a waiting split only waits for
// splits of its own row, which the same round holds.
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
  a.tickets = reinterpret_cast<unsigned *>(ws + p.off_err + kTicketOffset);
  a.B = p.B;
  a.Hq = p.Hq;
  a.Hkv = p.Hkv;
  a.T = p.T;
  a.S = p.S;
  a.npitch = p.npitch;
  a.invS = p.S ? 1.0f / (float)p.S : 0.0f;
  a.scale_log2 = scale_log2;
  return a;
}

}  // namespace

hipError_t launch_fused_bernoulli(const Plan &p, const KvView &kv, const KtView &kt,
                                 const void *q, float scale_log2, int Bd, int mode,
                                 const float *u_q, const float *u, int32_t *idx_out,
                                 uint8_t *mask_out, void *out, char *ws, hipStream_t st) {
  FusedArgs args = make_args(p, kv, q, out, scale_log2, ws);
  args.u = u;
  args.idx_out = idx_out;
  const CallTimer tm = call_timer();
  return with_types(p, false, [&](auto eptr, auto gc, auto) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    constexpr int G = decltype(gc)::value;
    void *params1[] = {&args, const_cast<KtView *>(&kt), &Bd, &mode, &u_q, &mask_out};
    const size_t lds1 = (size_t)G * kSplitMax * 4;
    hipError_t e = hipExtLaunchKernel(reinterpret_cast<const void *>(&k_bern_stream<E, G>),
                                      dim3(p.B * p.Hkv * p.T), dim3(kThreads), params1, lds1, st,
                                      tm.start, nullptr, 0);
    if (e != hipSuccess) return e;
    int g = G;
    void *params2[] = {&args, &g};
    const size_t lds2 = (size_t)value_heads_floats(p.T, (int)(p.npitch / kBlock)) * 4;
    return hipExtLaunchKernel(reinterpret_cast<const void *>(&k_value_heads<E, false, kSys>),
                              dim3(p.B * p.Hq), dim3(kThreads), params2, lds2, st, nullptr, tm.stop,
                              0);
  });
}

hipError_t launch_fused_flash(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                              int tile_log2, int S_tile, const float *u, int32_t *idx_out,
                              void *out, char *ws, hipStream_t st) {
  FusedArgs args = make_args(p, kv, q, out, scale_log2, ws);
  args.u = u;
  args.idx_out = idx_out;
  args.tile_log2 = tile_log2;
  args.S_tile = S_tile;
  args.Tmax = (p.n_k + (1 << tile_log2) - 1) >> tile_log2;
  return with_types(p, kv.bt != nullptr, [&](auto eptr, auto gc, auto paged) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    constexpr int G = decltype(gc)::value;
    constexpr bool PG = decltype(paged)::value;
    const size_t lds = (size_t)fused_flash_floats(G, kSplitMax, p.T) * 4;
    const bool ap = kv.k_new != nullptr;
    const void *res = ap ? reinterpret_cast<const void *>(&k_fused_dense<E, G, PG, true, true, true>)
                         : reinterpret_cast<const void *>(&k_fused_dense<E, G, PG, true, true>);
    const int rows = p.B * p.Hkv;
    if (rows * p.T <= capacity_of(res, lds))  // one resident round
      return launch_resident(res, p, args, lds, st);
    void *params[] = {&args};
    const CallTimer tm = call_timer();
    return hipExtLaunchKernel(ap ? reinterpret_cast<const void *>(&k_fused_dense<E, G, PG, false, true, true>)
                                 : reinterpret_cast<const void *>(&k_fused_dense<E, G, PG, false, true>),
                              dim3(rows * p.T), dim3(kThreads), params, lds, st, tm.start, tm.stop,
                              0);
  });
}

hipError_t launch_fused_dense(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                              void *out, char *ws, hipStream_t st) {
  FusedArgs args = make_args(p, kv, q, out, scale_log2, ws);
  return with_types(p, kv.bt != nullptr, [&](auto eptr, auto gc, auto paged) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    constexpr int G = decltype(gc)::value;
    constexpr bool PG = decltype(paged)::value;
    const size_t lds = (size_t)fused_dense_floats(G, kSplitMax, p.T) * 4;
    const bool ap = kv.k_new != nullptr;
    const void *res = ap ? reinterpret_cast<const void *>(&k_fused_dense<E, G, PG, true, false, true>)
                         : reinterpret_cast<const void *>(&k_fused_dense<E, G, PG, true>);
    const int rows = p.B * p.Hkv;
    if (rows * p.T <= capacity_of(res, lds))  // one resident round
      return launch_resident(res, p, args, lds, st);
    void *params[] = {&args};
    const CallTimer tm = call_timer();
    return hipExtLaunchKernel(ap ? reinterpret_cast<const void *>(&k_fused_dense<E, G, PG, false, false, true>)
                                 : reinterpret_cast<const void *>(&k_fused_dense<E, G, PG, false>),
                              dim3(rows * p.T), dim3(kThreads), params, lds, st, tm.start, tm.stop,
                              0);
  });
}

hipError_t launch_fused_sampled(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                                int mode, const float *u, int32_t *idx_out, void *out, char *ws,
                                hipStream_t st) {
  FusedArgs args = make_args(p, kv, q, out, scale_log2, ws);
  args.u = u;
  args.idx_out = idx_out;
  return with_types(p, kv.bt != nullptr, [&](auto eptr, auto gc, auto paged) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    constexpr int G = decltype(gc)::value;
    constexpr bool PG = decltype(paged)::value;
    if (p.split2 && p.queue) {
      // both stages in one launch: per XCD queue, the splits of its rows, then
      // one item per query head of those rows
      const int rows = p.B * p.Hkv;
      const size_t lds1 = (size_t)G * kSplitMax * 4;
      const size_t lds2 = (size_t)(value_heads_floats(p.T, (int)(p.npitch / kBlock)) +
                                   (mode == kIid ? p.S : 0)) * 4;
      const int nq = ((rows + 7) / 8) * (p.T + G);
      const void *fn = mode == kStrat ? reinterpret_cast<const void *>(&k_stream_value<E, G, PG, kStrat>)
                       : mode == kIid ? reinterpret_cast<const void *>(&k_stream_value<E, G, PG, kIid>)
                                      : reinterpret_cast<const void *>(&k_stream_value<E, G, PG, kSys>);
      void *params[] = {&args};
      const CallTimer tm = call_timer();
      return hipExtLaunchKernel(fn, dim3(8 * nq), dim3(kThreads), params, std::max(lds1, lds2), st,
                                tm.start, tm.stop, 0);
    }
    if (p.split2) {
      const CallTimer tm = call_timer();
      void *params[] = {&args};
      const size_t lds1 = (size_t)G * kSplitMax * 4;
      hipError_t e = hipExtLaunchKernel(kv.k_new ? reinterpret_cast<const void *>(&k_stream_cdf<E, G, PG, true>)
                                                 : reinterpret_cast<const void *>(&k_stream_cdf<E, G, PG>),
                                        dim3(p.B * p.Hkv * p.T), dim3(kThreads), params, lds1, st,
                                        tm.start, nullptr, 0);
      if (e != hipSuccess) return e;
      int g = G;
      void *params2[] = {&args, &g};
      const size_t lds2 = (size_t)(value_heads_floats(p.T, (int)(p.npitch / kBlock)) +
                                   (mode == kIid ? p.S : 0)) * 4;
      const void *fn2 = mode == kStrat ? reinterpret_cast<const void *>(&k_value_heads<E, PG, kStrat>)
                        : mode == kIid ? reinterpret_cast<const void *>(&k_value_heads<E, PG, kIid>)
                                       : reinterpret_cast<const void *>(&k_value_heads<E, PG, kSys>);
      return hipExtLaunchKernel(fn2, dim3(p.B * p.Hq), dim3(kThreads), params2, lds2, st, nullptr,
                                tm.stop, 0);
    }
    const bool ap = kv.k_new != nullptr;
    const void *fn =
        mode == kStrat ? (ap ? reinterpret_cast<const void *>(&k_fused_sampled<E, G, PG, kStrat, true>)
                             : reinterpret_cast<const void *>(&k_fused_sampled<E, G, PG, kStrat>))
        : mode == kIid ? (ap ? reinterpret_cast<const void *>(&k_fused_sampled<E, G, PG, kIid, true>)
                             : reinterpret_cast<const void *>(&k_fused_sampled<E, G, PG, kIid>))
                       : (ap ? reinterpret_cast<const void *>(&k_fused_sampled<E, G, PG, kSys, true>)
                             : reinterpret_cast<const void *>(&k_fused_sampled<E, G, PG, kSys>));
    // stage the group's uniforms in LDS when they are few (the host keeps the
    // i.i.d. ones within the limit; their sorted thresholds follow them)
    const size_t nu = (size_t)G * (mode == kIid ? p.S + 1 : (mode == kStrat ? p.S : 1));
    args.ustage = nu <= (size_t)kUStageMax;
    const size_t staged = args.ustage ? nu + (mode == kIid ? (size_t)G * p.S : 0) : 0;
    const size_t lds = (size_t)fused_sampled_floats(G, kSplitMax, p.T, (int)staged) * 4;
    return launch_resident(fn, p, args, lds, st);
  });
}

}  // namespace santa
