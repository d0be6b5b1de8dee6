// santa_fused.h -- the default decode kernels: shared definitions.  The kernels
// themselves are in santa_sampled.h (one-launch sampled step), santa_stream.h
// (two-launch sampled step and Bernoulli scores) and santa_dense.h (dense and
// flash steps); each is instantiated once per element type by the
// santa_{sampled,stream,dense}_{bf16,f32}.hip units, and santa_launch.hip
// dispatches on the element type.
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
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>

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
  int B, Hq, Hkv, T, S;
  int ustage;     // the group's uniforms (G*S stratified, G systematic) staged in LDS if 1
  int64_t npitch; // stash floats per head row (n_k rounded up to 64)
  float invS, scale_log2;
  int tile_log2;  // flash: log2 of the tile length (16 .. kSplitMax keys)
  int S_tile;     // flash: samples per tile and head
  int Tmax;       // flash: tiles of the longest row, ceil(n_k / tile)
  int Ls;         // scheduled sampled path: keys per split of every row (multiple of 64)
  int direct;     // scheduled sampled path: every wave polls the row's statistics mailbox
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
// splits l*ch .. l*ch+ch-1 (ch <= kMaxSplits / 64), with (m_t, l_t) = ld(t).
template <typename LD>
__device__ __forceinline__ float head_offsets_from(LD ld, int Tb, int lane, float *off, float *al) {
  constexpr int CHM = kMaxSplits / 64;
  const int ch = (Tb + 63) >> 6;
  const int t0 = lane * ch;
  float2 sv[CHM];
#pragma unroll
  for (int i = 0; i < CHM; ++i)
    sv[i] = (i < ch && t0 + i < Tb) ? ld(t0 + i) : make_float2(-kInf, 0.0f);
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

// The same over statistics in global memory, st[t] = (m_t, l_t).
template <bool COHERENT>
__device__ __forceinline__ float head_offsets_wave(const float2 *st, int Tb, int lane, float *off,
                                                   float *al) {
  return head_offsets_from([&](int t) { return ld2<COHERENT>(st + t); }, Tb, lane, off, al);
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

// Merge of the four heads of a group (G = 4) by one workgroup, the row's last
// arrival: thread (h, c) sums columns 2c and 2c + 1 of head h over the row's Tb
// split partials in split order, O = (1/S) sum_t o_t (Sec. 3.1), with up to NB
// partials in flight per thread.
template <int NB = 32, typename OE>
__device__ __forceinline__ void merge_group4(const float *part_row, int Tb, float scale,
                                             OE *out_row0) {
  constexpr int G = 4;
  const int tid = threadIdx.x, h = tid >> 6, o = (tid & 63) * 2;
  const float2 *ph = reinterpret_cast<const float2 *>(part_row + h * kHeadDim + o);
  float sx = 0.0f, sy = 0.0f;
  for (int t0 = 0; t0 < Tb; t0 += NB) {
    float2 v[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i)
      v[i] = t0 + i < Tb ? ld_coherent(ph + (int64_t)(t0 + i) * (G * kHeadDim / 2))
                         : make_float2(0.0f, 0.0f);
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      sx += v[i].x;
      sy += v[i].y;
    }
  }
  store_out(out_row0 + h * kHeadDim + o, sx * scale);
  store_out(out_row0 + h * kHeadDim + o + 1, sy * scale);
}


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

// #{j < nrows : a P_j <= x} over a non-decreasing LDS CDF P (nrows <=
// kSplitMax = 1024) in three dependent steps instead of ten: the number of
// 256-key quarters whose last value is <= x (three reads), then the 16-key
// chunks of that quarter whose last value is <= x (16 reads issued together),
// then the keys of that chunk (four 16-byte reads).  Entries at or past nrows
// hold stale values and are never counted.
__device__ __forceinline__ int lds_cdf_count(const float *Ph, int nrows, float a, float x) {
  static_assert(kSplitMax == 1024, "three levels of 4 x 16 x 16 keys");
  // every read is inside the 1024-entry row, so the reads of a level are
  // unconditional and issued together; the tests use non-short-circuit '&'
  float w[16];
#pragma unroll
  for (int k = 1; k < 4; ++k) w[k] = Ph[256 * k - 1];
  int q = 0;
#pragma unroll
  for (int k = 1; k < 4; ++k) q += ((256 * k - 1 < nrows) & (a * w[k] <= x)) ? 1 : 0;
  const float *pq = Ph + 256 * q + 15;
#pragma unroll
  for (int i = 0; i < 16; ++i) w[i] = pq[16 * i];
  int c2 = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) c2 += ((256 * q + 16 * i + 15 < nrows) & (a * w[i] <= x)) ? 1 : 0;
  if (c2 == 16) return 256 * (q + 1);  // only when the quarter is the last: q = 3
  const int j0 = 256 * q + 16 * c2;
  const float4 *pc = reinterpret_cast<const float4 *>(Ph + j0);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float4 t = pc[i];
    w[4 * i] = t.x;
    w[4 * i + 1] = t.y;
    w[4 * i + 2] = t.z;
    w[4 * i + 3] = t.w;
  }
  int c3 = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) c3 += ((j0 + i < nrows) & (a * w[i] <= x)) ? 1 : 0;
  return j0 + c3;
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

// ---------------------------------------------------------------------------
// host side (santa_launch.hip)
// ---------------------------------------------------------------------------
// Co-resident workgroups of kernel fn on the current device (cached).
int capacity_of(const void *fn, size_t lds);

// Launch R*T workgroups with R whole rows per round, R limited so that every
// workgroup of the grid is resident at once: a waiting split only waits for
// splits of its own row, which the same round holds.
hipError_t launch_resident(const void *fn, const Plan &p, FusedArgs &args, size_t lds,
                           hipStream_t st);

FusedArgs make_args(const Plan &p, const KvView &kv, const void *q, void *out, float scale_log2,
                    char *ws);

// Launchers of one element type E (instantiated per type).
template <typename E>
hipError_t launch_one_launch_e(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                               int mode, const float *u, int32_t *idx_out, void *out, char *ws,
                               hipStream_t st);
template <typename E>
hipError_t launch_two_launch_e(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                               int mode, const float *u, int32_t *idx_out, void *out, char *ws,
                               hipStream_t st);
template <typename E>
hipError_t launch_rows_e(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                         int mode, const float *u, int32_t *idx_out, void *out, char *ws,
                         hipStream_t st);
template <typename E>
hipError_t launch_row_flash_e(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                              int tile_log2, int S_tile, const float *u, int32_t *idx_out,
                              void *out, char *ws, hipStream_t st);
template <typename E>
hipError_t launch_bernoulli_e(const Plan &p, const KvView &kv, const KtView &kt, const void *q,
                              float scale_log2, int Bd, int mode, const float *u_q, const float *u,
                              int32_t *idx_out, uint8_t *mask_out, void *out, char *ws,
                              hipStream_t st);
template <typename E>
hipError_t launch_dense_e(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                          void *out, char *ws, hipStream_t st);
template <typename E>
hipError_t launch_flash_e(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                          int tile_log2, int S_tile, const float *u, int32_t *idx_out, void *out,
                          char *ws, hipStream_t st);

// Compile-time dispatch over the GQA group size and the cache kind.
template <typename F>
inline hipError_t with_g_paged(int G, bool paged, F &&f) {
  return with_g(G, [&](auto gc) -> hipError_t {
    if (paged) return f(gc, std::true_type{});
    return f(gc, std::false_type{});
  });
}

}  // namespace santa
