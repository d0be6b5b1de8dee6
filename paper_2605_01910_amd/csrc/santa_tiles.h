// santa_tiles.h -- device building blocks shared by the multi-kernel and the
// fused decode kernels: query registers, the key-streaming score tile, the
// split-local CDF, slot reductions, thresholds and the inverse-CDF search.
#pragma once

#include <hip/hip_runtime.h>

#include "santa_device.h"

namespace santa {

// ---------------------------------------------------------------------------
// shared device pieces
// ---------------------------------------------------------------------------
template <typename E, int G>
struct QRegs {
  Chunk<E> h[G];
};

// Quarter k (lanes 4k..4k+3) of a 16-lane row: with G = 4 the query registers
// of a lane are stored with head h in slot h ^ gray(k), gray(k) = k ^ (k >> 1),
// so that the mirrored lanes of score_tile's reduce-scatter hold matching heads.
__device__ __forceinline__ int quarter_gray(int c) {
  const int k = (c >> 2) & 3;
  return k ^ (k >> 1);
}

template <typename E, int G>
__device__ __forceinline__ QRegs<E, G> load_q(const E *q, int b, int Hq, int kvh, int c) {
  QRegs<E, G> r;
  const int perm = G == 4 ? quarter_gray(c) : 0;
#pragma unroll
  for (int h = 0; h < G; ++h)
    r.h[h] = Chunk<E>::load(q + ((int64_t)b * Hq + kvh * G + (h ^ perm)) * kHeadDim + c * 8);
  return r;
}

__device__ __forceinline__ float to_f32(uint16_t x) { return __uint_as_float((uint32_t)x << 16); }
__device__ __forceinline__ float to_f32(float x) { return x; }

__device__ __forceinline__ void store_out(uint16_t *p, float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) {
    *p = 0x7fc0;  // NaN
    return;
  }
  u += 0x7fffu + ((u >> 16) & 1u);  // round to nearest even
  *p = (uint16_t)(u >> 16);
}
__device__ __forceinline__ void store_out(float *p, float x) { *p = x; }

// Keys in flight per lane in the score tile (U 128-bit loads per lane).
#ifndef SANTA_SCORE_UNROLL
#define SANTA_SCORE_UNROLL 8
#endif
constexpr int kScoreUnroll = SANTA_SCORE_UNROLL;

// Running (max, sum of exp2(s - max)) of a stream of scores: adds y with one
// exp2 (the smaller of the two terms is rescaled).
__device__ __forceinline__ void stat_push(float &m, float &l, float y) {
  const float d = y - m;  // +inf while the stream is empty (m = -inf)
  const float e = fast_exp2(-fabsf(d));
  l = d > 0.0f ? fmaf(l, e, 1.0f) : l + e;
  m = fmaxf(m, y);
}
// Combination of two partial (max, sum) pairs.
__device__ __forceinline__ void stat_merge(float &m, float &l, float m2, float l2) {
  const float M = fmaxf(m, m2);
  const float e1 = m == M ? 1.0f : fast_exp2(m - M);
  const float e2 = m2 == M ? 1.0f : fast_exp2(m2 - M);
  l = l * e1 + l2 * e2;
  m = M;
}

// Score tile (Sec. 2, SDPA equation, the q K^T product):
// s[h*pitch + j] = scale_log2 * <q_h, K_{start+j}> for j < nrows.
// Lane c of each 16-lane row holds features 8c..8c+7 of one key; a wave covers
// 4 keys per 128-bit load and U loads are in flight per lane.  mx[h] receives
// this lane's running max of head h's scores and, if STATS, ls[h] the running
// sum of exp2(s - mx[h]) (G = 4: only the lane's own head, others -inf / 0).
template <typename E, int G, bool PAGED, int U, bool STATS = false>
__device__ __forceinline__ void score_tile(const KvView &kv, int b, int kvh, int start, int nrows,
                                           const QRegs<E, G> &qr, float scale_log2, float *s,
                                           int pitch, float (&mx)[G], float (&ls)[G]) {
  const int tid = threadIdx.x, slot = tid >> 4, c = tid & 15;
  const E *K = static_cast<const E *>(kv.k);
  float m1 = -kInf, l1 = 0.0f;  // G == 4: the lane's own head
#pragma unroll
  for (int h = 0; h < G; ++h) {
    mx[h] = -kInf;
    ls[h] = 0.0f;
  }
  for (int base = 0; base < nrows; base += 16 * U) {
    Chunk<E> ch[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = base + u * 16 + slot;
      ch[u] = j < nrows ? Chunk<E>::load(K + row_offset<PAGED>(kv, b, kvh, start + j) + c * 8)
                        : Chunk<E>::zero();
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = base + u * 16 + slot;
      if constexpr (G == 4) {
        // reduce-scatter over the 16 lanes: 5 DPP adds instead of 16; quarter k
        // ends with the full score of head gray(k)
        const float v0 = ch[u].dot(qr.h[0]), v1 = ch[u].dot(qr.h[1]);
        const float v2 = ch[u].dot(qr.h[2]), v3 = ch[u].dot(qr.h[3]);
        const float x0 = v0 + dpp<0x140>(v2);   // row_mirror
        const float x1 = v1 + dpp<0x140>(v3);
        float y = x0 + dpp<0x141>(x1);          // row_half_mirror
        y += dpp<0xB1>(y);
        y += dpp<0x4E>(y);
        y *= scale_log2;
        if (j < nrows) {
          if (STATS) stat_push(m1, l1, y);
          else m1 = fmaxf(m1, y);
          if ((c & 3) == 0) s[quarter_gray(c) * pitch + j] = y;
        }
      } else {
        float acc[G];
#pragma unroll
        for (int h = 0; h < G; ++h) acc[h] = row16_sum(ch[u].dot(qr.h[h])) * scale_log2;
        if (j < nrows) {
#pragma unroll
          for (int h = 0; h < G; ++h) {
            if (STATS) stat_push(mx[h], ls[h], acc[h]);
            else mx[h] = fmaxf(mx[h], acc[h]);
          }
          if (c == 0) {
#pragma unroll
            for (int h = 0; h < G; ++h) s[h * pitch + j] = acc[h];
          }
        }
      }
    }
  }
  if constexpr (G == 4) {
    const int hq = quarter_gray(c);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      mx[h] = h == hq ? m1 : -kInf;
      ls[h] = h == hq ? l1 : 0.0f;
    }
  }
}

// Without the running sums.
template <typename E, int G, bool PAGED, int U>
__device__ __forceinline__ void score_tile(const KvView &kv, int b, int kvh, int start, int nrows,
                                           const QRegs<E, G> &qr, float scale_log2, float *s,
                                           int pitch, float (&mx)[G]) {
  float ls[G];
  score_tile<E, G, PAGED, U, false>(kv, b, kvh, start, nrows, qr, scale_log2, s, pitch, mx, ls);
}

// Split (max, sum of exp2(s - max)) of every head from the score tile's
// per-lane running pairs (all threads get them in mh[h], lh[h]); tmp holds
// 8*G floats.
template <int G>
__device__ __forceinline__ void block_stats_heads(float (&mx)[G], float (&ls)[G], float *tmp,
                                                  float *mh, float *lh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if constexpr (G == 4) {
    // the four lanes of a quarter hold the same pair; combine the 4 rows
    const int hq = quarter_gray(lane & 15);
    float m = mx[0], l = ls[0];
#pragma unroll
    for (int h = 1; h < G; ++h) {
      m = h == hq ? mx[h] : m;
      l = h == hq ? ls[h] : l;
    }
    {
      const auto pm = __builtin_amdgcn_permlane16_swap(__float_as_uint(m), __float_as_uint(m), false, false);
      const auto pl = __builtin_amdgcn_permlane16_swap(__float_as_uint(l), __float_as_uint(l), false, false);
      m = __uint_as_float(pm[0]); l = __uint_as_float(pl[0]);
      stat_merge(m, l, __uint_as_float(pm[1]), __uint_as_float(pl[1]));
    }
    {
      const auto pm = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
      const auto pl = __builtin_amdgcn_permlane32_swap(__float_as_uint(l), __float_as_uint(l), false, false);
      m = __uint_as_float(pm[0]); l = __uint_as_float(pl[0]);
      stat_merge(m, l, __uint_as_float(pm[1]), __uint_as_float(pl[1]));
    }
    if (lane < 16 && (lane & 3) == 0) {
      tmp[(wave * G + hq) * 2] = m;
      tmp[(wave * G + hq) * 2 + 1] = l;
    }
  } else {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      // lanes of a 16-lane row hold the same pair; combine the 4 rows
      float m = mx[h], l = ls[h];
      {
        const auto pm = __builtin_amdgcn_permlane16_swap(__float_as_uint(m), __float_as_uint(m), false, false);
        const auto pl = __builtin_amdgcn_permlane16_swap(__float_as_uint(l), __float_as_uint(l), false, false);
        m = __uint_as_float(pm[0]); l = __uint_as_float(pl[0]);
        stat_merge(m, l, __uint_as_float(pm[1]), __uint_as_float(pl[1]));
      }
      {
        const auto pm = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
        const auto pl = __builtin_amdgcn_permlane32_swap(__float_as_uint(l), __float_as_uint(l), false, false);
        m = __uint_as_float(pm[0]); l = __uint_as_float(pl[0]);
        stat_merge(m, l, __uint_as_float(pm[1]), __uint_as_float(pl[1]));
      }
      if (lane == 0) {
        tmp[(wave * G + h) * 2] = m;
        tmp[(wave * G + h) * 2 + 1] = l;
      }
    }
  }
  __syncthreads();
  if (tid < G) {
    float m = tmp[tid * 2], l = tmp[tid * 2 + 1];
#pragma unroll
    for (int w = 1; w < 4; ++w) stat_merge(m, l, tmp[(w * G + tid) * 2], tmp[(w * G + tid) * 2 + 1]);
    mh[tid] = m;
    lh[tid] = l;
  }
  __syncthreads();
}

// Split max of every head from the score tile's per-lane maxima (all threads
// get it in mh[h]); tmp holds 4*G floats.
template <int G>
__device__ __forceinline__ void block_max_heads(float (&mx)[G], float *tmp, float *mh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float m = wave_max(mx[h]);
    if (lane == 0) tmp[wave * G + h] = m;
  }
  __syncthreads();
  if (tid < G) mh[tid] = fmaxf(fmaxf(tmp[tid], tmp[G + tid]), fmaxf(tmp[2 * G + tid], tmp[3 * G + tid]));
  __syncthreads();
}

// Split-local CDF of one head, computed by one wave (Sec. 2.1, "Construction":
// F is the running sum of the attention weights).  On return s[j] holds
// P_j = sum_{i<=j} exp2(s_i - m) for j < nrows, where m = max_j s_j is returned.
// Each lane owns a contiguous run of keys and sums it sequentially; the runs are
// joined by a wave prefix sum.
__device__ __forceinline__ void wave_split_cdf_m(float *s, int nrows, int lane, float m) {
  // rows of 64 keys: lane l holds key 64*i + l of row i; each row is a DPP
  // prefix sum, offset by the previous row's last value (carried exactly, so
  // the CDF never decreases from one row to the next)
  float carry = 0.0f;
  for (int j0 = 0; j0 < nrows; j0 += 64) {
    const int j = j0 + lane;
    const float x = s[min(j, nrows - 1)];
    const float e = j < nrows ? fast_exp2(x - m) : 0.0f;
    const float p = carry + wave_incl_scan(e);
    if (j < nrows) s[j] = p;
    carry = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p), 63));
  }
}

__device__ __forceinline__ float wave_split_cdf(float *s, int nrows, int lane) {
  float m = -kInf;
  for (int j = lane; j < nrows; j += 64) m = fmaxf(m, s[j]);
  m = wave_max(m);
  wave_split_cdf_m(s, nrows, lane, m);
  return m;
}

// After the split's scores are in s[]: build each head's split CDF and write
// the split statistics (m_t, l_t = P_last) and the CDF stash.
template <int G>
__device__ __forceinline__ void finish_split_cdf(float *s, float *mh, int nrows, int64_t row0,
                                                 int T, int t, int64_t stash_pitch, int start,
                                                 float2 *stats, float *stash) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int h = wave; h < G; h += kThreads / 64) {
    const float m = wave_split_cdf(s + h * kSplitMax, nrows, lane);
    if (lane == 0) mh[h] = m;
  }
  __syncthreads();
  if (tid < G) stats[(row0 + tid) * T + t] = make_float2(mh[tid], s[tid * kSplitMax + nrows - 1]);
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float *dst = stash + (row0 + h) * stash_pitch + start;
    for (int j = tid; j < nrows; j += kThreads) dst[j] = s[h * kSplitMax + j];
  }
}

// Sum of acc[G][8] over the 16 row slots of the workgroup (4 per wave, 4 waves)
// into red[G*128] (fixed order); thread tid then owns outputs tid, tid+256, ...
template <int G>
__device__ __forceinline__ void reduce_slots(float (&acc)[G][8], float *red /* [4][G*128] */) {
  const int tid = threadIdx.x, wave = tid >> 6, c = tid & 15;
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[h][i] = xor32_sum(xor16_sum(acc[h][i]));
  if ((tid & 63) < 16) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int i = 0; i < 8; ++i) red[wave * G * kHeadDim + h * kHeadDim + c * 8 + i] = acc[h][i];
  }
  __syncthreads();
}

__device__ __forceinline__ float threshold(int r, float ur, float invS, float Z) {
  return ((float)r + ur) * invS * Z;
}

// Number of j < n with a * P[j] <= x (P non-decreasing): branch-free binary lifting.
__device__ __forceinline__ int cdf_count(const float *P, int n, float a, float x) {
  int pos = 0;
#pragma unroll
  for (int step = kSplitMax; step > 0; step >>= 1) {
    const int np = pos + step;
    if (np <= n && a * P[np - 1] <= x) pos = np;
  }
  return pos;
}


// ---------------------------------------------------------------------------
// Cross-workgroup data exchange without cache-wide maintenance: every shared
// word is written and read with relaxed agent-scope atomics (coherent per
// access), and a writer waits for its stores to complete before it signals.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void st_coherent(float2 *p, float2 v) {
  __hip_atomic_store(reinterpret_cast<unsigned long long *>(p),
                     __builtin_bit_cast(unsigned long long, v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_coherent(const float2 *p) {
  return __builtin_bit_cast(
      float2, __hip_atomic_load(reinterpret_cast<unsigned long long *>(const_cast<float2 *>(p)),
                                __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}
__device__ __forceinline__ float ld_coherent(const float *p) {
  return __hip_atomic_load(const_cast<float *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coherent(int *p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int ld_coherent(const int *p) {
  return __hip_atomic_load(const_cast<int *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Wait until this wave's outstanding memory operations have completed; also a
// compiler barrier for memory accesses.
__device__ __forceinline__ void wait_stores() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Per-split claim state of one head: the split owns thresholds tau with
// lo <= tau < hi (global CDF units); a is exp2(m_t - m*), Z the row total.
struct HeadClaim {
  float lo, hi, Z, a;
};

// 1 if any threshold of any head falls in this split (block-uniform result).
template <int G, bool STRAT>
__device__ __forceinline__ bool any_claims(const HeadClaim *hc, int64_t row0, int S, float invS,
                                           const float *__restrict__ u) {
  const int tid = threadIdx.x;
  int any = 0;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const HeadClaim c = hc[h];
    const float *uh = STRAT ? u + (row0 + h) * S : u + (row0 + h);
    for (int r = tid; r < S; r += kThreads) {
      const float tau = threshold(r, STRAT ? uh[r] : uh[0], invS, c.Z);
      any |= (tau >= c.lo) & (tau < c.hi);
    }
  }
  return __syncthreads_or(any) != 0;
}

// Claims and inverse-CDF search of one split whose CDF P[h*pitch + j]
// (j < nrows) is in LDS and whose sample counts cnt[h*pitch + j] are zero.
// Threshold m of head h is tau = ((m + u)/S) Z (systematic: u = us[h*ustride];
// stratified: u = us[h*ustride + m]); the split owns lo <= tau < hi and maps
// tau to the key #{j : a P_j <= tau - lo} (the CDF interval containing it,
// App. A), clamped to the split.  Counts go to LDS, indices to idx_out.
// Returns (block-uniform) whether any threshold fell in this split.
template <int G, bool STRAT>
__device__ __forceinline__ bool claim_search(int start, int nrows, int64_t row0, int S, float invS,
                                             const float *us, int64_t ustride, const HeadClaim *hc,
                                             const float *P, int pitch, int *cnt,
                                             int32_t *__restrict__ idx_out) {
  const int tid = threadIdx.x;
  HeadClaim cl[G];
#pragma unroll
  for (int h = 0; h < G; ++h) cl[h] = hc[h];
  const int step0 = 1 << (31 - __clz(nrows));
  int any = 0;
  for (int r = tid; r < S; r += kThreads) {
    float x[G];
    bool in[G];
    int pos[G];
    bool anyin = false;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float ur = STRAT ? us[h * ustride + r] : us[h * ustride];
      const float tau = threshold(r, ur, invS, cl[h].Z);
      in[h] = (tau >= cl[h].lo) & (tau < cl[h].hi);
      x[h] = tau - cl[h].lo;
      pos[h] = 0;
      anyin |= in[h];
    }
    if (!anyin) continue;
    // the G searches advance together: all reads of a step are issued before
    // any is used, and the step is a select (no branch)
    for (int step = step0; step > 0; step >>= 1) {
      float v[G];
#pragma unroll
      for (int h = 0; h < G; ++h) v[h] = P[h * pitch + min(pos[h] + step, nrows) - 1];
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const int np = pos[h] + step;
        const bool ok = (np <= nrows) & (cl[h].a * v[h] <= x[h]);
        pos[h] = ok ? np : pos[h];
      }
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
      if (in[h]) {
        const int j = pos[h] < nrows ? pos[h] : nrows - 1;
        atomicAdd(&cnt[h * pitch + j], 1);
        if (idx_out) idx_out[(row0 + h) * S + r] = start + j;
      }
    }
    any = 1;
  }
  return __syncthreads_or(any) != 0;
}

// Union over the group's heads of the keys with a nonzero count (cnt[h*pitch
// + j], j < nrows), compacted in key order into list[]; returns its length
// (block-uniform).  One ballot mask per 64 keys, then an exclusive prefix.
template <int G>
__device__ __forceinline__ int compact_union(const int *cnt, int pitch, int nrows, int *list) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ unsigned long long masks[kSplitMax / 64];
  const int nch = (nrows + 63) >> 6;
  for (int ch = wave; ch < nch; ch += kThreads / 64) {
    const int j = ch * 64 + lane;
    const int jc = min(j, nrows - 1);
    bool need = false;
#pragma unroll
    for (int h = 0; h < G; ++h) need |= cnt[h * pitch + jc] != 0;
    const unsigned long long m = __ballot(need && j < nrows);
    if (lane == 0) masks[ch] = m;
  }
  __syncthreads();
  // lane i < nch holds the popcount of mask i; an exclusive prefix gives offsets
  const unsigned long long mine = lane < nch ? masks[lane] : 0ull;
  const float inc = wave_incl_scan((float)__popcll(mine));  // exact: counts <= kSplitMax
  const int excl = (int)wave_prev(0.0f, inc);
  const int nlist = (int)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(inc), 63));
  for (int ch = wave; ch < nch; ch += kThreads / 64) {
    const unsigned long long m = masks[ch];
    const int off = __builtin_amdgcn_readlane(excl, ch);
    if ((m >> lane) & 1ull) list[off + __popcll(m & ((1ull << lane) - 1ull))] = ch * 64 + lane;
  }
  __syncthreads();
  return nlist;
}

// Value stage of one split after claim_search: the union over the group's
// heads of the chosen keys is compacted in key order and each chosen V row is
// read once: O_h += c_{h,j} V_j (Sec. 2, Eq. "stochastic-add-only-attn").  The
// G x 128 partial sums are written to part_out (global; coherent stores if
// COHERENT).  P is reused as the reduction buffer.
template <typename E, int G, bool PAGED, bool COHERENT>
__device__ __forceinline__ void gather_union(const KvView &kv, int b, int kvh, int start, int nrows,
                                             float *P, int pitch, const int *cnt, int *list,
                                             int *wave_cnt, float *__restrict__ part_out) {
  const int tid = threadIdx.x, slot = tid >> 4, c = tid & 15;
  (void)wave_cnt;
  const int nlist = compact_union<G>(cnt, pitch, nrows, list);
  // gather-add: slot takes list entries slot, slot+16, ...; 4 rows in flight
  const E *V = static_cast<const E *>(kv.v);
  float acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[h][i] = 0.0f;
  constexpr int U = 4;
  for (int e0 = slot; e0 < nlist; e0 += 16 * U) {
    Chunk<E> ch[U];
    int jj[U];
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
      const int e = e0 + uu * 16;
      jj[uu] = e < nlist ? list[e] : -1;
      ch[uu] = jj[uu] >= 0
                   ? Chunk<E>::load(V + row_offset<PAGED>(kv, b, kvh, start + jj[uu]) + c * 8)
                   : Chunk<E>::zero();
    }
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
      if (jj[uu] < 0) continue;
      float f[8];
      ch[uu].to_float(f);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float w = (float)cnt[h * pitch + jj[uu]];
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[h][i] = fmaf(w, f[i], acc[h][i]);
      }
    }
  }
  reduce_slots<G>(acc, P);
  for (int o2 = tid; o2 < G * kHeadDim / 2; o2 += kThreads) {
    float2 v = make_float2(0.0f, 0.0f);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      v.x += P[w * G * kHeadDim + 2 * o2];
      v.y += P[w * G * kHeadDim + 2 * o2 + 1];
    }
    if (COHERENT)
      st_coherent(reinterpret_cast<float2 *>(part_out) + o2, v);
    else
      reinterpret_cast<float2 *>(part_out)[o2] = v;
  }
}

}  // namespace santa
