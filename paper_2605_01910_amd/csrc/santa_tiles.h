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
// The G query rows of a KV group, 8 features per lane, in the query element
// type QE<E> (bfloat16 for an FP8 cache).
template <typename E, int G>
struct QRegs {
  Chunk<QE<E>> h[G];
  // Makes every register available (the compiler waits for their loads here).
  __device__ __forceinline__ void require() const {
#pragma unroll
    for (int i = 0; i < G; ++i) h[i].require();
  }
};

// Quarter k (lanes 4k..4k+3) of a 16-lane row: with G = 4 the query registers
// of a lane are stored with head h in slot h ^ gray(k), gray(k) = k ^ (k >> 1),
// so that the mirrored lanes of score_tile's reduce-scatter hold matching heads.
__device__ __forceinline__ int quarter_gray(int c) {
  const int k = (c >> 2) & 3;
  return k ^ (k >> 1);
}

template <typename E, int G>
__device__ __forceinline__ QRegs<E, G> load_q(const QE<E> *q, int b, int Hq, int kvh, int c) {
  QRegs<E, G> r;
  const int perm = G == 4 ? quarter_gray(c) : 0;
#pragma unroll
  for (int h = 0; h < G; ++h)
    r.h[h] = Chunk<QE<E>>::load(q + ((int64_t)b * Hq + kvh * G + (h ^ perm)) * kHeadDim + c * 8);
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

// Key rows per lane and batch of the score tile (U loads per lane in flight,
// twice that while a batch is scored): 8 for bf16 with G <= 4, 4 for the
// wider register sets of fp32 rows or G = 8; FP8 rows take half the bytes and
// registers per load, so twice as many for G <= 4 (G = 8 keeps 4: its query
// registers and the bf16 conversions leave no room for more).
template <typename E, int G>
constexpr int score_unroll() {
  return sizeof(E) == 1 ? (G <= 4 ? 16 : 4) : (sizeof(E) == 2 && G <= 4) ? 8 : 4;
}

// Block-table entries of the pages one split covers, one per lane: lane l of
// every wave holds the entry of page p0 + l.  They are loaded once per split,
// so the key stream does not wait on a table lookup every 16 rows.  A split
// of at most kSplitMax keys starting at a multiple of 16 spans at most 64
// pages when pages hold at least 16 keys (smaller pages are addressed per
// row and use no window).
struct PageWin {
  int p0, entry;
};

template <bool PAGED>
__device__ __forceinline__ PageWin page_window(const KvView &kv, int b, int start, int nrows) {
  PageWin w{0, 0};
  if constexpr (PAGED) {
    if (kv.ps_log2 >= 4 && nrows > 0) {
      const int lane = threadIdx.x & 63;
      w.p0 = start >> kv.ps_log2;
      const int np = ((start + nrows - 1) >> kv.ps_log2) - w.p0 + 1;
      w.entry = lane < np ? kv.bt[(int64_t)b * kv.max_pages + w.p0 + lane] : 0;
    }
  }
  return w;
}

// Byte offset, from the cache base, of key row row0 (feature 0) of sequence
// b, KV head kvh, for a row0 that is a multiple of 16 (one page-table entry
// per 16 rows when pages hold at least 16 keys, taken from the split's page
// window).  Uniform over the workgroup.
template <bool PAGED>
__device__ __forceinline__ int64_t row16_offset(const KvView &kv, const PageWin &pw, int b, int kvh,
                                                int row0) {
  if constexpr (PAGED) {
    const int page = __builtin_amdgcn_readlane(pw.entry, (row0 >> kv.ps_log2) - pw.p0);
    return (int64_t)page * kv.sb + (int64_t)(row0 & ((1 << kv.ps_log2) - 1)) * kv.sn +
           (int64_t)kvh * kv.sh;
  } else {
    return (int64_t)b * kv.sb + (int64_t)row0 * kv.sn + (int64_t)kvh * kv.sh;
  }
}

// 16 bytes at byte offset lb from p through a buffer resource (uniform base in
// scalar registers, one 32-bit lane offset; no range limit is used).  The load
// is non-temporal (cache-policy bit nt = 2): every key is read once per step,
// and marking the stream so keeps it from evicting the lines that are reused
// (the CDF stash, statistics, gathered value rows); measured, it also streams
// faster than the default policy.
__device__ __forceinline__ uint4 buffer_load16(const void *p, uint32_t lb) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, 0x7fffffff, 0x00020000);
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(rs, lb, 0, 2);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// 8 bytes at byte offset lb from p, as buffer_load16 (FP8 rows: 8 features).
__device__ __forceinline__ uint2 buffer_load8(const void *p, uint32_t lb) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, 0x7fffffff, 0x00020000);
  const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, lb, 0, 2);
  return make_uint2(v[0], v[1]);
}

// Features 8c..8c+7 of key row (row0 + slot); lb = (slot*stride_n + 8c) *
// sizeof(E) is the lane's byte offset (32 bits; the host bounds the stride).
template <typename E, bool PAGED>
__device__ __forceinline__ Chunk<E> load_key_row(const E *base, const KvView &kv, const PageWin &pw,
                                                 int b, int kvh, int row0, int slot, int c,
                                                 uint32_t lb) {
  if constexpr (PAGED) {
    if (kv.ps_log2 < 4) return Chunk<E>::load_nt(base + row_offset<true>(kv, b, kvh, row0 + slot) + c * 8);
  }
  const E *p = base + row16_offset<PAGED>(kv, pw, b, kvh, row0);
  if constexpr (sizeof(E) == 1) {
    return Chunk<E>{buffer_load8(p, lb)};
  } else if constexpr (sizeof(E) == 2) {
    return Chunk<E>{buffer_load16(p, lb)};
  } else {
    const uint4 x = buffer_load16(p, lb), y = buffer_load16(p, lb + 16);
    return Chunk<E>{make_float4(__uint_as_float(x.x), __uint_as_float(x.y), __uint_as_float(x.z),
                                __uint_as_float(x.w)),
                    make_float4(__uint_as_float(y.x), __uint_as_float(y.y), __uint_as_float(y.z),
                                __uint_as_float(y.w))};
  }
}

// Scores of key row j for the G heads from the lane's 8 features in ch (Sec.
// 2, SDPA equation, the q K^T product), written to s[h*pitch + j] and folded
// into the running maxima when valid.  G = 4: a reduce-scatter over the 16
// lanes (5 DPP adds instead of 16) leaves quarter k of the row with the full
// score of head gray(k), kept in m1; other G: full row sums, kept in mx[h].
template <typename E, int G>
__device__ __forceinline__ void score_key(const Chunk<E> &ch, const QRegs<E, G> &qr,
                                          float scale_log2, int c, int j, bool valid, float *s,
                                          int pitch, float &m1, float (&mx)[G]) {
  if constexpr (G == 4) {
    const float v0 = ch.dot(qr.h[0]), v1 = ch.dot(qr.h[1]);
    const float v2 = ch.dot(qr.h[2]), v3 = ch.dot(qr.h[3]);
    const float x0 = v0 + dpp<0x140>(v2);  // row_mirror
    const float x1 = v1 + dpp<0x140>(v3);
    float y = x0 + dpp<0x141>(x1);         // row_half_mirror
    y += dpp<0xB1>(y);
    y += dpp<0x4E>(y);
    y *= scale_log2;
    if (valid) {
      m1 = fmaxf(m1, y);
      if ((c & 3) == 0) s[quarter_gray(c) * pitch + j] = y;
    }
  } else {
    float acc[G];
#pragma unroll
    for (int h = 0; h < G; ++h) acc[h] = row16_sum(ch.dot(qr.h[h])) * scale_log2;
    if (valid) {
#pragma unroll
      for (int h = 0; h < G; ++h) mx[h] = fmaxf(mx[h], acc[h]);
      if (c == 0) {
#pragma unroll
        for (int h = 0; h < G; ++h) s[h * pitch + j] = acc[h];
      }
    }
  }
}

// Score tile (Sec. 2, SDPA equation, the q K^T product):
// s[h*pitch + j] = scale_log2 * <q_h, K_{start+j}> for j < nrows (start a
// multiple of 16).  Lane c of each 16-lane row holds features 8c..8c+7 of one
// key; a wave covers 4 keys per 128-bit load.  Whole batches of 16*U rows are
// loaded without predicates and double-buffered (the next batch's U loads per
// lane are in flight while this batch is scored); a ragged tail of fewer rows
// is loaded with per-row predicates.  mx[h] receives this lane's running max
// of head h's scores (G = 4: only the lane's own head, others -inf).
template <typename E, int G, bool PAGED, int U>
__device__ __forceinline__ void score_tile(const KvView &kv, int b, int kvh, int start, int nrows,
                                           const QRegs<E, G> &qr, float scale_log2, float *s,
                                           int pitch, float (&mx)[G]) {
  const int tid = threadIdx.x, slot = tid >> 4, c = tid & 15;
  const E *K = static_cast<const E *>(kv.k);
  const uint32_t lb = (uint32_t)(((int64_t)slot * kv.sn + c * 8) * (int64_t)sizeof(E));
  const PageWin pw = page_window<PAGED>(kv, b, start, nrows);
  float m1 = -kInf;
#pragma unroll
  for (int h = 0; h < G; ++h) mx[h] = -kInf;
  constexpr int RB = 16 * U;
  const int nfull = nrows - nrows % RB;
  auto load = [&](Chunk<E>(&ch)[U], int base) {
#pragma unroll
    for (int u = 0; u < U; ++u)
      ch[u] = load_key_row<E, PAGED>(K, kv, pw, b, kvh, start + base + u * 16, slot, c, lb);
  };
  auto score = [&](const Chunk<E>(&ch)[U], int base) {
#pragma unroll
    for (int u = 0; u < U; ++u)
      score_key<E, G>(ch[u], qr, scale_log2, c, base + u * 16 + slot, true, s, pitch, m1, mx);
  };
  // two buffers in a rolled loop whose loads are unconditional (so the
  // compiler's wait counts leave the other buffer's loads in flight), then at
  // most two more batches; four batch bodies of code in all
  Chunk<E> A[U], B[U];
  if (nfull > 0) load(A, 0);
  // the query registers are complete before the batches (their loads were
  // issued first), so the waits below count only key loads
  qr.require();
  int base = 0;
#pragma unroll 1
  for (; base + 2 * RB < nfull; base += 2 * RB) {
    load(B, base + RB);
    score(A, base);
    load(A, base + 2 * RB);
    score(B, base + RB);
  }
  if (nfull > 0) {
    const bool two = base + RB < nfull;
    if (two) load(B, base + RB);
    score(A, base);
    if (two) score(B, base + RB);
  }
  Chunk<E>(&cur)[U] = A;
  if (nfull < nrows) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = nfull + u * 16 + slot;
      cur[u] = j < nrows ? load_key_row<E, PAGED>(K, kv, pw, b, kvh, start + nfull + u * 16, slot, c, lb)
                         : Chunk<E>::zero();
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = nfull + u * 16 + slot;
      score_key<E, G>(cur[u], qr, scale_log2, c, j, j < nrows, s, pitch, m1, mx);
    }
  }
  if constexpr (G == 4) {
    const int hq = quarter_gray(c);
#pragma unroll
    for (int h = 0; h < G; ++h) mx[h] = h == hq ? m1 : -kInf;
  }
}

// Value tile of the exact decode (Sec. 2, SDPA equation, the weighted sum of
// V): acc[h][i] = sum_j w[h*pitch + j] * V_{start+j}[8c + i] over the rows j
// < nrows this lane's 16-lane row slot covers (weights in LDS; start a
// multiple of 16).  Same batching as score_tile: whole batches of 16*U rows
// without predicates, double-buffered; a ragged tail with per-row masks.
template <typename E, int G, bool PAGED, int U>
__device__ __forceinline__ void value_tile(const KvView &kv, int b, int kvh, int start, int nrows,
                                           const float *w, int pitch, float (&acc)[G][8]) {
  const int tid = threadIdx.x, slot = tid >> 4, c = tid & 15;
  const E *V = static_cast<const E *>(kv.v);
  const uint32_t lb = (uint32_t)(((int64_t)slot * kv.sn + c * 8) * (int64_t)sizeof(E));
  const PageWin pw = page_window<PAGED>(kv, b, start, nrows);
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[h][i] = 0.0f;
  constexpr int RB = 16 * U;
  const int nfull = nrows - nrows % RB;
  auto load = [&](Chunk<E>(&ch)[U], int base) {
#pragma unroll
    for (int u = 0; u < U; ++u)
      ch[u] = load_key_row<E, PAGED>(V, kv, pw, b, kvh, start + base + u * 16, slot, c, lb);
  };
  auto add = [&](const Chunk<E>(&ch)[U], int base) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = base + u * 16 + slot;
      float f[8];
      ch[u].to_float(f);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float wr = w[h * pitch + j];  // j < pitch: in bounds, stale past nrows
        const float wt = j < nrows ? wr : 0.0f;
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[h][i] = fmaf(wt, f[i], acc[h][i]);
      }
    }
  };
  Chunk<E> A[U], B[U];
  if (nfull > 0) load(A, 0);
  int base = 0;
#pragma unroll 1
  for (; base + 2 * RB < nfull; base += 2 * RB) {
    load(B, base + RB);
    add(A, base);
    load(A, base + 2 * RB);
    add(B, base + RB);
  }
  if (nfull > 0) {
    const bool two = base + RB < nfull;
    if (two) load(B, base + RB);
    add(A, base);
    if (two) add(B, base + RB);
  }
  Chunk<E>(&cur)[U] = A;
  if (nfull < nrows) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = nfull + u * 16 + slot;
      cur[u] = j < nrows ? load_key_row<E, PAGED>(V, kv, pw, b, kvh, start + nfull + u * 16, slot, c, lb)
                         : Chunk<E>::zero();
    }
    add(cur, nfull);
  }
}

// Split max of every head from the score tile's per-lane maxima (all threads
// get it in mh[h]); tmp holds 4*G floats.
template <int G>
__device__ __forceinline__ void block_max_heads(float (&mx)[G], float *tmp, float *mh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if constexpr (G == 4) {
    // score_tile leaves only the lane's own head finite: combine the 4 lanes
    // of a quarter, then the 4 rows of the wave (quarter k of every row holds
    // head gray(k))
    float m = fmaxf(fmaxf(mx[0], mx[1]), fmaxf(mx[2], mx[3]));
    m = fmaxf(m, dpp<0xB1>(m));
    m = fmaxf(m, dpp<0x4E>(m));
    m = xor32_max(xor16_max(m));
    if (lane < 16 && (lane & 3) == 0) tmp[wave * G + quarter_gray(lane)] = m;
  } else {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float m = wave_max(mx[h]);
      if (lane == 0) tmp[wave * G + h] = m;
    }
  }
  __syncthreads();
  if (tid < G) mh[tid] = fmaxf(fmaxf(tmp[tid], tmp[G + tid]), fmaxf(tmp[2 * G + tid], tmp[3 * G + tid]));
  __syncthreads();
}

// Split-local CDF of one head, computed by one wave (Sec. 2.1, "Construction":
// F is the running sum of the attention weights).  On return s[j] holds
// P_j = sum_{i<=j} exp2(s_i - m) for j < nrows (nrows <= kSplitMax; s has room
// for kSplitMax values).  Lane l owns keys 16l..16l+15 and sums them
// sequentially (four 16-byte LDS reads, no branches); the 64 run totals are
// joined by one wave prefix sum, made non-decreasing over the lanes by a prefix
// max, and every value of a run is capped at its lane's inclusive prefix, so P
// never decreases.  The summation order is fixed: equal inputs give
// bitwise-equal CDFs.
__device__ __forceinline__ void wave_split_cdf_m(float *s, int nrows, int lane, float m) {
  constexpr int CH = kSplitMax / 64;
  const int j0 = lane * CH;
  float x[CH];
#pragma unroll
  for (int i = 0; i < CH / 4; ++i) {
    const float4 v = reinterpret_cast<const float4 *>(s + j0)[i];
    x[4 * i] = v.x;
    x[4 * i + 1] = v.y;
    x[4 * i + 2] = v.z;
    x[4 * i + 3] = v.w;
  }
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const float e = fast_exp2(x[i] - m);
    acc += (j0 + i < nrows) ? e : 0.0f;  // keys past the split hold stale values
    x[i] = acc;
  }
  const float incl = wave_incl_max(wave_incl_scan(acc));
  const float base = wave_prev(0.0f, incl);
  if (j0 < nrows) {
#pragma unroll
    for (int i = 0; i < CH / 4; ++i)
      reinterpret_cast<float4 *>(s + j0)[i] =
          make_float4(fminf(base + x[4 * i], incl), fminf(base + x[4 * i + 1], incl),
                      fminf(base + x[4 * i + 2], incl), fminf(base + x[4 * i + 3], incl));
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

// Threshold r of a row in global CDF units, ((r + u_r)/S) Z (Sec. 2.1,
// "Construction"), kept strictly below Z.  In float32, r + u rounds up to
// r + 1 when u lies within half an ulp of 1 (u = 1 - 2^-24 with r >= 1), and
// (r + u) * fl(1/S) can round up to 1 when S is not a power of two; at r =
// S - 1 either would put the threshold at Z, past every key's CDF interval.
// The fraction is capped at the largest float below 1, whose product with a
// normal Z rounds below Z.  The cap keeps tau non-decreasing in r.
__device__ __forceinline__ float threshold(int r, float ur, float invS, float Z) {
  return fminf(((float)r + ur) * invS, 0x1.fffffep-1f) * Z;
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

// Fused current-token append (App. Decode-Step Kernel Microbenchmark Details,
// note on KV-cache appends: the decode step stores the new token's key and
// value before attending).  When kv.k_new is set, the workgroup whose split
// [start, start + nrows) holds position L - 1 copies the rows (b, kvh) of
// k_new / v_new ([B, Hkv, 128]) into the cache there and waits for the stores
// before it reads its split.  No other workgroup of the launch reads that row
// (every split reads and gathers only its own keys).  Called by every thread;
// the condition is uniform over the workgroup.
template <typename E, bool PAGED>
__device__ __forceinline__ void append_current(const KvView &kv, int b, int kvh, int Hkv, int start,
                                               int nrows, int L) {
  if (!kv.k_new || L - 1 < start || L - 1 >= start + nrows) return;
  constexpr int n16 = kHeadDim * (int)sizeof(E) / 16;  // 16-byte chunks per row
  const int tid = threadIdx.x;
  if (tid < 2 * n16) {
    const bool isv = tid >= n16;
    const int c = isv ? tid - n16 : tid;
    const uint4 *src = reinterpret_cast<const uint4 *>(static_cast<const E *>(isv ? kv.v_new : kv.k_new) +
                                                       ((int64_t)b * Hkv + kvh) * kHeadDim);
    E *dst = const_cast<E *>(static_cast<const E *>(isv ? kv.v : kv.k)) + row_offset<PAGED>(kv, b, kvh, L - 1);
    reinterpret_cast<uint4 *>(dst)[c] = src[c];
  }
  wait_stores();
  __syncthreads();
}

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

// Value stage of one split over a compacted union list (the group's chosen
// keys in key order, list[0..nlist)): each chosen V row is read once and
// added to every head with its count, O_h += c_{h,j} V_j (Sec. 2, Eq.
// "stochastic-add-only-attn").  The workgroup's 16 row slots share the list,
// U rows in flight each.  The G x 128 partial sums are written to part_out
// (global; coherent stores if COHERENT).  P is reused as the reduction
// buffer.  FW: cnt holds float weights (bit patterns) instead of integer counts.
template <typename E, int G, bool PAGED, bool COHERENT, bool FW = false, int U = 4>
__device__ __forceinline__ void gather_list(const KvView &kv, int b, int kvh, int start,
                                            const int *list, int nlist, float *P, int pitch,
                                            const int *cnt, float *__restrict__ part_out) {
  const int tid = threadIdx.x, slot = tid >> 4, c = tid & 15;
  // gather-add: slot takes list entries slot, slot+16, ...; U rows in flight
  const E *V = static_cast<const E *>(kv.v);
  float acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[h][i] = 0.0f;
  for (int e0 = slot; e0 < nlist; e0 += 16 * U) {
    Chunk<E> ch[U];
    int jj[U];
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
      const int e = e0 + uu * 16;
      jj[uu] = e < nlist ? list[e] : -1;
      ch[uu] = jj[uu] >= 0
                   ? Chunk<E>::load_nt(V + row_offset<PAGED>(kv, b, kvh, start + jj[uu]) + c * 8)
                   : Chunk<E>::zero();
    }
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
      if (jj[uu] < 0) continue;
      float f[8];
      ch[uu].to_float(f);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const int cw = cnt[h * pitch + jj[uu]];
        const float w = FW ? __int_as_float(cw) : (float)cw;
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

// Value stage of one split after the claims: the union over the group's heads
// of the chosen keys is compacted in key order, then gathered by gather_list.
template <typename E, int G, bool PAGED, bool COHERENT, bool FW = false, int U = 4>
__device__ __forceinline__ void gather_union(const KvView &kv, int b, int kvh, int start, int nrows,
                                             float *P, int pitch, const int *cnt, int *list,
                                             float *__restrict__ part_out) {
  const int nlist = compact_union<G>(cnt, pitch, nrows, list);
  gather_list<E, G, PAGED, COHERENT, FW, U>(kv, b, kvh, start, list, nlist, P, pitch, cnt, part_out);
}

}  // namespace santa
