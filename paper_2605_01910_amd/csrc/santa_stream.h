// santa_stream.h -- the two-launch sampled step (k_stream_cdf, then
// k_value_heads one workgroup per query head) and the Bernoulli score stage
// (k_bern_stream) that feeds the same value kernel (see santa_fused.h).
#pragma once

#include "santa_fused.h"

namespace santa {

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
  if constexpr (sizeof(E) == 1) return G <= 4 ? 5 : 2;  // 8 FP8 rows per lane and batch
  return sizeof(E) == 2 && G <= 4 && !PAGED ? 8 : (G <= 4 ? 4 : 2);
}

// Split t of KV row rowkv (= b * Hkv + kvh): scores, CDF, then the stash, the
// block ends and the statistics.  Splits past the row's last (t >= Tb) write
// nothing.
template <typename E, int G, bool PAGED, bool APPEND>
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

  const QRegs<E, G> qr = load_q<E, G>(static_cast<const QE<E> *>(a.q), b, a.Hq, kvh, tid & 15);
  const float ksc = kv_scales<E>(a.kv, b, kvh, a.Hkv).x;  // FP8 cache: K scale
  float mx[G];
  // 4 rows per lane and batch: this kernel relies on many resident waves
  // (64 VGPRs) rather than on deep per-wave buffering
  score_tile<E, G, PAGED, sizeof(E) == 1 ? 8 : 4>(a.kv, b, kvh, start, nrows, qr, a.scale_log2 * ksc,
                                                  P, pitch, mx);
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
  __shared__ float tmp[2 * G];
  __shared__ int wc[2];
  const int i = threadIdx.x, lane = i & 63, wave = i >> 6;
  const bool act = i < kHeadDim;
  // the query and the Bernoulli uniforms are loaded together, up front
  float qv[G], uq[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    qv[g] = act ? to_f32(q[(row0 + g) * kHeadDim + i]) : 0.0f;
    uq[g] = !act ? 1.0f : mode == 0 ? u_q[(row0 + g) * kHeadDim + i]
                                    : (g == 0 ? u_q[grp * kHeadDim + i] : 1.0f);
  }
  float w[G];
  const float fB = (float)Bd;
  if (mode == 0) {
    // the G norms max_i |q_{g,i}| at once: one exchange of the two waves' maxima
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float v = wave_max(fabsf(qv[g]));
      if (lane == 0 && wave < 2) tmp[2 * g + wave] = v;
    }
    __syncthreads();
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float norm = fmaxf(tmp[2 * g], tmp[2 * g + 1]);
      const float pi = norm > 0.0f ? fabsf(qv[g]) / norm : 0.0f;
      const float ug = uq[g];
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
    const float wm = wave_max(m);
    if (lane == 0 && wave < 2) tmp[wave] = wm;
    __syncthreads();
    const float norm = fmaxf(tmp[0], tmp[1]);
    const float pi = norm > 0.0f ? m / norm : 0.0f;
    const float ug = uq[0];
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
  // slot partials in a fixed order: with room for two copies of the split
  // (2 Ls <= kSplitMax), even slots accumulate in the first copy and odd
  // slots in the second, FS/2 rounds, and the scale pass adds the two copies;
  // otherwise slot 0 stores and slots 1.. add in turn
  const bool two = 2 * Ls <= pitch && (FS & 1) == 0;
  const int nr = two ? FS / 2 : FS;
  for (int r = 0; r < nr; ++r) {
    if ((two ? fs >> 1 : fs) == r) {
      float *d0 = P + (two ? (fs & 1) * Ls : 0) + kc * 8;
#pragma unroll
      for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          float *d = d0 + h * pitch + e;
          *d = r == 0 ? acc[h][e] : *d + acc[h][e];
        }
    }
    __syncthreads();
  }
  for (int o = tid; o < G * nrows; o += kThreads) {
    const int h = o / nrows, j = o - h * nrows;
    float *d = P + h * pitch + j;
    *d = (two ? *d + d[Ls] : *d) * a.scale_log2;
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
template <typename E, bool PAGED, int MODE>
__device__ __forceinline__ void value_head_item(const FusedArgs &a, int G, int64_t rowq) {
  constexpr bool STRAT = MODE == kStrat;
  extern __shared__ __attribute__((aligned(16))) float dyn[];
  __shared__ int wave_cnt[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, slot = tid >> 4, c = tid & 15;
  const int b = (int)(rowq / a.Hq), kvh = (int)(rowq % a.Hq) / G;
  QE<E> *out = static_cast<QE<E> *>(a.out) + rowq * kHeadDim;
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
  if (wave == 0) head_offsets_wave<false>(a.stats + rowq * a.T, Tb, lane, off, al);
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
    store_out(out + tid, s * (a.invS * kv_scales<E>(a.kv, b, kvh, a.Hkv).y));
  }
}

template <typename E, bool PAGED, int MODE>
__global__ __launch_bounds__(kThreads) void k_value_heads(FusedArgs a, int G) {
  value_head_item<E, PAGED, MODE>(a, G, blockIdx.x);
}

template <typename E>
hipError_t launch_two_launch_e(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                               int mode, const float *u, int32_t *idx_out, void *out, char *ws,
                               hipStream_t st) {
  FusedArgs args = make_args(p, kv, q, out, scale_log2, ws);
  args.u = u;
  args.idx_out = idx_out;
  return with_g_paged(p.G, kv.bt != nullptr, [&](auto gc, auto paged) -> hipError_t {
    constexpr int G = decltype(gc)::value;
    constexpr bool PG = decltype(paged)::value;
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
  });
}

template <typename E>
hipError_t launch_bernoulli_e(const Plan &p, const KvView &kv, const KtView &kt, const void *q,
                              float scale_log2, int Bd, int mode, const float *u_q, const float *u,
                              int32_t *idx_out, uint8_t *mask_out, void *out, char *ws,
                              hipStream_t st) {
  FusedArgs args = make_args(p, kv, q, out, scale_log2, ws);
  args.u = u;
  args.idx_out = idx_out;
  const CallTimer tm = call_timer();
  return with_g(p.G, [&](auto gc) -> hipError_t {
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

}  // namespace santa
