// santa_sampled.h -- the one-launch sampled step (k_fused_sampled): key
// stream, split CDF, row barrier, exact global claims, union gather and
// last-arrival merge in one persistent launch (see santa_fused.h).
#pragma once

#include "santa_fused.h"

namespace santa {

// ---------------------------------------------------------------------------
// Small-batch sampled step
// ---------------------------------------------------------------------------
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

// Claims of the group without a workgroup barrier between ranges and keys
// (sorted thresholds with a closed-form count and staged uniforms; 2G <= 64):
// in every wave, lanes 2h and 2h + 1 count head h's thresholds below lo and
// hi (count_below), so each wave holds all G claimed ranges [N(lo), N(hi))
// at once; the claims are then dealt to all threads of the workgroup (a hot
// split of one head is not left to one wave), each r mapped to the key #{j :
// a P_j <= tau_r - lo} (the CDF interval holding tau, App. A), clamped to the
// split.  Counts go to cnt (LDS), and every chosen key sets its bit in the
// split's key mask kmask (LDS, one bit per key) for the union compaction.
template <int G, int MODE>
__device__ __forceinline__ void claim_keys_mask(const HeadClaim *hc, const float *ul, int S,
                                                float invS, const float *P, int pitch, int nrows,
                                                int start, int64_t row0, int *cnt, unsigned *kmask,
                                                int32_t *__restrict__ idx_out) {
  static_assert(2 * G <= 64, "one lane per range end");
  const int lane = threadIdx.x & 63;
  int n = 0;
  if (lane < 2 * G) {
    const int h = lane >> 1;
    const HeadClaim c = hc[h];
    const float *uh = ul + h * (MODE == kSys ? 1 : S);
    n = count_below<MODE>(uh, MODE == kSys ? uh[0] : 0.0f, S, invS, c.Z, (float)S / c.Z,
                          (lane & 1) ? c.hi : c.lo);
  }
  int lo[G], first[G + 1];
  first[0] = 0;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    lo[h] = __builtin_amdgcn_readlane(n, 2 * h);
    first[h + 1] = first[h] + max(0, __builtin_amdgcn_readlane(n, 2 * h + 1) - lo[h]);
  }
  for (int i = threadIdx.x; i < first[G]; i += kThreads) {
    int h = 0, r = lo[0] + i;
#pragma unroll
    for (int k = 1; k < G; ++k)
      if (i >= first[k]) h = k, r = lo[k] + (i - first[k]);
    const HeadClaim c = hc[h];
    const float tau = tau_of<MODE>(ul + h * (MODE == kSys ? 1 : S), r, invS, c.Z);
    const int pos = lds_cdf_count(P + h * pitch, nrows, c.a, tau - c.lo);
    const int j = pos < nrows ? pos : nrows - 1;
    atomicAdd(&cnt[h * pitch + j], 1);
    atomicOr(&kmask[j >> 5], 1u << (j & 31));
    if (idx_out) idx_out[(row0 + h) * S + r] = start + j;
  }
}

// The union over the group's heads of the chosen keys, in key order, from the
// split's key mask (nwords <= 64 32-bit words), by a prefix sum of the words'
// bit counts.  Sparse words (at most 8 bits each) are walked bit by bit by
// the lanes of wave 0; denser masks are expanded by all waves, two words per
// pass (lane i holds bit i % 32 of word 2p + i / 32).  Returns the list
// length (block-uniform).
__device__ __forceinline__ int compact_union_mask(const unsigned *kmask, int nwords, int *list) {
  static_assert(kSplitMax / 32 <= 64, "one key-mask word per lane");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned mine = lane < nwords ? kmask[lane] : 0u;
  const int pc = __popc(mine);
  const float inc = wave_incl_scan((float)pc);  // exact: at most kSplitMax
  const int excl = (int)inc - pc;
  const int total = (int)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(inc), 63));
  if (wave_max((float)pc) <= 8.0f) {  // uniform: every lane holds the maximum
    if (wave == 0) {
      unsigned m = mine;
      int pos = excl;
      while (m) {
        list[pos++] = lane * 32 + (__ffs(m) - 1);
        m &= m - 1u;
      }
    }
  } else {
    const int bit = lane & 31;
    for (int w0 = 2 * wave; w0 < nwords; w0 += 2 * (kThreads / 64)) {
      const int wd = w0 + (lane >> 5);  // < 64: a valid source lane
      const unsigned m = (unsigned)__shfl((int)mine, wd);
      const int off = __shfl(excl, wd);
      if ((m >> bit) & 1u) list[off + __popc(m & ((1u << bit) - 1u))] = wd * 32 + bit;
    }
  }
  __syncthreads();
  return total;
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
  __shared__ unsigned kmask[kSplitMax / 32];  // one bit per key of the split (G = 4 claims)

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nrk = a.B * a.Hkv;
  const int R = gridDim.x / T;  // rows per round
  int rho, t;
  map_item(blockIdx.x, T, R, rho, t);
  QE<E> *out = static_cast<QE<E> *>(a.out);

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
    const QRegs<E, G> qr = load_q<E, G>(static_cast<const QE<E> *>(a.q), b, a.Hq, kvh, tid & 15);
    const float2 sc = kv_scales<E>(a.kv, b, kvh, a.Hkv);  // FP8 cache: K and V scales
    float mx[G];
    score_tile<E, G, PAGED, score_unroll<E, G>()>(a.kv, b, kvh, start, nrows, qr, a.scale_log2 * sc.x, P,
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
    if (tid < kSplitMax / 32) kmask[tid] = 0u;
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
    if constexpr (G >= 4 && MODE != kIid) {
      if (a.ustage) {
        claim_keys_mask<G, MODE>(hc, ul, a.S, a.invS, P, pitch, nrows, start, row0, cnt, kmask,
                                 a.idx_out);
        __syncthreads();  // counts and mask complete; offl/all are no longer needed
        const int nlist = compact_union_mask(kmask, (nrows + 31) >> 5, list);
        float *po = part_row + (int64_t)t * G * kHeadDim;
        if (nlist == 0) {  // a split without samples contributes zeros
          for (int o2 = tid; o2 < G * kHeadDim / 2; o2 += kThreads)
            st_coherent(reinterpret_cast<float2 *>(po) + o2, make_float2(0.f, 0.f));
        } else if (nlist <= 16) {
          gather_heads_waves<E, G, PAGED>(a.kv, b, kvh, start, cnt, pitch, list, nlist, po);
        } else {
          constexpr int UG = sizeof(E) <= 2 ? 8 : 4;
          gather_list<E, G, PAGED, true, false, UG>(a.kv, b, kvh, start, list, nlist, P, pitch, cnt,
                                                    po);
        }
        goto arrive2;
      }
    }
    {
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
        constexpr int UG = (sizeof(E) <= 2 && G <= 4) ? 8 : 4;
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
    }

    // 4. arrive; the last min(G, Tb) arrivals merge one or more heads each
  arrive2:
    const int W = G == 4 ? 1 : min(G, Tb);  // G = 4: the last arrival merges the group
    const int rank = row_arrive(sync, base + (unsigned long long)Tb, &rank_lds);
    if (rank < Tb - W) continue;
    if (rank == Tb - 1) {
      if (tid == 0)
        __hip_atomic_store(sync + 1, base + 2ull * Tb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      row_wait(sync, base + 2ull * Tb, a.err);
    }
    if constexpr (G == 4) {
      merge_group4(part_row, Tb, a.invS * sc.y, out + row0 * kHeadDim);
    } else {
      for (int h = rank - (Tb - W); h < G; h += W)
        merge_head<QE<E>, G>(part_row, h, Tb, nullptr, nullptr, a.invS * sc.y, P,
                             out + (row0 + h) * kHeadDim);
    }
  }
}

template <typename E>
hipError_t launch_one_launch_e(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                               int mode, const float *u, int32_t *idx_out, void *out, char *ws,
                               hipStream_t st) {
  FusedArgs args = make_args(p, kv, q, out, scale_log2, ws);
  args.u = u;
  args.idx_out = idx_out;
  return with_g_paged(p.G, kv.bt != nullptr, [&](auto gc, auto paged) -> hipError_t {
    constexpr int G = decltype(gc)::value;
    constexpr bool PG = decltype(paged)::value;
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
