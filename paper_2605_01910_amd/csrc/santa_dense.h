// santa_dense.h -- the exact dense step and the S2ANTA-flash step
// (k_fused_dense; see santa_fused.h).
#pragma once

#include "santa_fused.h"

namespace santa {

// ---------------------------------------------------------------------------
// S2ANTA-flash value stage (Sec. 3.3; App. "S2ANTA-Flash Pseudocode", Kernel 1)
// ---------------------------------------------------------------------------
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
  QE<E> *out = static_cast<QE<E> *>(a.out);
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

    const QRegs<E, G> qr = load_q<E, G>(static_cast<const QE<E> *>(a.q), b, a.Hq, kvh, c);
    const float2 sc = kv_scales<E>(a.kv, b, kvh, a.Hkv);  // FP8 cache: K and V scales
    float mx[G];
    constexpr int U = PERSIST ? score_unroll<E, G>() : (sizeof(E) == 1 && G <= 4 ? 8 : 4);
    score_tile<E, G, PAGED, U>(a.kv, b, kvh, start, nrows, qr, a.scale_log2 * sc.x, s, pitch, mx);
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
        constexpr int UG = (sizeof(E) <= 2 && G <= 4) ? 8 : 4;
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
      merge_head<QE<E>, G>(part_row, h, Tb, al, &den, sc.y, red, out + (row0 + h) * kHeadDim);
    }
  }
}

template <typename E>
hipError_t launch_dense_e(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                          void *out, char *ws, hipStream_t st) {
  FusedArgs args = make_args(p, kv, q, out, scale_log2, ws);
  return with_g_paged(p.G, kv.bt != nullptr, [&](auto gc, auto paged) -> hipError_t {
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

template <typename E>
hipError_t launch_flash_e(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                          int tile_log2, int S_tile, const float *u, int32_t *idx_out, void *out,
                          char *ws, hipStream_t st) {
  FusedArgs args = make_args(p, kv, q, out, scale_log2, ws);
  args.u = u;
  args.idx_out = idx_out;
  args.tile_log2 = tile_log2;
  args.S_tile = S_tile;
  args.Tmax = (p.n_k + (1 << tile_log2) - 1) >> tile_log2;
  return with_g_paged(p.G, kv.bt != nullptr, [&](auto gc, auto paged) -> hipError_t {
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

}  // namespace santa
