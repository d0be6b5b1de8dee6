// santa_rows.h -- the scheduled kernels: k_row_sampled (systematic,
// stratified and, at G <= 4, i.i.d. SANTA) and k_row_flash
// (S2ANTA-flash, G <= 4).  One workgroup per (row, split), scheduled by the
// hardware like the two-launch key stream, but the split's CDF stays in LDS:
// the split publishes its statistics, waits at its row's barrier (flash:
// none), claims its thresholds, gathers their V rows and publishes partial
// sums; the row's last arrival merges.  No CDF stash goes through HBM.
// Shared pieces are in santa_fused.h.
#pragma once

#include "santa_fused.h"

namespace santa {


// Waves per SIMD: the key stream relies on many resident workgroups, as in
// the two-launch stream (64 VGPRs for 16-bit rows with G <= 4).
template <typename E, int G, bool PAGED>
constexpr int row_waves() {
  if constexpr (sizeof(E) == 1) return G <= 4 ? 8 : 2;
  return sizeof(E) == 2 && G <= 4 && !PAGED ? 8 : (G <= 4 ? 4 : 2);
}

// Statistics mailbox of one row: word (h, t) holds the bits of (m_t, l_t) of
// head h in split t, l_t in the high half.  l_t >= 1 (the split's largest
// key adds exp2(0)), so a word whose high half is zero is empty.  Each word is
// written and read whole with 64-bit atomics, so a reader that sees it
// non-empty sees both values; the row's merger empties the words after every
// split has read them.
__device__ __forceinline__ void post_stats(unsigned long long *w, float m, float l) {
  const unsigned long long v = ((unsigned long long)__float_as_uint(l) << 32) | __float_as_uint(m);
  __hip_atomic_store(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One wave: lane t < Tb waits for word t (bounded spin; on giving up the
// error flag is set and the caller's results are not valid) and returns its
// (m_t, l_t).
__device__ __forceinline__ float2 wait_stats(const unsigned long long *w, int Tb, int lane,
                                             int *err) {
  unsigned long long v = 0;
  for (int spins = 0;; ++spins) {
    if (lane < Tb && (v >> 32) == 0)
      v = __hip_atomic_load(const_cast<unsigned long long *>(w + lane), __ATOMIC_RELAXED,
                            __HIP_MEMORY_SCOPE_AGENT);
    if (__all(lane >= Tb || (v >> 32) != 0)) break;
    if (spins > kSpinLimit) {
      if (lane == 0) atomicOr(err, 1);
      break;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  return make_float2(__uint_as_float((unsigned)v), __uint_as_float((unsigned)(v >> 32)));
}

// Sorted thresholds of the i.i.d. estimator (S <= 256) for one head, by one
// wave, in the register layout of the stratified uniforms: on entry ureg[k]
// of lane l holds u_r, r = l + 64 k < S, and uS the row's last uniform u_S; on
// return ureg[k] holds T_r = C_r / C_S with E_i = -log2(1 - u_i) and C_m =
// sum_{i <= m} E_i in double (the normalised partial sums of S + 1
// exponentials are the order statistics of S uniforms; the ln 2 factor
// cancels).  Each register's 64 partial sums come from a wave scan made
// non-decreasing by a prefix max and are offset by the sum of the earlier
// registers, so T is non-decreasing in r and at most 1.
__device__ __forceinline__ void iid_thresholds_regs(float (&ureg)[4], float uS, int S, int lane) {
  double carry = 0.0, c[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int r = lane + 64 * k;
    double incl = r < S ? -(double)__builtin_amdgcn_logf(1.0f - ureg[k]) : 0.0;
    for (int d = 1; d < 64; d <<= 1) {
      const double y = __shfl_up(incl, d);
      incl += lane >= d ? y : 0.0;
    }
    for (int d = 1; d < 64; d <<= 1) {
      const double y = __shfl_up(incl, d);
      incl = lane >= d ? fmax(incl, y) : incl;
    }
    c[k] = carry + incl;
    carry += __shfl(incl, 63);
  }
  const double total = carry - (double)__builtin_amdgcn_logf(1.0f - uS);
  const double inv = total > 0.0 ? 1.0 / total : 0.0;
#pragma unroll
  for (int k = 0; k < 4; ++k) ureg[k] = (float)(c[k] * inv);
}

// merge_group4 for a workgroup with Tb * 4 * 128 floats of free LDS at lds
// (16-byte aligned): every partial is copied straight into LDS
// (global_load_lds, agent-coherent like ld_coherent; 1 KiB, half a split, per
// wave instruction), so the merge takes one round trip, and then summed in
// split order, as merge_group4 does.
template <typename OE>
__device__ __forceinline__ void merge_group4_lds(const float *part_row, int Tb, float scale,
                                                 float *lds, OE *out_row0) {
  constexpr int G = 4, SPL = G * kHeadDim;  // floats per split
  constexpr int kCoherent = 16;               // sc1, as agent-scope loads
  typedef __attribute__((address_space(3))) void *lds_ptr;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const char *src = reinterpret_cast<const char *>(part_row);
  for (int k = wave; k < 2 * Tb; k += kThreads / 64)
    __builtin_amdgcn_global_load_lds(src + k * 1024 + lane * 16,
                                     (lds_ptr)(reinterpret_cast<char *>(lds) + k * 1024), 16, 0,
                                     kCoherent);
  wait_stores();  // vmcnt(0): this wave's copies have landed in LDS
  __syncthreads();
  const int h = wave, o = lane * 2;
  const float2 *l2 = reinterpret_cast<const float2 *>(lds + h * kHeadDim + o);
  float sx = 0.0f, sy = 0.0f;
  for (int t = 0; t < Tb; ++t) {
    const float2 w = l2[t * (SPL / 2)];
    sx += w.x;
    sy += w.y;
  }
  store_out(out_row0 + h * kHeadDim + o, sx * scale);
  store_out(out_row0 + h * kHeadDim + o + 1, sy * scale);
}

// A claim of the value stage: split-local key j and weight factor f.
struct Claim {
  int j;
  float f;
};

// One wave: claims r in [r0, r1), 64 per pass.  claim(r, ok) is called by
// every lane of a pass (ok: r < r1; the call may use lane shuffles) and
// returns claim r's key and factor (read only where ok).  The keys of
// successive claims are non-decreasing, so equal keys form runs with one
// factor; the runs of successive passes go to a per-wave list (keyl, cntl:
// 64 entries of key and weight count * factor) in LDS, gathered when the next
// pass's runs would not fit and at the end: each listed V row is read once per
// entry and added with its weight by one of the wave's four 16-lane slots, U
// rows in flight each.  acc: the weighted sum of V rows, reduced over the four
// slots in lanes 0..15 (8 columns each).
template <typename E, bool PAGED, typename CL>
__device__ __forceinline__ void wave_claims_gather(const FusedArgs &a, int b, int kvh, int start,
                                                   int r0, int r1, CL claim, int16_t *keyl,
                                                   float *cntl, float (&acc)[8]) {
  constexpr int U = 4;
  const int lane = threadIdx.x & 63, slot = lane >> 4, col = lane & 15;
  const E *V = static_cast<const E *>(a.kv.v);
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.0f;
  auto sync_lists = [] {  // list writes visible to the whole wave, in order
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  };
  auto gather = [&](int nl) {  // add the nl listed rows with their weights
    for (int q0 = 0; q0 < nl; q0 += 4 * U) {
      Chunk<E> ch[U];
      float w[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int q = q0 + slot + 4 * u;
        if (q < nl) {
          ch[u] = Chunk<E>::load(V + row_offset<PAGED>(a.kv, b, kvh, start + keyl[q]) + col * 8);
          w[u] = cntl[q];
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
  };
  int nl = 0;  // entries in the list (the same in every lane)
  for (int c0 = r0;; c0 += 64) {  // one pass past the last claims gathers the rest
    const bool done = c0 >= r1;
    const int r = c0 + lane, nv = min(64, r1 - c0);
    int j = -1;
    float f = 0.0f;
    if (!done) {
      const Claim cl = claim(r, r < r1);
      j = r < r1 ? cl.j : -1;
      f = cl.f;
    }
    const int jp = __shfl_up(j, 1);
    const bool first = !done && r < r1 && (lane == 0 || j != jp);
    const unsigned long long m = __ballot(first);
    const int nruns = __popcll(m);
    if (done || nl + nruns > 64) {  // the end, or the list is full: gather it
      gather(nl);
      sync_lists();
      nl = 0;
      if (done) break;
    }
    if (first) {
      const unsigned long long rest = lane < 63 ? m >> (lane + 1) : 0ull;
      const int e = nl + __popcll(m & ((1ull << lane) - 1ull));
      keyl[e] = (int16_t)j;
      cntl[e] = (float)(rest ? __builtin_ctzll(rest) + 1 : nv - lane) * f;
    }
    nl += nruns;
    sync_lists();
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = xor32_sum(xor16_sum(acc[i]));
}

// Value stage of head h in split t, by one wave, for sorted thresholds: the
// split claims r in [N(lo), N(hi)), N(y) = #{r : tau_r < y}.  ureg: the
// head's uniforms fetched before the row barrier -- kSys: u in ureg[0];
// kStrat with S <= 256 and staged (one head per wave): u_r in ureg[r / 64]
// of lane r % 64, so every lane counts its own thresholds and the claims
// read u_r with lane shuffles; kIid (always so held): the sorted threshold
// T_r in that place, tau_r = T_r Z; otherwise lanes 0 and 1 evaluate N(lo)
// and N(hi) in closed form (count_below) and u_r comes from global memory.
// Claim r takes the key #{j : a P_j <= tau_r - lo} of the split's LDS CDF
// (App. A, clamped to the split) with weight 1.  Returns the head's partial
// sum O_h = sum_j c_{h,j} V_j (Sec. 2) in lanes 0..15.
template <typename E, bool PAGED, int MODE>
__device__ __forceinline__ void row_head_value(const FusedArgs &a, const HeadClaim &c,
                                               const float *uh, const float (&ureg)[4], bool staged,
                                               const float *Ph, int nrows, int start, int b,
                                               int kvh, int64_t rowq, int16_t *keyl, float *cntl,
                                               float (&acc)[8]) {
  const int lane = threadIdx.x & 63;
  // kIid: in registers for S <= 256, else in LDS (uh)
  const bool regs = MODE == kSys || (staged && a.S <= 4 * 64);
  // tau_r from the register value v (u_r, or T_r for kIid)
  auto tau_reg = [&](int r, float v) {
    return MODE == kIid ? v * c.Z : threshold(r, v, a.invS, c.Z);
  };
  int rlo = 0, rhi = 0;
  if (MODE != kSys && regs) {  // N(lo), N(hi) over the registers
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int r = lane + 64 * k;
      const float tau = r < a.S ? tau_reg(r, ureg[k]) : kInf;
      rlo += __popcll(__ballot(tau < c.lo));
      rhi += __popcll(__ballot(tau < c.hi));
    }
  } else {
    int n = 0;
    if (lane < 2) {
      const float y = lane ? c.hi : c.lo;
      if constexpr (MODE == kIid) {  // binary search over the sorted T_r Z
        for (int step = 1 << (31 - __clz(a.S)); step > 0; step >>= 1)
          n = (n + step <= a.S && uh[n + step - 1] * c.Z < y) ? n + step : n;
      } else {
        n = count_below<MODE>(uh, MODE == kSys ? ureg[0] : 0.0f, a.S, a.invS, c.Z,
                              (float)a.S / c.Z, y);
      }
    }
    rlo = __builtin_amdgcn_readlane(n, 0);
    rhi = __builtin_amdgcn_readlane(n, 1);
  }
  auto claim = [&](int r, bool ok) {
    float ur = ureg[0];
    if (MODE != kSys && regs) {  // u_r (T_r) from lane r % 64 (every lane takes part)
      const int src = r & 63, k = (r >> 6) & 3;
      const float v0 = __shfl(ureg[0], src), v1 = __shfl(ureg[1], src);
      const float v2 = __shfl(ureg[2], src), v3 = __shfl(ureg[3], src);
      ur = k == 0 ? v0 : (k == 1 ? v1 : (k == 2 ? v2 : v3));
    }
    int j = 0;
    if (ok) {
      const float tau = MODE == kIid ? (regs ? ur : uh[r]) * c.Z
                                     : threshold(r, (MODE == kStrat && !regs) ? uh[r] : ur,
                                                 a.invS, c.Z);
      const int pos = lds_cdf_count(Ph, nrows, c.a, tau - c.lo);
      j = pos < nrows ? pos : nrows - 1;
      if (a.idx_out) a.idx_out[rowq * a.S + r] = start + j;
    }
    return Claim{j, 1.0f};
  };
  wave_claims_gather<E, PAGED>(a, b, kvh, start, rlo, rhi, claim, keyl, cntl, acc);
}

// S2ANTA-flash value stage of head h in split t, by one wave (Sec. 3.3; App.
// "S2ANTA-Flash Pseudocode", Kernel 1): every tile tau of the split takes
// S_tile systematic draws on its own CDF (tile CDFs in Ph, tile maxima tm and
// sums tl): draw i is the key whose tile-CDF interval holds ((i + a)/S_tile)
// l_tau, a = the head's uniform of the tile (App. A's inverse CDF, clamped to
// the tile), with weight exp2(m_tau - m_w) l_tau / S_tile (m_w: the split
// maximum), so that the split's partial sum is o_w = sum_tau exp2(m_tau -
// m_w) l_tau O_tau with O_tau the tile estimate.  Draw d = tau * S_tile + i;
// its key is non-decreasing in d.
template <typename E, bool PAGED>
__device__ __forceinline__ void row_head_flash(const FusedArgs &a, const float *Ph,
                                               const float *tm, const float *tl, float mw,
                                               int nrows, int start, int b, int kvh, int64_t rowq,
                                               int16_t *keyl, float *cntl, float (&acc)[8]) {
  const int tl2 = a.tile_log2, St = a.S_tile;
  const int ntile = (nrows + (1 << tl2) - 1) >> tl2;
  const int gt0 = start >> tl2;  // global index of the split's first tile
  const float invSt = 1.0f / (float)St;
  const float *uh = a.u + rowq * a.Tmax + gt0;
  auto claim = [&](int d, bool ok) {
    int j = 0;
    float f = 0.0f;
    if (ok) {
      const int tau = d / St, is = d - tau * St;
      const int t0 = tau << tl2, n = min(1 << tl2, nrows - t0);
      const float l = tl[tau];
      const float x = (((float)is + uh[tau]) * invSt) * l;
      const int k = lds_count_le(Ph + t0, n, x);
      j = t0 + (k < n ? k : n - 1);
      f = fast_exp2(tm[tau] - mw) * l * invSt;
      if (a.idx_out) a.idx_out[(rowq * a.Tmax + gt0 + tau) * St + is] = start + j;
    }
    return Claim{j, f};
  };
  wave_claims_gather<E, PAGED>(a, b, kvh, start, 0, ntile * St, claim, keyl, cntl, acc);
}

// One workgroup per work item (rowkv, t < T), items row-major so that a row's
// splits are dispatched together.  A split waits only for splits of its own
// row; with the dispatcher starting workgroups in index order those have all
// started or finished before any later row's, so every wait ends (and the
// wait is bounded regardless).  Row barrier, direct (grids of at most
// kDirectPollMax workgroups, one per CU): the split posts its statistics to
// the row's mailbox and each wave polls its head's words of all Tb splits;
// the partial sums take one arrival per split on the row counter (sync[0];
// sync[1] holds its value at the start of the call), and the merger moves the
// base on and empties the mailbox.  Otherwise, where waiting workgroups share
// CUs with streaming ones, thread 0 polls the counter: two arrivals per
// split, after the statistics and after the partial sums.
template <typename E, int G, bool PAGED, int MODE, bool APPEND = false, bool USTAGE = false>
__global__ __launch_bounds__(kThreads)
__attribute__((amdgpu_waves_per_eu(row_waves<E, G, PAGED>()))) void k_row_sampled(FusedArgs a) {
  static_assert(MODE == kSys || MODE == kStrat || (MODE == kIid && G <= 4),
                "thresholds with a closed-form count or in registers");
  extern __shared__ __attribute__((aligned(16))) float dyn[];
  constexpr int pitch = kSplitMax;
  float *P = dyn;  // [G][pitch]: scores, then the split CDF; merge scratch at the end
  __shared__ float offl[G][2 * kRowTMax + 1];  // per head: offsets [T+1], split factors [T]
  __shared__ float mh[G], mtmp[4 * G];
  __shared__ int16_t keyl[4][64];
  __shared__ float cntl[4][64];
  __shared__ int rank_lds;

  const int T = a.T, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rowkv = blockIdx.x / T, t = blockIdx.x % T;
  const int b = rowkv / a.Hkv, kvh = rowkv % a.Hkv;
  const int64_t row0 = (int64_t)b * a.Hq + kvh * G;
  QE<E> *out = static_cast<QE<E> *>(a.out);
  // splits of a.Ls keys in every row (the last one shorter), so a short row
  // takes few splits of full length rather than T tiny ones
  const int L = seq_len(a.kv, b);
  const int Ls = a.Ls, Tb = L > 0 ? (L + Ls - 1) / Ls : 0;
  if (t >= Tb) {
    if (Tb == 0 && t == 0) {  // empty sequence: zero output, no samples
      for (int o = tid; o < G * kHeadDim; o += kThreads) store_out(out + row0 * kHeadDim + o, 0.0f);
      if (a.idx_out)
        for (int o = tid; o < G * a.S; o += kThreads) a.idx_out[row0 * a.S + o] = -1;
    }
    return;
  }
  const int start = t * Ls, nrows = min(Ls, L - start);
  if constexpr (APPEND) append_current<E, PAGED>(a.kv, b, kvh, a.Hkv, start, nrows, L);

  // 1. scores of the G heads into LDS, split max, split CDF and statistics
  {
    const QRegs<E, G> qr = load_q<E, G>(static_cast<const QE<E> *>(a.q), b, a.Hq, kvh, tid & 15);
    const float ksc = kv_scales<E>(a.kv, b, kvh, a.Hkv).x;  // FP8 cache: K scale
    float mx[G];
    score_tile<E, G, PAGED, 4>(a.kv, b, kvh, start, nrows, qr,
                                                    a.scale_log2 * ksc, P, pitch, mx);
    block_max_heads<G>(mx, mtmp, mh);
  }
  // the row's counter base: it moves on only after every split of the row,
  // this one included, has made its last arrival, so it can be read this late
  unsigned long long *sync = a.sync + (int64_t)rowkv * (kSyncStride / 2);
  unsigned long long *mail = sync + kMailOffset;
  const unsigned long long base =
      __hip_atomic_load(sync + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (int h = wave; h < G; h += kThreads / 64) {
    float *Ph = P + h * pitch;
    wave_split_cdf_m(Ph, nrows, lane, mh[h]);
    if (lane == 0) {
      if (a.direct) post_stats(mail + h * kRowTMax + t, mh[h], Ph[nrows - 1]);
      else st_coherent(a.stats + (row0 + h) * T + t, make_float2(mh[h], Ph[nrows - 1]));
    }
  }
  unsigned long long arrived = 0;
  if (!a.direct) {  // first arrival, once the statistics are stored
    wait_stores();
    __syncthreads();
    if (tid == 0)
      arrived = __hip_atomic_fetch_add(sync, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1;
  }
  // the uniforms of head `wave` (G <= 4), fetched while the row arrives;
  // i.i.d.: turned into the head's sorted thresholds.  Budgets above the
  // registers' 256 go to LDS after the split CDFs in the USTAGE form:
  // stratified uniforms copied (global_load_lds, 4 bytes per lane, no
  // registers held), i.i.d. thresholds built there (wave_iid_thresholds)
  const int upr = MODE == kStrat ? a.S : (MODE == kIid ? a.S + 1 : 1);  // uniforms per head
  float ureg[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (G <= 4 && wave < G) {
    const float *uw = a.u + (row0 + wave) * upr;
    if (MODE == kSys) {
      ureg[0] = uw[0];
    } else if (a.S <= 4 * 64) {
#pragma unroll
      for (int k = 0; k < 4; ++k) ureg[k] = lane + 64 * k < a.S ? uw[lane + 64 * k] : 0.0f;
      if (MODE == kIid) iid_thresholds_regs(ureg, uw[a.S], a.S, lane);
    } else if constexpr (MODE == kStrat && USTAGE) {
      typedef __attribute__((address_space(3))) void *lds_ptr;
      float *ul = P + G * pitch + wave * a.S;
      for (int i = 0; i < a.S; i += 64)
        if (i + lane < a.S) __builtin_amdgcn_global_load_lds(uw + i + lane, (lds_ptr)(ul + i), 4, 0, 0);
    } else if constexpr (MODE == kIid && USTAGE) {  // the sorted thresholds, into LDS
      wave_iid_thresholds(uw, a.S, P + G * pitch + wave * a.S, lane);
    }
  }
  // 2. the row barrier, then per head, by wave h: global offsets, its claims
  // and V gather.  Direct: the wave polls its head's mailbox words.
  // Otherwise thread 0 polls the counter and the waves read the statistics.
  if (!a.direct) row_wait_unless(sync, base + (unsigned long long)Tb, arrived, a.err);
  float *part = a.part + ((int64_t)rowkv * T + t) * G * kHeadDim;
  for (int h = wave; h < G; h += kThreads / 64) {
    float2 sv = make_float2(0.0f, 0.0f);
    if (a.direct) sv = wait_stats(mail + h * kRowTMax, Tb, lane, a.err);
    else if (lane < Tb) sv = ld_coherent(a.stats + (row0 + h) * T + lane);
    float *oh = offl[h], *ah = offl[h] + (T + 1);
    head_offsets_from([&](int) { return sv; }, Tb, lane, oh, ah);  // Tb <= 64: split t in lane t
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    const HeadClaim c{oh[t], t == Tb - 1 ? kInf : oh[t + 1], oh[Tb], ah[t]};
    float acc[8];
    const float *uh = a.u + (row0 + h) * upr;
    if (G > 4) {  // two heads per wave: the head's own uniforms, from global memory
      ureg[0] = MODE == kSys ? uh[0] : 0.0f;
    }
    if constexpr (MODE != kSys && G <= 4 && USTAGE) {  // this wave's LDS copy
      wait_stores();  // vmcnt(0): the copies into LDS have landed
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      __builtin_amdgcn_wave_barrier();
      uh = P + G * pitch + h * a.S;
    }
    row_head_value<E, PAGED, MODE>(a, c, uh, ureg, G <= 4, P + h * pitch, nrows, start, b, kvh,
                                   row0 + h, keyl[wave], cntl[wave], acc);
    if (lane < 16) {
      float2 *d = reinterpret_cast<float2 *>(part + h * kHeadDim + lane * 8);
#pragma unroll
      for (int i = 0; i < 4; ++i) st_coherent(d + i, make_float2(acc[2 * i], acc[2 * i + 1]));
    }
  }

  // 3. last arrival of the split; the row's last one merges
  // O = (1/S) sum_t o_t, and (direct) empties the mailbox
  const unsigned long long arrivals = a.direct ? Tb : 2ull * Tb;  // of this call
  const int rank = row_arrive(sync, base + arrivals - Tb, &rank_lds);
  if (rank != Tb - 1) return;
  if (tid == 0)
    __hip_atomic_store(sync + 1, base + arrivals, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (a.direct)
    for (int i = tid; i < G * Tb; i += kThreads)
      __hip_atomic_store(mail + (i / Tb) * kRowTMax + i % Tb, 0ull, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  const float *part_row = a.part + (int64_t)rowkv * T * G * kHeadDim;
  const float scale = a.invS * kv_scales<E>(a.kv, b, kvh, a.Hkv).y;  // FP8 cache: V scale
  if constexpr (G == 4) {
    if (a.direct) merge_group4_lds(part_row, Tb, scale, P, out + row0 * kHeadDim);
    else merge_group4<16>(part_row, Tb, scale, out + row0 * kHeadDim);
  } else {
    for (int h = 0; h < G; ++h)
      merge_head<QE<E>, G>(part_row, h, Tb, nullptr, nullptr, scale, P, out + (row0 + h) * kHeadDim);
  }
}

// S2ANTA-flash on the scheduled skeleton (Sec. 3.3; App. "S2ANTA-Flash
// Pseudocode", Kernels 1 and 2), G <= 4: one workgroup per (row, split),
// splits of a.Ls keys rounded up to whole tiles.  No barrier stands before
// the value stage: each head's wave builds its tile CDFs (wave_tile_cdf),
// takes its draws (row_head_flash) and publishes o_w and (m_w, l_w), l_w =
// sum_tau exp2(m_tau - m_w) l_tau; one arrival per split on the row counter,
// and the row's last arrival merges O = sum_t a_t o_t / sum_t a_t l_t with
// a_t = exp2(m_t - m*) (Kernel 2), through LDS copies of the partials on
// direct grids.
template <typename E, int G, bool PAGED, bool APPEND = false>
__global__ __launch_bounds__(kThreads)
__attribute__((amdgpu_waves_per_eu(row_waves<E, G, PAGED>()))) void k_row_flash(FusedArgs a) {
  static_assert(G <= 4, "one head per wave");
  extern __shared__ __attribute__((aligned(16))) float dyn[];
  constexpr int pitch = kSplitMax, TS = kSplitMax / 16;
  float *P = dyn;  // [G][pitch]: scores, then the tile CDFs; merge copies at the end
  __shared__ float tst[G][2][TS];  // per head: tile maxima, tile sums
  __shared__ float mh[G], mtmp[4 * G];
  __shared__ float al[G][kRowTMax], den[G];
  __shared__ int16_t keyl[4][64];
  __shared__ float cntl[4][64];
  __shared__ int rank_lds;

  const int T = a.T, tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform in the wave
  const int rowkv = blockIdx.x / T, t = blockIdx.x % T;
  const int b = rowkv / a.Hkv, kvh = rowkv % a.Hkv;
  const int64_t row0 = (int64_t)b * a.Hq + kvh * G;
  QE<E> *out = static_cast<QE<E> *>(a.out);
  const int L = seq_len(a.kv, b);
  const int tl2 = a.tile_log2, align = max(kAlign, 1 << tl2);
  const int Ls = (a.Ls + align - 1) / align * align, Tb = L > 0 ? (L + Ls - 1) / Ls : 0;
  // tiles no split covers (past the row's length) have no draws
  if (a.idx_out && (t == Tb - 1 || (Tb == 0 && t == 0))) {
    const int t_end = (L + (1 << tl2) - 1) >> tl2;
    const int nt = (a.Tmax - t_end) * a.S_tile;
    for (int i = tid; i < G * nt; i += kThreads) {
      const int h = i / nt, k = i - h * nt;
      a.idx_out[((row0 + h) * a.Tmax + t_end) * a.S_tile + k] = -1;
    }
  }
  if (t >= Tb) {
    if (Tb == 0 && t == 0)  // empty sequence: zero output
      for (int o = tid; o < G * kHeadDim; o += kThreads) store_out(out + row0 * kHeadDim + o, 0.0f);
    return;
  }
  const int start = t * Ls, nrows = min(Ls, L - start);
  if constexpr (APPEND) append_current<E, PAGED>(a.kv, b, kvh, a.Hkv, start, nrows, L);
  {
    const QRegs<E, G> qr = load_q<E, G>(static_cast<const QE<E> *>(a.q), b, a.Hq, kvh, tid & 15);
    const float ksc = kv_scales<E>(a.kv, b, kvh, a.Hkv).x;  // FP8 cache: K scale
    float mx[G];
    score_tile<E, G, PAGED, 4>(a.kv, b, kvh, start, nrows, qr, a.scale_log2 * ksc, P, pitch, mx);
    block_max_heads<G>(mx, mtmp, mh);
  }
  unsigned long long *sync = a.sync + (int64_t)rowkv * (kSyncStride / 2);
  const unsigned long long base =
      __hip_atomic_load(sync + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  float *part = a.part + ((int64_t)rowkv * T + t) * G * kHeadDim;
  if (wave < G) {
    const int h = wave;
    float *Ph = P + h * pitch;
    wave_tile_cdf(Ph, nrows, lane, tl2, tst[h][0], tst[h][1]);
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    const int ntile = (nrows + (1 << tl2) - 1) >> tl2;
    float l = 0.0f;
    for (int tau = lane; tau < ntile; tau += 64) l += fast_exp2(tst[h][0][tau] - mh[h]) * tst[h][1][tau];
    l = wave_sum(l);
    float acc[8];
    row_head_flash<E, PAGED>(a, Ph, tst[h][0], tst[h][1], mh[h], nrows, start, b, kvh, row0 + h,
                             keyl[wave], cntl[wave], acc);
    if (lane < 16) {
      float2 *d = reinterpret_cast<float2 *>(part + h * kHeadDim + lane * 8);
#pragma unroll
      for (int i = 0; i < 4; ++i) st_coherent(d + i, make_float2(acc[2 * i], acc[2 * i + 1]));
    }
    if (lane == 0) st_coherent(a.stats + (row0 + h) * T + t, make_float2(mh[h], l));
  }

  // one arrival; the row's last arrival merges
  const int rank = row_arrive(sync, base, &rank_lds);
  if (rank != Tb - 1) return;
  if (tid == 0)
    __hip_atomic_store(sync + 1, base + (unsigned long long)Tb, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  const float *part_row = a.part + (int64_t)rowkv * T * G * kHeadDim;
  const float vsc = kv_scales<E>(a.kv, b, kvh, a.Hkv).y;  // FP8 cache: V scale
  constexpr int SPL = G * kHeadDim;  // floats per split: whole KiB for G >= 2
  const bool in_lds = G >= 2 && a.direct;
  if (in_lds) {  // all partials of the row into LDS (1 KiB per wave instruction)
    typedef __attribute__((address_space(3))) void *lds_ptr;
    const char *src = reinterpret_cast<const char *>(part_row);
    const int nk = Tb * (SPL / 256);  // 1 KiB pieces
    for (int k = wave; k < nk; k += kThreads / 64)
      __builtin_amdgcn_global_load_lds(src + k * 1024 + lane * 16,
                                       (lds_ptr)(reinterpret_cast<char *>(P) + k * 1024), 16, 0,
                                       16 /* sc1: agent-coherent */);
  }
  if (wave < G) {  // a_t and the denominator of head `wave`
    const float2 st = lane < Tb ? ld_coherent(a.stats + (row0 + wave) * T + lane)
                                : make_float2(-kInf, 0.0f);
    const float m = wave_max(st.x);
    const float at = lane < Tb ? fast_exp2(st.x - m) : 0.0f;
    const float d = wave_sum(at * st.y);
    if (lane < Tb) al[wave][lane] = at;
    if (lane == 0) den[wave] = d;
  }
  wait_stores();  // vmcnt(0): the copies into LDS have landed as well
  __syncthreads();
  for (int o2 = tid; o2 < SPL / 2; o2 += kThreads) {  // column pairs; split order, 16 in flight
    const int o = 2 * o2, h = o / kHeadDim;
    float sx = 0.0f, sy = 0.0f;
    for (int t0 = 0; t0 < Tb; t0 += 16) {
      float2 v[16];
#pragma unroll
      for (int i = 0; i < 16; ++i)
        v[i] = t0 + i >= Tb ? make_float2(0.0f, 0.0f)
               : in_lds     ? *reinterpret_cast<const float2 *>(P + (t0 + i) * SPL + o)
                            : ld_coherent(reinterpret_cast<const float2 *>(part_row + (int64_t)(t0 + i) * SPL + o));
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (t0 + i < Tb) {
          sx = fmaf(al[h][t0 + i], v[i].x, sx);
          sy = fmaf(al[h][t0 + i], v[i].y, sy);
        }
    }
    store_out(out + row0 * kHeadDim + o, sx * vsc / den[h]);
    store_out(out + row0 * kHeadDim + o + 1, sy * vsc / den[h]);
  }
}

template <typename E>
hipError_t launch_row_flash_e(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                              int tile_log2, int S_tile, const float *u, int32_t *idx_out,
                              void *out, char *ws, hipStream_t st) {
  if (p.T > kRowTMax || p.G > 4) return hipErrorInvalidValue;
  FusedArgs args = make_args(p, kv, q, out, scale_log2, ws);
  args.direct = (int64_t)p.B * p.Hkv * p.T <= kDirectPollMax;
  args.u = u;
  args.idx_out = idx_out;
  args.tile_log2 = tile_log2;
  args.S_tile = S_tile;
  args.Tmax = (p.n_k + (1 << tile_log2) - 1) >> tile_log2;
  return with_g_paged(p.G, kv.bt != nullptr, [&](auto gc, auto paged) -> hipError_t {
    constexpr int G = decltype(gc)::value;
    constexpr bool PG = decltype(paged)::value;
    if constexpr (G > 4) {
      return hipErrorInvalidValue;
    } else {
      const void *fn = kv.k_new ? reinterpret_cast<const void *>(&k_row_flash<E, G, PG, true>)
                                : reinterpret_cast<const void *>(&k_row_flash<E, G, PG>);
      void *params[] = {&args};
      // direct grids of G >= 2 merge through LDS copies of the T partials
      // (at most 128 KiB)
      const size_t lds = std::max((size_t)G * kSplitMax * 4,
                                  args.direct && G >= 2 ? (size_t)p.T * G * kHeadDim * 4 : 0);
      const CallTimer tm = call_timer();
      return hipExtLaunchKernel(fn, dim3(p.B * p.Hkv * p.T), dim3(kThreads), params, lds, st,
                                tm.start, tm.stop, 0);
    }
  });
}

template <typename E>
hipError_t launch_rows_e(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                         int mode, const float *u, int32_t *idx_out, void *out, char *ws,
                         hipStream_t st) {
  FusedArgs args = make_args(p, kv, q, out, scale_log2, ws);
  args.direct = (int64_t)p.B * p.Hkv * p.T <= kDirectPollMax;
  // stratified uniforms and i.i.d. thresholds beyond the registers, into LDS
  // on direct grids
  args.ustage = args.direct && (mode == kStrat || mode == kIid) && p.G <= 4 && p.S > 4 * 64 &&
                p.S <= 2048;
  if (p.T > kRowTMax || (mode != kSys && mode != kStrat && mode != kIid) ||
      (mode == kIid && (p.G > 4 || (p.S > 4 * 64 && !args.ustage))))
    return hipErrorInvalidValue;
  args.u = u;
  args.idx_out = idx_out;
  return with_g_paged(p.G, kv.bt != nullptr, [&](auto gc, auto paged) -> hipError_t {
    constexpr int G = decltype(gc)::value;
    constexpr bool PG = decltype(paged)::value;
    const bool ap = kv.k_new != nullptr;
    const void *fn = nullptr;
    if (mode == kStrat)
      fn = ap ? reinterpret_cast<const void *>(&k_row_sampled<E, G, PG, kStrat, true>)
              : reinterpret_cast<const void *>(&k_row_sampled<E, G, PG, kStrat>);
    else if (mode == kSys)
      fn = ap ? reinterpret_cast<const void *>(&k_row_sampled<E, G, PG, kSys, true>)
              : reinterpret_cast<const void *>(&k_row_sampled<E, G, PG, kSys>);
    if constexpr (G <= 4) {
      if (mode == kIid)
        fn = args.ustage
                 ? (ap ? reinterpret_cast<const void *>(&k_row_sampled<E, G, PG, kIid, true, true>)
                       : reinterpret_cast<const void *>(&k_row_sampled<E, G, PG, kIid, false, true>))
                 : (ap ? reinterpret_cast<const void *>(&k_row_sampled<E, G, PG, kIid, true>)
                       : reinterpret_cast<const void *>(&k_row_sampled<E, G, PG, kIid>));
      if (mode == kStrat && args.ustage)  // uniforms staged in LDS
        fn = ap ? reinterpret_cast<const void *>(&k_row_sampled<E, G, PG, kStrat, true, true>)
                : reinterpret_cast<const void *>(&k_row_sampled<E, G, PG, kStrat, false, true>);
    }
    if (!fn) return hipErrorInvalidValue;
    void *params[] = {&args};
    // direct grids of G = 4 merge through LDS (merge_group4_lds: T partials,
    // at most 128 KiB, within the 160 KiB of a CU); staged stratified
    // uniforms (at most 2048 per head) follow the split CDFs
    const size_t lds = std::max({(size_t)G * kSplitMax * 4,
                                 args.direct && G == 4 ? (size_t)p.T * G * kHeadDim * 4 : 0,
                                 args.ustage ? (size_t)G * (kSplitMax + p.S) * 4 : 0});
    const CallTimer tm = call_timer();
    return hipExtLaunchKernel(fn, dim3(p.B * p.Hkv * p.T), dim3(kThreads), params, lds, st,
                              tm.start, tm.stop, 0);
  });
}

}  // namespace santa
