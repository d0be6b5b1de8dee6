// santa_fused.hip -- single-launch decode kernels (persistent).
//
// Every (batch b, KV head k) row is cut into T splits; split t of a row is one
// work item and one 256-thread workgroup.  The grid holds R whole rows per
// round (R*T workgroups, no more than fit on the GPU at once, so all of them
// are resident), and loops over rounds for larger batches.  Split lengths are per row (ceil(L_b/T) rounded
// to 16 keys), so ragged batches keep T splits of similar length per row.
//
// Sampled step, per work item:
//   1. stream the split's keys, scores for the G heads into LDS, split-local
//      CDF in LDS (Sec. 2.1: F is the running sum of the attention weights);
//   2. publish (m_t, l_t) and wait until every split of the row has (per-row
//      barrier, see row_arrive_wait; bounded spin);
//   3. every workgroup of the row computes the same global offsets
//      Off_t = sum_{t'<t} exp2(m_t' - m*) l_t' and Z, so threshold tau falls
//      in exactly one split; the split claims its thresholds, inverts its own
//      LDS CDF and gathers the chosen V rows (claim_gather);
//   4. after a second barrier every workgroup of the row sums its own slice of
//      the row's outputs over the split partials in split order, scales by 1/S
//      and writes it.
// Dense step: 1 and the exact V stream per split, one barrier, then the same
// distributed merge with the max/sum-exp rescaling.
//
// Cross-workgroup data (split statistics, partial sums, flags, counters) is
// written and read with relaxed agent-scope atomics, which are coherent per
// access across the XCDs' L2s; a writer waits for its stores to complete
// before it arrives at a barrier.  No cache-wide write-back or invalidation is
// issued.
//
// Each row's workgroups are placed on one XCD when the round holds a multiple
// of 8 rows (workgroups are dispatched round-robin over the 8 XCDs), so the
// row's barrier and merge traffic stays in one L2.
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
  float2 *stats;  // [B*Hq][T]        (m_t, l_t) per head and split
  float *part;    // [B*Hkv][T][G*128] split partial outputs
  int *flags;     // [B*Hkv][T]        sampled: split holds samples
  unsigned long long *sync;  // [B*Hkv][kSyncStride/2] arrival counter, counter base
  int *err;       // [1]               set if a barrier wait gave up
  int B, Hq, Hkv, T, S;
  int Lsmax;  // longest split (keys) of any row: LDS arrays are sized by it
  int ustage; // stratified uniforms of the group staged in LDS (G*S floats) if 1
  float invS, scale_log2;
  int xcd;
};

constexpr int kSpinLimit = 1 << 22;

// LDS layout of the fused kernels (dynamic shared memory), in floats.  The
// reduction buffers hold both the slot reduction (4 x G x 128 floats) and the
// per-thread merge partial sums (kThreads floats).
__host__ __device__ constexpr int fused_red_floats(int G) {
  return 4 * G * kHeadDim > kThreads ? 4 * G * kHeadDim : kThreads;
}
__host__ __device__ constexpr int fused_p_floats(int G, int Lsmax) {
  return G * Lsmax > fused_red_floats(G) ? G * Lsmax : fused_red_floats(G);
}

__device__ __forceinline__ void split_geometry(int L, int T, int &Ls, int &Tb) {
  if (L <= 0) {
    Ls = 16;
    Tb = 0;
    return;
  }
  Ls = (((L + T - 1) / T) + 15) & ~15;
  Tb = (L + Ls - 1) / Ls;
}

// Work item of workgroup w within a round: row rho (0..R-1), split t.
__device__ __forceinline__ void map_item(int w, int T, int R, int xcd, int &rho, int &t) {
  if (xcd && (R & 7) == 0) {
    const int x = w & 7, l = w >> 3;
    rho = x + 8 * (l / T);
    t = l % T;
  } else {
    rho = w / T;
    t = w % T;
  }
}

// Per-row barrier.  sync[0] counts arrivals and only ever grows; sync[1] holds
// its value when the current call started (the base).  The k-th barrier of a
// call waits until the count reaches base + k*n; the row's first split
// advances the base for the next call once every split has read it (after the
// first barrier).  Arrival is a fire-and-forget atomic add, so no workgroup
// waits on another's read-modify-write, and nothing has to be reset.
__device__ __forceinline__ void row_arrive_wait(unsigned long long *sync, unsigned long long target,
                                                int *err) {
  __hip_atomic_fetch_add(sync, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  int spins = 0;
  while (__hip_atomic_load(sync, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
    if (++spins > kSpinLimit) {
      atomicOr(err, 1);
      break;
    }
    __builtin_amdgcn_s_sleep(1);
  }
}

// All threads: make this workgroup's shared stores visible, arrive, wait.
__device__ __forceinline__ void row_sync(unsigned long long *sync, unsigned long long target,
                                         int *err) {
  wait_stores();
  __syncthreads();
  if (threadIdx.x == 0) row_arrive_wait(sync, target, err);
  __syncthreads();
}

// One wave: global offsets of one head over the row's Tb splits.  off[0..Tb]
// receives Off_0 = 0, Off_{t+1} = Off_t + exp2(m_t - m*) l_t, made exactly
// non-decreasing; returns m*.  Identical in every workgroup of the row.  Lane l
// owns splits l*ch .. l*ch+ch-1 (ch <= kMaxSplits / 64).
__device__ __forceinline__ float row_offsets_wave(const float2 *st, int Tb, int lane, float *off) {
  constexpr int CHM = kMaxSplits / 64;
  const int ch = (Tb + 63) >> 6;
  const int t0 = lane * ch;
  float2 sv[CHM];
#pragma unroll
  for (int i = 0; i < CHM; ++i)
    sv[i] = (i < ch && t0 + i < Tb) ? ld_coherent(st + t0 + i) : make_float2(-kInf, 0.0f);
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
    if (i < ch && t0 + i < Tb) off[t0 + i + 1] = fmaxf(run, floor_v);
  }
  if (lane == 0) off[0] = 0.0f;
  return m;
}

// This workgroup's slice of the row's G*128 outputs after the partials of all
// Tb splits are published: out[o] = scale_h * sum_t w_t * part[t][o] with
// h = o / 128.  Thread (group g, output o) sums splits t = g, g + ng, ... in
// order; groups are then summed in order.  w == nullptr means weight 1 and
// scale_h = `scale`; otherwise w is [G][T] in LDS and scale_h = 1 / den[h].
template <typename E, int G>
__device__ __forceinline__ void merge_slice(const float *part_row, int T, int Tb, int t,
                                            const float *w, const float *den, float scale,
                                            float *red, E *out_rows) {
  constexpr int NOUT = G * kHeadDim;
  const int tid = threadIdx.x;
  const int sl = (NOUT + Tb - 1) / Tb;
  const int o0 = t * sl, o1 = min(NOUT, o0 + sl);
  if (o0 >= o1) return;  // uniform for the workgroup
  const int n = o1 - o0;
  for (int ob = 0; ob < n; ob += kThreads) {
    const int m = min(kThreads, n - ob);
    int mp = 1;
    while (mp < m) mp <<= 1;
    const int ng = kThreads / mp;
    const int ol = tid % mp, g = tid / mp;
    float acc = 0.0f;
    if (ol < m) {
      const int o = o0 + ob + ol, h = o / kHeadDim;
      for (int tt = g; tt < Tb; tt += ng) {
        const float v = ld_coherent(part_row + (int64_t)tt * NOUT + o);
        acc = w ? fmaf(w[h * T + tt], v, acc) : acc + v;
      }
    }
    red[tid] = acc;
    __syncthreads();
    // pairwise tree over the ng groups (fixed order)
    for (int half = ng >> 1; half > 0; half >>= 1) {
      if (g < half) red[tid] += red[tid + half * mp];
      __syncthreads();
    }
    if (tid < m) {
      const int o = o0 + ob + tid, h = o / kHeadDim;
      store_out(out_rows + o, red[tid] * (w ? 1.0f / den[h] : scale));
    }
    __syncthreads();
  }
}

template <typename E, int G, bool PAGED, bool STRAT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(G <= 4 ? 4 : 2))) void k_fused_sampled(FusedArgs a) {
  // dynamic LDS: P [G][pitch] split CDF (reused as reduction buffer), cnt
  // [G][pitch] sample counts, then the compaction list, which is also the
  // offsets table [G][T+1] before the claims and the split flags [T] in the
  // merge, then (stratified, if staged) the group's uniforms [G][S].
  extern __shared__ float dyn[];
  const int pitch = a.Lsmax;
  float *P = dyn;
  int *cnt = reinterpret_cast<int *>(dyn + fused_p_floats(G, a.Lsmax));
  int *list = cnt + G * pitch;
  float *offl = reinterpret_cast<float *>(list);
  float *ul = reinterpret_cast<float *>(list + (pitch > G * (a.T + 1) ? pitch : G * (a.T + 1)));
  __shared__ HeadClaim hc[G];
  __shared__ float mh[G], mtmp[4 * G];
  __shared__ int wave_cnt[4];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nrk = a.B * a.Hkv, T = a.T;
  const int R = gridDim.x / T;
  int rho, t;
  map_item(blockIdx.x, T, R, a.xcd, rho, t);
  E *out = static_cast<E *>(a.out);

  for (int rbase = 0; rbase < nrk; rbase += R) {
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
    unsigned long long *sync = a.sync + (int64_t)rowkv * (kSyncStride / 2);
    const unsigned long long base =
        __hip_atomic_load(sync + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    float *part_row = a.part + (int64_t)rowkv * T * G * kHeadDim;

    // uniforms of the group (read while the keys stream)
    const float *us = STRAT ? a.u + row0 * a.S : a.u + row0;
    int64_t ustride = STRAT ? a.S : 1;
    if (STRAT && a.ustage) {
      for (int i = tid; i < G * a.S; i += kThreads) ul[i] = us[i];
      us = ul;
    }

    // 1. scores and split-local CDF
    const QRegs<E, G> qr = load_q<E, G>(static_cast<const E *>(a.q), b, a.Hq, kvh, tid & 15);
    float mx[G];
    score_tile<E, G, PAGED, kScoreUnroll>(a.kv, b, kvh, start, nrows, qr, a.scale_log2, P, pitch, mx);
    block_max_heads<G>(mx, mtmp, mh);
    for (int h = wave; h < G; h += kThreads / 64) wave_split_cdf_m(P + h * pitch, nrows, lane, mh[h]);
    __syncthreads();
    if (tid < G)
      st_coherent(a.stats + (row0 + tid) * T + t, make_float2(mh[tid], P[tid * pitch + nrows - 1]));
    for (int i = tid; i < G * pitch; i += kThreads) cnt[i] = 0;

    // 2. every split of the row has published its statistics
    row_sync(sync, base + (unsigned long long)Tb, a.err);
    if (t == 0 && tid == 0)
      __hip_atomic_store(sync + 1, base + 2ull * Tb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

    // 3. global offsets (one wave per head), claims, inverse CDF, gather
    for (int h = wave; h < G; h += kThreads / 64) {
      float *oh = offl + h * (T + 1);
      const float mstar = row_offsets_wave(a.stats + (row0 + h) * T, Tb, lane, oh);
      if (lane == 0)
        hc[h] = HeadClaim{oh[t], t == Tb - 1 ? kInf : oh[t + 1], oh[Tb], fast_exp2(mh[h] - mstar)};
    }
    __syncthreads();
    const bool has = claim_search<G, STRAT>(start, nrows, row0, a.S, a.invS, us, ustride, hc, P,
                                            pitch, cnt, a.idx_out);
    if (has) {
      gather_union<E, G, PAGED, true>(a.kv, b, kvh, start, nrows, P, pitch, cnt, list, wave_cnt,
                                      part_row + (int64_t)t * G * kHeadDim);
    } else {  // a split without samples contributes zeros
      float2 *pz = reinterpret_cast<float2 *>(part_row + (int64_t)t * G * kHeadDim);
      for (int o2 = tid; o2 < G * kHeadDim / 2; o2 += kThreads) st_coherent(pz + o2, make_float2(0.f, 0.f));
    }

    // 4. every split has published its partial sums; merge this split's slice
    row_sync(sync, base + 2ull * Tb, a.err);
    merge_slice<E, G>(part_row, T, Tb, t, nullptr, nullptr, a.invS, P, out + row0 * kHeadDim);
    __syncthreads();
  }
}

template <typename E, int G, bool PAGED>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(G <= 4 ? 4 : 2))) void k_fused_dense(FusedArgs a) {
  // dynamic LDS: s [G][pitch] scores / weights, red [fused_red_floats(G)], al [G][T]
  extern __shared__ float dyn[];
  const int pitch = a.Lsmax;
  float *s = dyn;
  float *red = s + G * pitch;
  float *al = red + fused_red_floats(G);
  __shared__ float mh[G], lh[G], den[G], mtmp[4 * G];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, slot = tid >> 4, c = tid & 15;
  const int nrk = a.B * a.Hkv, T = a.T;
  const int R = gridDim.x / T;
  int rho, t;
  map_item(blockIdx.x, T, R, a.xcd, rho, t);
  E *out = static_cast<E *>(a.out);
  const E *V = static_cast<const E *>(a.kv.v);

  for (int rbase = 0; rbase < nrk; rbase += R) {
    const int rowkv = rbase + rho;
    if (rowkv >= nrk) break;
    const int b = rowkv / a.Hkv, kvh = rowkv % a.Hkv;
    const int64_t row0 = (int64_t)b * a.Hq + kvh * G;
    const int L = seq_len(a.kv, b);
    int Ls, Tb;
    split_geometry(L, T, Ls, Tb);
    if (t >= Tb) {
      if (Tb == 0 && t == 0)
        for (int o = tid; o < G * kHeadDim; o += kThreads) store_out(out + row0 * kHeadDim + o, 0.0f);
      continue;
    }
    const int start = t * Ls, nrows = min(Ls, L - start);
    unsigned long long *sync = a.sync + (int64_t)rowkv * (kSyncStride / 2);
    const unsigned long long base =
        __hip_atomic_load(sync + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    float *part_row = a.part + (int64_t)rowkv * T * G * kHeadDim;

    const QRegs<E, G> qr = load_q<E, G>(static_cast<const E *>(a.q), b, a.Hq, kvh, c);
    float mx[G];
    score_tile<E, G, PAGED, kScoreUnroll>(a.kv, b, kvh, start, nrows, qr, a.scale_log2, s, pitch, mx);
    block_max_heads<G>(mx, mtmp, mh);
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
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[h][i] = 0.0f;
    constexpr int U = 4;
    for (int base_j = 0; base_j < nrows; base_j += 16 * U) {
      Chunk<E> ch[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = base_j + u * 16 + slot;
        ch[u] = j < nrows ? Chunk<E>::load(V + row_offset<PAGED>(a.kv, b, kvh, start + j) + c * 8)
                          : Chunk<E>::zero();
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = base_j + u * 16 + slot;
        float f[8];
        ch[u].to_float(f);
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float w = j < nrows ? s[h * pitch + j] : 0.0f;
#pragma unroll
          for (int i = 0; i < 8; ++i) acc[h][i] = fmaf(w, f[i], acc[h][i]);
        }
      }
    }
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
    if (tid < G) st_coherent(a.stats + (row0 + tid) * T + t, make_float2(mh[tid], lh[tid]));

    // all splits of the row have published (m_t, l_t, o_t)
    row_sync(sync, base + (unsigned long long)Tb, a.err);
    if (t == 0 && tid == 0)
      __hip_atomic_store(sync + 1, base + (unsigned long long)Tb, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    // rescale factors a_t = exp2(m_t - m*) and denominators sum_t a_t l_t
    for (int h = wave; h < G; h += kThreads / 64) {
      const float2 *st = a.stats + (row0 + h) * T;
      float m = -kInf;
      for (int tt = lane; tt < Tb; tt += 64) m = fmaxf(m, ld_coherent(st + tt).x);
      m = wave_max(m);
      float d = 0.0f;
      for (int tt = lane; tt < Tb; tt += 64) {
        const float2 v = ld_coherent(st + tt);
        const float aa = fast_exp2(v.x - m);
        al[h * T + tt] = aa;
        d = fmaf(aa, v.y, d);
      }
      d = wave_sum(d);
      if (lane == 0) den[h] = d;
    }
    __syncthreads();
    merge_slice<E, G>(part_row, T, Tb, t, al, den, 1.0f, red, out + row0 * kHeadDim);
    __syncthreads();
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
// workgroup of the grid is resident at once (the per-row barrier needs it).
hipError_t launch_resident(const void *fn, const Plan &p, FusedArgs &args, size_t lds,
                           hipStream_t st) {
  const int nrk = p.B * p.Hkv;
  const int cap = capacity_of(fn, lds);
  if (cap < p.T) return hipErrorInvalidConfiguration;
  const int R = std::min(nrk, cap / p.T);
  void *params[] = {&args};
  return hipLaunchKernel(fn, dim3(R * p.T), dim3(kThreads), params, lds, st);
}

FusedArgs make_args(const Plan &p, const KvView &kv, const void *q, void *out, float scale_log2,
                    char *ws) {
  FusedArgs a{};
  a.kv = kv;
  a.q = q;
  a.out = out;
  a.stats = reinterpret_cast<float2 *>(ws + p.off_stats);
  a.part = reinterpret_cast<float *>(ws + p.off_part);
  a.flags = reinterpret_cast<int *>(ws + p.off_flag);
  a.sync = reinterpret_cast<unsigned long long *>(ws + p.off_sync);
  a.err = reinterpret_cast<int *>(ws + p.off_err);
  a.B = p.B;
  a.Hq = p.Hq;
  a.Hkv = p.Hkv;
  a.T = p.T;
  a.S = p.S;
  a.Lsmax = p.Ls;
  a.invS = p.S ? 1.0f / (float)p.S : 0.0f;
  a.scale_log2 = scale_log2;
  a.xcd = p.xcd;
  return a;
}

}  // namespace

hipError_t launch_fused_dense(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                              void *out, char *ws, hipStream_t st) {
  FusedArgs args = make_args(p, kv, q, out, scale_log2, ws);
  return with_types(p, kv.bt != nullptr, [&](auto eptr, auto gc, auto paged) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    constexpr int G = decltype(gc)::value;
    constexpr bool PG = decltype(paged)::value;
    const size_t lds = ((size_t)G * p.Ls + fused_red_floats(G) + (size_t)G * p.T) * 4;
    return launch_resident(reinterpret_cast<const void *>(&k_fused_dense<E, G, PG>), p, args, lds,
                           st);
  });
}

hipError_t launch_fused_sampled(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                                bool strat, const float *u, int32_t *idx_out, void *out, char *ws,
                                hipStream_t st) {
  FusedArgs args = make_args(p, kv, q, out, scale_log2, ws);
  args.u = u;
  args.idx_out = idx_out;
  return with_types(p, kv.bt != nullptr, [&](auto eptr, auto gc, auto paged) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    constexpr int G = decltype(gc)::value;
    constexpr bool PG = decltype(paged)::value;
    const void *fn = strat ? reinterpret_cast<const void *>(&k_fused_sampled<E, G, PG, true>)
                           : reinterpret_cast<const void *>(&k_fused_sampled<E, G, PG, false>);
    // stage the group's stratified uniforms in LDS when they are small
    args.ustage = strat && (size_t)G * p.S <= 4096;
    const size_t lds = ((size_t)fused_p_floats(G, p.Ls) + (size_t)G * p.Ls +
                        std::max<size_t>((size_t)p.Ls, (size_t)G * (p.T + 1)) +
                        (args.ustage ? (size_t)G * p.S : 0)) * 4;
    return launch_resident(fn, p, args, lds, st);
  });
}

}  // namespace santa
