// santa_kernels.hip -- gfx950 kernels of one SANTA / S2ANTA decode step.
//
// Work decomposition: every (batch b, KV head k) row is cut into splits of Ls
// keys; one 256-thread workgroup owns one split and all G = Hq/Hkv query heads
// of the GQA group, so each key row is read once for the whole group.
//
//   dense       k_dense_split   scores, split max / sum-exp, sum_j e_j V_j
//               k_merge_dense   max/sum-exp merge of the split partials
//   sampled     k_score_cdf     scores, split max, split-local CDF (stashed)
//               k_offsets       global split offsets of the row's CDF
//               k_sample        threshold claim, inverse-CDF search, V gather-add
//               k_merge_sampled fixed-order sum of split partials, times 1/S
//   Bernoulli   k_bern_prep     ternary / mean-group query weights, feature list
//               k_bern_score    scores over the selected K^T feature rows
//               (then k_offsets, k_sample, k_merge_sampled)
//
// Scores are kept in log2 units (s * scale * log2 e) so exponentials are one
// v_exp_f32 each.  Every reduction has a fixed order, so repeated calls on the
// same inputs give bitwise-identical outputs.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "santa_kernels.h"
#include "santa_tiles.h"

namespace santa {

// ---------------------------------------------------------------------------
// dense: split partials and merge
// ---------------------------------------------------------------------------
template <typename E, int G, bool PAGED>
__global__ __launch_bounds__(kThreads) void k_dense_split(KvView kv, const E *__restrict__ q,
                                                           int Hq, int Ls, int T, float scale_log2,
                                                           float2 *__restrict__ stats,
                                                           float *__restrict__ part) {
  const int t = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int L = seq_len(kv, b);
  const int start = t * Ls;
  if (start >= L) return;
  const int nrows = min(Ls, L - start);
  __shared__ __attribute__((aligned(16))) float s[G * kSplitMax];
  __shared__ float red[4 * G * kHeadDim];
  __shared__ float mh[G], lh[G];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, slot = tid >> 4, c = tid & 15;
  const int64_t row0 = (int64_t)b * Hq + kvh * G;

  const QRegs<E, G> qr = load_q<E, G>(q, b, Hq, kvh, c);
  float mx[G];
  score_tile<E, G, PAGED, score_unroll<E, G>()>(kv, b, kvh, start, nrows, qr, scale_log2, s, kSplitMax, mx);
  __syncthreads();
  // split max and exponentials e_j = exp2(s_j - m_t), l_t = sum_j e_j
  for (int h = wave; h < G; h += kThreads / 64) {
    float *sh = s + h * kSplitMax;
    float m = -kInf;
    for (int j = lane; j < nrows; j += 64) m = fmaxf(m, sh[j]);
    m = wave_max(m);
    float l = 0.0f;
    for (int j = lane; j < nrows; j += 64) {
      const float e = fast_exp2(sh[j] - m);
      sh[j] = e;
      l += e;
    }
    l = wave_sum(l);
    if (lane == 0) {
      mh[h] = m;
      lh[h] = l;
    }
  }
  __syncthreads();
  // o_t = sum_j e_j V_j
  const E *V = static_cast<const E *>(kv.v);
  float acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[h][i] = 0.0f;
  constexpr int U = 8;
  for (int base = 0; base < nrows; base += 16 * U) {
    Chunk<E> ch[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = base + u * 16 + slot;
      ch[u] = j < nrows ? Chunk<E>::load(V + row_offset<PAGED>(kv, b, kvh, start + j) + c * 8)
                        : Chunk<E>::zero();
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = base + u * 16 + slot;
      float f[8];
      ch[u].to_float(f);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float w = j < nrows ? s[h * kSplitMax + j] : 0.0f;
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[h][i] = fmaf(w, f[i], acc[h][i]);
      }
    }
  }
  reduce_slots<G>(acc, red);
  const int64_t sid = ((int64_t)b * gridDim.y + kvh) * T + t;
  for (int o = tid; o < G * kHeadDim; o += kThreads) {
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) v += red[w * G * kHeadDim + o];
    part[sid * G * kHeadDim + o] = v;
  }
  if (tid < G) stats[(row0 + tid) * T + t] = make_float2(mh[tid], lh[tid]);
}

// out = sum_t a_t o_t / sum_t a_t l_t with a_t = exp2(m_t - max_t m_t).
template <typename E, int G>
__global__ __launch_bounds__(kHeadDim) void k_merge_dense(KvView kv, int Hq, int Hkv, int Ls,
                                                          int T, const float2 *__restrict__ stats,
                                                          const float *__restrict__ part,
                                                          E *__restrict__ out) {
  const int row = blockIdx.x, b = row / Hq, h = row % Hq, kvh = h / G, g = h % G,
            f = threadIdx.x;
  const int L = seq_len(kv, b);
  const int Tb = (L + Ls - 1) / Ls;
  const float2 *st = stats + (int64_t)row * T;
  float m = -kInf;
  for (int t = 0; t < Tb; ++t) m = fmaxf(m, st[t].x);
  float num = 0.0f, den = 0.0f;
  const int64_t sid0 = ((int64_t)b * Hkv + kvh) * T;
  for (int t = 0; t < Tb; ++t) {
    const float a = fast_exp2(st[t].x - m);
    num = fmaf(a, part[(sid0 + t) * G * kHeadDim + g * kHeadDim + f], num);
    den = fmaf(a, st[t].y, den);
  }
  store_out(out + (int64_t)row * kHeadDim + f, Tb ? num / den : 0.0f);
}

// ---------------------------------------------------------------------------
// sampled: scores + split CDF
// ---------------------------------------------------------------------------
template <typename E, int G, bool PAGED>
__global__ __launch_bounds__(kThreads) void k_score_cdf(KvView kv, const E *__restrict__ q, int Hq,
                                                         int Ls, int T, float scale_log2,
                                                         float2 *__restrict__ stats,
                                                         float *__restrict__ stash) {
  const int t = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int L = seq_len(kv, b);
  const int start = t * Ls;
  if (start >= L) return;
  const int nrows = min(Ls, L - start);
  __shared__ __attribute__((aligned(16))) float s[G * kSplitMax];
  __shared__ float mh[G];
  const QRegs<E, G> qr = load_q<E, G>(q, b, Hq, kvh, threadIdx.x & 15);
  float mx[G];
  score_tile<E, G, PAGED, score_unroll<E, G>()>(kv, b, kvh, start, nrows, qr, scale_log2, s, kSplitMax, mx);
  __syncthreads();
  finish_split_cdf<G>(s, mh, nrows, (int64_t)b * Hq + kvh * G, T, t, (int64_t)T * Ls, start,
                      stats, stash);
}

// Global CDF offsets of one row (one wave per row): with m* = max_t m_t,
// a_t = exp2(m_t - m*), W_t = a_t l_t, Off_0 = 0, Off_{t+1} = Off_t + W_t and
// Z = Off_{Tb}.  Threshold T_m * Z then falls in exactly one split, the t with
// Off_t <= T_m Z < Off_{t+1}.  The prefix is made exactly non-decreasing (a
// running max over lane runs) so the split intervals partition [0, Z).
__global__ __launch_bounds__(64) void k_offsets(KvView kv, int Hq, int Ls, int T,
                                                const float2 *__restrict__ stats,
                                                float *__restrict__ offs,
                                                float *__restrict__ alpha,
                                                float2 *__restrict__ rowst) {
  const int row = blockIdx.x, b = row / Hq, lane = threadIdx.x;
  const int L = seq_len(kv, b);
  const int Tb = (L + Ls - 1) / Ls;
  if (Tb == 0) return;
  const float2 *st = stats + (int64_t)row * T;
  float *off = offs + (int64_t)row * (T + 1);
  float *al = alpha + (int64_t)row * T;
  float m = -kInf;
  for (int t = lane; t < Tb; t += 64) m = fmaxf(m, st[t].x);
  m = wave_max(m);
  const int ch = (Tb + 63) >> 6;
  const int t0 = lane * ch;
  float tot = 0.0f;
  for (int i = 0; i < ch; ++i) {
    const int t = t0 + i;
    if (t < Tb) {
      const float a = fast_exp2(st[t].x - m);
      al[t] = a;
      tot = fmaf(a, st[t].y, tot);
    }
  }
  const float base = wave_prev(0.0f, wave_incl_scan(tot));
  // lane runs are non-decreasing; lift each run to the max of all earlier runs' ends
  float run = base;
  for (int i = 0; i < ch; ++i) {
    const int t = t0 + i;
    if (t < Tb) run = fmaf(al[t], st[t].y, run);
  }
  const float pm = wave_incl_max(run);
  const float floor_v = wave_prev(0.0f, pm);
  run = base;
  for (int i = 0; i < ch; ++i) {
    const int t = t0 + i;
    if (t < Tb) {
      run = fmaf(al[t], st[t].y, run);
      off[t + 1] = fmaxf(run, floor_v);
    }
  }
  // Z is the inclusive max over all lanes, i.e. the last offset written
  const float Z = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pm), 63));
  if (lane == 0) {
    off[0] = 0.0f;
    rowst[row] = make_float2(m, Z);
  }
}

// Threshold claim, inverse-CDF search and gather-add for one split, from the
// stashed split CDF (see claim_gather).
template <typename E, int G, bool PAGED, bool STRAT>
__global__ __launch_bounds__(kThreads) void k_sample(
    KvView kv, int Hq, int Ls, int T, int S, float invS, const float *__restrict__ u,
    const float *__restrict__ stash, const float *__restrict__ offs,
    const float *__restrict__ alpha, const float2 *__restrict__ rowst, int *__restrict__ flags,
    float *__restrict__ part, int32_t *__restrict__ idx_out) {
  const int t = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int L = seq_len(kv, b);
  const int start = t * Ls;
  if (start >= L) return;
  const int nrows = min(Ls, L - start);
  const int Tb = (L + Ls - 1) / Ls;
  const int tid = threadIdx.x;
  const int64_t row0 = (int64_t)b * Hq + kvh * G;
  const int64_t sid = ((int64_t)b * gridDim.y + kvh) * T + t;

  __shared__ HeadClaim hc[G];
  __shared__ __attribute__((aligned(16))) float P[G * kSplitMax];  // split CDF; reused as the slot-reduction buffer
  __shared__ int cnt[G * kSplitMax];
  __shared__ int list[kSplitMax];

  if (tid < G) {
    const int64_t r = row0 + tid;
    hc[tid] = HeadClaim{offs[r * (T + 1) + t], t == Tb - 1 ? kInf : offs[r * (T + 1) + t + 1],
                        rowst[r].y, alpha[r * T + t]};
  }
  __syncthreads();
  if (!any_claims<G, STRAT>(hc, row0, S, invS, u)) {
    if (tid == 0) flags[sid] = 0;
    return;
  }
  const int64_t pitch = (int64_t)T * Ls;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float *src = stash + (row0 + h) * pitch + start;
    for (int j = tid; j < nrows; j += kThreads) {
      P[h * kSplitMax + j] = src[j];
      cnt[h * kSplitMax + j] = 0;
    }
  }
  __syncthreads();
  claim_search<G, STRAT>(start, nrows, row0, S, invS, STRAT ? u + row0 * S : u + row0,
                         STRAT ? S : 1, hc, P, kSplitMax, cnt, idx_out);
  gather_union<E, G, PAGED, false>(kv, b, kvh, start, nrows, P, kSplitMax, cnt, list,
                                   part + sid * G * kHeadDim);
  if (tid == 0) flags[sid] = 1;
}

// out = (1/S) sum_t O_t over the row's splits, in split order
// (Sec. 2, Eq. "stochastic-add-only-attn").
template <typename E, int G>
__global__ __launch_bounds__(kHeadDim) void k_merge_sampled(KvView kv, int Hq, int Hkv, int Ls,
                                                            int T, int S, float invS,
                                                            const int *__restrict__ flags,
                                                            const float *__restrict__ part,
                                                            E *__restrict__ out,
                                                            int32_t *__restrict__ idx_out) {
  const int row = blockIdx.x, b = row / Hq, h = row % Hq, kvh = h / G, g = h % G,
            f = threadIdx.x;
  const int L = seq_len(kv, b);
  const int Tb = (L + Ls - 1) / Ls;
  const int64_t sid0 = ((int64_t)b * Hkv + kvh) * T;
  float acc = 0.0f;
  for (int t = 0; t < Tb; ++t)
    if (flags[sid0 + t]) acc += part[(sid0 + t) * G * kHeadDim + g * kHeadDim + f];
  store_out(out + (int64_t)row * kHeadDim + f, acc * invS);
  if (Tb == 0 && idx_out)
    for (int r = f; r < S; r += kHeadDim) idx_out[(int64_t)row * S + r] = -1;
}

// ---------------------------------------------------------------------------
// Bernoulli score stage
// ---------------------------------------------------------------------------
__device__ __forceinline__ float block128_max(float v, float *tmp /* [2] */) {
  v = wave_max(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) tmp[wave] = v;
  __syncthreads();
  return fmaxf(tmp[0], tmp[1]);
}

// Query weights of one GQA group (one thread per feature i).  Decisions in
// float32: pi = |q_i|/norm (mode 0) or m_i/norm (mode 1), and
// c_i = #{n < B : (n + u_i)/B < pi_i} (Sec. 5, Eq. "qk_estimator"; App. C).
template <typename E, int G>
__global__ __launch_bounds__(kHeadDim) void k_bern_prep(const E *__restrict__ q, int Hq, int Hkv,
                                                        int Bd, int mode,
                                                        const float *__restrict__ u_q,
                                                        float *__restrict__ wout,
                                                        int *__restrict__ flist,
                                                        int *__restrict__ fcount,
                                                        uint8_t *__restrict__ mask_out) {
  const int grp = blockIdx.x, b = grp / Hkv, kvh = grp % Hkv, i = threadIdx.x;
  const int lane = i & 63, wave = i >> 6;
  __shared__ float tmp[2];
  __shared__ int wc[2];
  float qv[G];
#pragma unroll
  for (int g = 0; g < G; ++g) qv[g] = to_f32(q[((int64_t)b * Hq + kvh * G + g) * kHeadDim + i]);
  float w[G];
  const float fB = (float)Bd;
  if (mode == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float norm = block128_max(fabsf(qv[g]), tmp);
      const float pi = norm > 0.0f ? fabsf(qv[g]) / norm : 0.0f;
      const float ug = u_q[((int64_t)b * Hq + kvh * G + g) * kHeadDim + i];
      int cnt = 0;
      for (int n = 0; n < Bd; ++n) cnt += (((float)n + ug) / fB) < pi;
      const float sgn = qv[g] > 0.0f ? 1.0f : (qv[g] < 0.0f ? -1.0f : 0.0f);
      w[g] = sgn * (float)cnt * (norm / fB);
    }
  } else {
    float a = 0.0f;
#pragma unroll
    for (int g = 0; g < G; ++g) a += fabsf(qv[g]);
    const float m = a / (float)G;
    const float norm = block128_max(m, tmp);
    const float pi = norm > 0.0f ? m / norm : 0.0f;
    const float ug = u_q[((int64_t)b * Hkv + kvh) * kHeadDim + i];
    int cnt = 0;
    for (int n = 0; n < Bd; ++n) cnt += (((float)n + ug) / fB) < pi;
    const float mhat = (float)cnt * (norm / fB);
#pragma unroll
    for (int g = 0; g < G; ++g) w[g] = m > 0.0f ? mhat * qv[g] / m : 0.0f;
  }
  bool keep = false;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    wout[((int64_t)b * Hq + kvh * G + g) * kHeadDim + i] = w[g];
    keep |= w[g] != 0.0f;
  }
  if (mask_out) mask_out[(int64_t)grp * kHeadDim + i] = keep ? 1 : 0;
  const uint64_t bm = __ballot(keep);
  if (lane == 0) wc[wave] = __popcll(bm);
  __syncthreads();
  const int pos = (wave ? wc[0] : 0) + __popcll(bm & ((1ull << lane) - 1ull));
  if (keep) flist[(int64_t)grp * kHeadDim + pos] = i;
  if (i == 0) fcount[grp] = wc[0] + wc[1];
}

// Scores from the selected feature rows of K^T only: s_j = scale * sum_{i in F} w_i K^T_{i,j}.
// Thread (feature slot fs, key chunk kc) reads 8 consecutive keys of one
// feature row with a 128-bit load; slots are summed in slot order.
template <typename E, int G>
__global__ __launch_bounds__(kThreads) void k_bern_score(KvView kv, KtView kt, int Hq, int Ls,
                                                          int T, float scale_log2,
                                                          const float *__restrict__ w,
                                                          const int *__restrict__ flist,
                                                          const int *__restrict__ fcount,
                                                          float2 *__restrict__ stats,
                                                          float *__restrict__ stash) {
  const int t = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int L = seq_len(kv, b);
  const int start = t * Ls;
  if (start >= L) return;
  const int nrows = min(Ls, L - start);
  const int tid = threadIdx.x;
  const int grp = b * gridDim.y + kvh;
  const int64_t row0 = (int64_t)b * Hq + kvh * G;
  __shared__ __attribute__((aligned(16))) float s[G * kSplitMax];
  __shared__ float wl[G * kHeadDim];
  __shared__ int fl[kHeadDim];
  __shared__ float mh[G];
  const int nf = fcount[grp];
  for (int o = tid; o < G * kHeadDim; o += kThreads) wl[o] = w[row0 * kHeadDim + o];
  for (int o = tid; o < nf; o += kThreads) fl[o] = flist[(int64_t)grp * kHeadDim + o];
  __syncthreads();
  const int nchunk = Ls >> 3;
  const int FS = kThreads / nchunk;
  const int kc = tid % nchunk, fs = tid / nchunk;
  const E *ktb = static_cast<const E *>(kt.kt) + (int64_t)b * kt.sb + (int64_t)kvh * kt.sh;
  const int p0 = start + kc * 8;
  const bool full = p0 + 8 <= L;
  float acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.0f;
  if (fs < FS) {
    for (int fi = fs; fi < nf; fi += FS) {
      const int i = fl[fi];
      const E *rp = ktb + (int64_t)i * kt.sd + p0;
      float kf[8];
      if (full) {
        Chunk<E>::load(rp).to_float(kf);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) kf[e] = p0 + e < L ? to_f32(rp[e]) : 0.0f;
      }
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float wv = wl[h * kHeadDim + i];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(wv, kf[e], acc[h][e]);
      }
    }
  }
  for (int r = 0; r < FS; ++r) {
    if (fs == r) {
#pragma unroll
      for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int j = kc * 8 + e;
          if (r == 0)
            s[h * kSplitMax + j] = acc[h][e];
          else
            s[h * kSplitMax + j] += acc[h][e];
        }
    }
    __syncthreads();
  }
  for (int o = tid; o < G * nrows; o += kThreads) {
    const int h = o / nrows, j = o % nrows;
    s[h * kSplitMax + j] *= scale_log2;
  }
  __syncthreads();
  finish_split_cdf<G>(s, mh, nrows, row0, T, t, (int64_t)T * Ls, start, stats, stash);
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename T>
static T *ws_at(char *ws, size_t off) {
  return reinterpret_cast<T *>(ws + off);
}

hipError_t launch_dense(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                        void *out, char *ws, hipStream_t st) {
  const dim3 grid(p.T, p.Hkv, p.B);
  float2 *stats = ws_at<float2>(ws, p.off_stats);
  float *part = ws_at<float>(ws, p.off_part);
  return with_types(p, kv.bt != nullptr, [&](auto eptr, auto gc, auto paged) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    constexpr int G = decltype(gc)::value;
    constexpr bool PG = decltype(paged)::value;
    const CallTimer tm = call_timer();
    hipExtLaunchKernelGGL(k_dense_split<E, G, PG>, grid, dim3(kThreads), 0, st, tm.start, nullptr,
                          0, kv, static_cast<const E *>(q), p.Hq, p.Ls, p.T, scale_log2, stats,
                          part);
    hipExtLaunchKernelGGL(k_merge_dense<E, G>, dim3(p.B * p.Hq), dim3(kHeadDim), 0, st, nullptr,
                          tm.stop, 0, kv, p.Hq, p.Hkv, p.Ls, p.T, stats, part,
                          static_cast<E *>(out));
    return hipGetLastError();
  });
}

template <typename E, int G, bool PG>
static hipError_t launch_value_stage(const Plan &p, const KvView &kv, bool strat, const float *u,
                                     int32_t *idx_out, void *out, char *ws, hipStream_t st) {
  const dim3 grid(p.T, p.Hkv, p.B);
  float2 *stats = ws_at<float2>(ws, p.off_stats);
  float *stash = ws_at<float>(ws, p.off_stash);
  float *offs = ws_at<float>(ws, p.off_offs);
  float *alpha = ws_at<float>(ws, p.off_alpha);
  float2 *rowst = ws_at<float2>(ws, p.off_rowst);
  float *part = ws_at<float>(ws, p.off_part);
  int *flags = ws_at<int>(ws, p.off_flag);
  const float invS = 1.0f / (float)p.S;
  k_offsets<<<p.B * p.Hq, 64, 0, st>>>(kv, p.Hq, p.Ls, p.T, stats, offs, alpha, rowst);
  if (strat)
    k_sample<E, G, PG, true><<<grid, kThreads, 0, st>>>(kv, p.Hq, p.Ls, p.T, p.S, invS, u, stash,
                                                        offs, alpha, rowst, flags, part, idx_out);
  else
    k_sample<E, G, PG, false><<<grid, kThreads, 0, st>>>(kv, p.Hq, p.Ls, p.T, p.S, invS, u, stash,
                                                         offs, alpha, rowst, flags, part, idx_out);
  hipExtLaunchKernelGGL(k_merge_sampled<E, G>, dim3(p.B * p.Hq), dim3(kHeadDim), 0, st, nullptr,
                        call_timer().stop, 0, kv, p.Hq, p.Hkv, p.Ls, p.T, p.S, invS, flags, part,
                        static_cast<E *>(out), idx_out);
  return hipGetLastError();
}

hipError_t launch_sampled(const Plan &p, const KvView &kv, const void *q, float scale_log2,
                          bool strat, const float *u, int32_t *idx_out, void *out, char *ws,
                          hipStream_t st) {
  const dim3 grid(p.T, p.Hkv, p.B);
  float2 *stats = ws_at<float2>(ws, p.off_stats);
  float *stash = ws_at<float>(ws, p.off_stash);
  return with_types(p, kv.bt != nullptr, [&](auto eptr, auto gc, auto paged) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    constexpr int G = decltype(gc)::value;
    constexpr bool PG = decltype(paged)::value;
    hipExtLaunchKernelGGL(k_score_cdf<E, G, PG>, grid, dim3(kThreads), 0, st, call_timer().start,
                          nullptr, 0, kv, static_cast<const E *>(q), p.Hq, p.Ls, p.T, scale_log2,
                          stats, stash);
    return launch_value_stage<E, G, PG>(p, kv, strat, u, idx_out, out, ws, st);
  });
}

hipError_t launch_bern_prep(const Plan &p, const void *q, int Bd, int mode, const float *u_q,
                            float *bw, int *blist, int *bn, uint8_t *mask_out, hipStream_t st,
                            hipEvent_t start) {
  return with_types(p, false, [&](auto eptr, auto gc, auto) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    constexpr int G = decltype(gc)::value;
    hipExtLaunchKernelGGL(k_bern_prep<E, G>, dim3(p.B * p.Hkv), dim3(kHeadDim), 0, st, start,
                          nullptr, 0, static_cast<const E *>(q), p.Hq, p.Hkv, Bd, mode, u_q, bw,
                          blist, bn, mask_out);
    return hipGetLastError();
  });
}

hipError_t launch_bernoulli(const Plan &p, const KvView &kv, const KtView &kt, const void *q,
                            float scale_log2, int Bd, int mode, const float *u_q, const float *u,
                            int32_t *idx_out, uint8_t *mask_out, void *out, char *ws,
                            hipStream_t st) {
  const dim3 grid(p.T, p.Hkv, p.B);
  float2 *stats = ws_at<float2>(ws, p.off_stats);
  float *stash = ws_at<float>(ws, p.off_stash);
  float *bw = ws_at<float>(ws, p.off_bw);
  int *blist = ws_at<int>(ws, p.off_blist);
  int *bn = ws_at<int>(ws, p.off_bn);
  return with_types(p, false, [&](auto eptr, auto gc, auto) -> hipError_t {
    using E = std::remove_pointer_t<decltype(eptr)>;
    constexpr int G = decltype(gc)::value;
    hipExtLaunchKernelGGL(k_bern_prep<E, G>, dim3(p.B * p.Hkv), dim3(kHeadDim), 0, st,
                          call_timer().start, nullptr, 0, static_cast<const E *>(q), p.Hq, p.Hkv,
                          Bd, mode, u_q, bw, blist, bn, mask_out);
    k_bern_score<E, G><<<grid, kThreads, 0, st>>>(kv, kt, p.Hq, p.Ls, p.T, scale_log2, bw, blist,
                                                  bn, stats, stash);
    return launch_value_stage<E, G, false>(p, kv, false, u, idx_out, out, ws, st);
  });
}

__global__ void k_fill_zero(uint4 *p, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0, 0, 0, 0);
}

hipError_t launch_zero(void *ws, size_t bytes, hipStream_t st) {
  const size_t n16 = bytes / 16;
  if (n16) {
    const size_t blocks = (n16 + 255) / 256 < 4096 ? (n16 + 255) / 256 : 4096;
    k_fill_zero<<<(unsigned)blocks, 256, 0, st>>>(static_cast<uint4 *>(ws), n16);
  }
  return hipGetLastError();
}

}  // namespace santa
