/*
 * santa_oracle.c -- plain double-precision CPU oracle for one decode step of
 * SANTA / S2ANTA attention ("Stochastic Sparse Attention for Memory-Bound
 * Inference", arXiv 2605.01910).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may load this
 * library: only the tests, the package smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no code, header, table or helper with the
 * GPU library; inputs reach it as raw arrays produced by the seeded input
 * generator.
 *
 * Every function below is one step of the method written from its plain
 * definition, in double precision, one query row at a time, with no blocking,
 * fusion or reordering:
 *
 *   orc_scores            s_j = scale * <q, k_j>                  (Sec. 2, SDPA equation)
 *   orc_softmax           p = softmax(s), max-shifted             (Sec. 2, SDPA equation)
 *   orc_weighted_sum      sum_j p_j v_j  (dense AV)               (Sec. 2, SDPA equation)
 *   orc_cdf               F(j) = sum_{i<=j} p_i                   (Sec. 2.1, "Construction")
 *   orc_thresholds        T_m for systematic / stratified / iid   (Sec. 2.1; Sec. 2 i.i.d. draws)
 *   orc_inverse_cdf       J = F^{-1}(T): the j with F(j-1) <= T < F(j)
 *                                                                  (App. A, "Unbiasedness of S2ANTA")
 *   orc_gather_mean       (1/S) sum_m v_{J_m}                     (Sec. 2, Eq. "stochastic-add-only-attn")
 *   orc_bernoulli_weights ternary / mean-group query weights      (Sec. 5, Eq. "qk_estimator";
 *                                                                  App. C, Eq. "mean_group_query")
 *   orc_fp8_e4m3          OCP FP8 E4M3 code -> value (a quantised cache; Sec. 1,
 *                         Related Work: complementary to SANTA)
 *   orc_flash             S2ANTA-flash: per-tile systematic sampling with a
 *                         fixed budget, tiles merged by their softmax mass
 *                                                                  (Sec. 3.3; App. "S2ANTA-Flash
 *                                                                  Pseudocode", Kernels 1 and 2)
 *   orc_decode            all of the above over the rows of a batch
 *   orc_decode_flash      orc_flash over the rows of a batch
 *
 * Readings of points the paper leaves open:
 *   - F^{-1}(T) counts the CDF values <= T ("right" side of a boundary), so a
 *     key of zero mass is never chosen; a threshold at or above the last CDF
 *     value (rounding) takes the last key.
 *   - Systematic thresholds are T_m = (m + u)/S with one u in [0,1) per row
 *     (U = u/S is uniform on [0, 1/S)); stratified ones are (m + u_m)/S.
 *   - The i.i.d. estimator draws its S categorical samples by inverting the
 *     CDF at S sorted independent uniforms (same multiset as S i.i.d. draws).
 *   - Bernoulli decisions b = [u < pi] are taken in float32, the precision of
 *     the inputs, so that a GPU taking the same decision in float32 agrees bit
 *     for bit; everything after the decision is double precision.
 *   - A row with zero context length has no attention distribution: its
 *     output is zero and its indices are -1.
 *
 * Element arrays hold bfloat16 bit patterns (uint16, kind 0), float32 values
 * (kind 1) or float64 values (kind 2); all widen to double exactly.  A cache
 * of OCP FP8 E4M3 codes with per-(batch, KV head) scales is decoded to
 * float64 first (orc_fp8_e4m3), one (batch, KV head) slab per row.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Exact widening of one stored element to double (kind: 0 bfloat16 bits,
 * 1 float32, 2 float64). */
static double elem(const void *base, int is_f32, int64_t i) {
  if (is_f32 == 2) return ((const double *)base)[i];
  if (is_f32) return (double)((const float *)base)[i];
  uint32_t w = (uint32_t)((const uint16_t *)base)[i] << 16;
  float f;
  memcpy(&f, &w, sizeof f);
  return (double)f;
}

/* Bytes per element of kind 0, 1, 2. */
static size_t esize(int kind) { return kind == 2 ? 8 : kind == 1 ? 4 : 2; }

/* Same widening, but to float (used where a decision is taken in float32). */
static float elemf(const void *base, int is_f32, int64_t i) {
  if (is_f32) return ((const float *)base)[i];
  uint32_t w = (uint32_t)((const uint16_t *)base)[i] << 16;
  float f;
  memcpy(&f, &w, sizeof f);
  return f;
}

/* OCP FP8 E4M3 ("E4M3FN") code -> value, from the format's definition: bit 7
 * the sign, bits 6..3 the exponent field e (bias 7), bits 2..0 the mantissa
 * field m.  e = 0: subnormal, m/8 * 2^-6; e = 15 and m = 7: NaN (the format
 * has no infinities); otherwise (1 + m/8) * 2^(e - 7).  Largest finite value
 * 448, smallest subnormal 2^-9.  Keys and values stored this way are a
 * quantised KV cache, which the paper treats as complementary to SANTA
 * (Sec. 1; Related Work). */
double orc_fp8_e4m3(uint8_t code) {
  const int sign = code >> 7, e = (code >> 3) & 15, m = code & 7;
  double v;
  if (e == 15 && m == 7)
    v = NAN;
  else if (e == 0)
    v = ldexp((double)m / 8.0, -6);
  else
    v = ldexp(1.0 + (double)m / 8.0, e - 7);
  return sign ? -v : v;
}

void orc_fp8_e4m3_decode(const uint8_t *codes, int64_t n, double *out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_fp8_e4m3(codes[i]);
}

/* Score stage (Sec. 2, SDPA equation): s_j = scale * sum_i w_i k_{j,i} for j < L, with
 * the query given in double; key j starts at element j*row_stride of k. */
void orc_scores(const double *w, int d, const void *k, int k_f32, int64_t row_stride, int L,
                double scale, double *s) {
  for (int j = 0; j < L; ++j) {
    double acc = 0.0;
    for (int i = 0; i < d; ++i) acc += w[i] * elem(k, k_f32, (int64_t)j * row_stride + i);
    s[j] = scale * acc;
  }
}

/* Softmax of the SDPA equation (Sec. 2) in its numerically stable form: p_j = exp(s_j - m) / Z,
 * m = max_j s_j, Z = sum_j exp(s_j - m). */
void orc_softmax(const double *s, int L, double *p) {
  if (L <= 0) return;
  double m = s[0];
  for (int j = 1; j < L; ++j)
    if (s[j] > m) m = s[j];
  double Z = 0.0;
  for (int j = 0; j < L; ++j) {
    p[j] = exp(s[j] - m);
    Z += p[j];
  }
  for (int j = 0; j < L; ++j) p[j] /= Z;
}

/* Dense value aggregation AV (Sec. 2, SDPA equation): out_i = sum_j p_j v_{j,i}. */
void orc_weighted_sum(const double *p, const void *v, int v_f32, int64_t row_stride, int L, int d,
                      double *out) {
  for (int i = 0; i < d; ++i) out[i] = 0.0;
  for (int j = 0; j < L; ++j)
    for (int i = 0; i < d; ++i) out[i] += p[j] * elem(v, v_f32, (int64_t)j * row_stride + i);
}

/* CDF of the attention distribution (Sec. 2.1, "Construction"): F(j) = sum_{i<=j} p_i,
 * accumulated in index order. */
void orc_cdf(const double *p, int L, double *C) {
  double acc = 0.0;
  for (int j = 0; j < L; ++j) {
    acc += p[j];
    C[j] = acc;
  }
}

/* Sampling thresholds on [0,1) (Sec. 2.1, "Construction"):
 *   scheme 0, systematic:  T_m = U + m/S with U = u[0]/S uniform on [0, 1/S);
 *   scheme 1, stratified:  T_m uniform on I_m = [m/S, (m+1)/S): T_m = (m + u[m])/S;
 *   scheme 2, i.i.d.:      S independent uniforms u[0..S) in increasing order, whose
 *                          inverse-CDF images are S i.i.d. categorical draws (Sec. 2);
 *   scheme 3, i.i.d. by spacings: the same S sorted uniforms built from S + 1
 *                          independent uniforms u[0..S] without a sort: with
 *                          E_i = -ln(1 - u_i) (unit exponentials), T_m = C_m / C_S,
 *                          C_m = sum_{i<=m} E_i -- the normalised partial sums of
 *                          S + 1 exponentials are distributed as the order statistics
 *                          of S independent uniforms (Renyi's representation). */
static int cmp_double(const void *a, const void *b) {
  double x = *(const double *)a, y = *(const double *)b;
  return (x > y) - (x < y);
}

void orc_thresholds(int scheme, const float *u, int S, double *T) {
  if (scheme == 3) {
    double C = 0.0;
    for (int m = 0; m < S; ++m) {
      C += -log(1.0 - (double)u[m]);
      T[m] = C;
    }
    const double total = C - log(1.0 - (double)u[S]);
    for (int m = 0; m < S; ++m) T[m] /= total;
    return;
  }
  for (int m = 0; m < S; ++m) {
    if (scheme == 0)
      T[m] = ((double)m + (double)u[0]) / (double)S;
    else if (scheme == 1)
      T[m] = ((double)m + (double)u[m]) / (double)S;
    else
      T[m] = (double)u[m];
  }
  if (scheme == 2) qsort(T, (size_t)S, sizeof(double), cmp_double);
}

/* Inverse CDF (App. A, "Unbiasedness of S2ANTA"): J = F^{-1}(T) is the key j
 * whose interval [F(j-1), F(j)) contains T, i.e. J = #{j : F(j) <= T}, taken as the
 * last key L-1 when T is at or above F(L-1). */
void orc_inverse_cdf(const double *C, int L, const double *T, int S, int32_t *idx) {
  for (int m = 0; m < S; ++m) {
    int count = 0;
    for (int j = 0; j < L; ++j)
      if (C[j] <= T[m]) ++count;
    idx[m] = count < L ? count : L - 1;
  }
}

/* SANTA value estimate (Sec. 2, Eq. "stochastic-add-only-attn"):
 * out_i = (1/S) sum_m v_{idx_m, i}. */
void orc_gather_mean(const void *v, int v_f32, int64_t row_stride, int d, const int32_t *idx,
                     int S, double *out) {
  for (int i = 0; i < d; ++i) out[i] = 0.0;
  for (int m = 0; m < S; ++m)
    for (int i = 0; i < d; ++i) out[i] += elem(v, v_f32, (int64_t)idx[m] * row_stride + i);
  for (int i = 0; i < d; ++i) out[i] /= (double)S;
}

/* Bernoulli query weights for one GQA group of G heads (query rows q_g at
 * q + g*d), returned as w[g*d + i] such that the estimated score is
 * p_hat = scale * <w_g, k_j>.
 *
 * mode 0, per-head ternary query (Sec. 5, Eq. "qk_estimator"; App. C):
 *   norm = max_i |q_i|, pi_i = |q_i| / norm, b_i^(n) ~ Bernoulli(pi_i),
 *   w_i = (norm / B) * sign(q_i) * sum_n b_i^(n).
 * mode 1, mean group query (Sec. 5, "Mean Group Query", Eq. "mean_group_query"; App. C, GQA subsection):
 *   m_i = mean_g |q_{g,i}|, norm = max_i m_i, pi_i = m_i / norm,
 *   m_hat_i = (norm / B) * sum_n b_i^(n),  w_{g,i} = m_hat_i * q_{g,i} / m_i  (0 if m_i = 0).
 *
 * Draws: iid = 0 uses one uniform per feature and the stratified count
 * #{n < B : (n + u_i)/B < pi_i}; iid = 1 uses B independent uniforms per feature,
 * u[n*d + i], and counts #{n : u^(n)_i < pi_i}.  u is laid out per head
 * (mode 0: G blocks) or per group (mode 1: one block).  The decision and the
 * quantities it depends on (|q|, m, norm, pi) are float32.
 * mask[i] = 1 when some head of the group has w_{g,i} != 0. */
void orc_bernoulli_weights(const void *q, int q_f32, int G, int d, const float *u, int B,
                           int iid, int mode, double *w, uint8_t *mask) {
  for (int i = 0; i < d; ++i) mask[i] = 0;
  if (mode == 0) {
    for (int g = 0; g < G; ++g) {
      float norm = 0.0f;
      for (int i = 0; i < d; ++i) {
        float a = fabsf(elemf(q, q_f32, (int64_t)g * d + i));
        if (a > norm) norm = a;
      }
      const float *ug = u + (int64_t)g * d * (iid ? B : 1);
      for (int i = 0; i < d; ++i) {
        float qi = elemf(q, q_f32, (int64_t)g * d + i);
        float pi = norm > 0.0f ? fabsf(qi) / norm : 0.0f;
        int c = 0;
        for (int n = 0; n < B; ++n) {
          int hit = iid ? (ug[(int64_t)n * d + i] < pi) : ((((float)n + ug[i]) / (float)B) < pi);
          c += hit;
        }
        double sgn = qi > 0.0f ? 1.0 : (qi < 0.0f ? -1.0 : 0.0);
        w[(int64_t)g * d + i] = ((double)norm / (double)B) * sgn * (double)c;
        if (w[(int64_t)g * d + i] != 0.0) mask[i] = 1;
      }
    }
  } else {
    float *m = (float *)malloc(sizeof(float) * (size_t)d);
    float norm = 0.0f;
    for (int i = 0; i < d; ++i) {
      float acc = 0.0f;
      for (int g = 0; g < G; ++g) acc += fabsf(elemf(q, q_f32, (int64_t)g * d + i));
      m[i] = acc / (float)G;
      if (m[i] > norm) norm = m[i];
    }
    for (int i = 0; i < d; ++i) {
      float pi = norm > 0.0f ? m[i] / norm : 0.0f;
      int c = 0;
      for (int n = 0; n < B; ++n) {
        int hit = iid ? (u[(int64_t)n * d + i] < pi) : ((((float)n + u[i]) / (float)B) < pi);
        c += hit;
      }
      double mhat = ((double)norm / (double)B) * (double)c;
      for (int g = 0; g < G; ++g) {
        double qg = elem(q, q_f32, (int64_t)g * d + i);
        double wg = m[i] > 0.0f ? mhat * qg / (double)m[i] : 0.0;
        w[(int64_t)g * d + i] = wg;
        if (wg != 0.0) mask[i] = 1;
      }
    }
    free(m);
  }
}

/* S2ANTA-flash for one query row (Sec. 3.3; App. "S2ANTA-Flash Pseudocode").
 * Kernel 1, per tile t = [t*tile, min((t+1)*tile, L)): m_t = max s, e_j =
 * exp(s_j - m_t), l_t = sum e_j; S_tile systematic draws on the tile's own
 * distribution e_j / l_t with the tile's uniform a[t] (thresholds (i + a[t]) /
 * S_tile, inverse CDF as in orc_inverse_cdf); tile estimate O_t = (1/S_tile)
 * sum_i v_{J_{t,i}}.  Kernel 2: W_t = exp(m_t - m*) l_t, Z = sum_t W_t,
 * O = (1/Z) sum_t W_t O_t.
 * s: scores [L]; v: value rows (row j at j*row_stride); a: [T] uniforms,
 * T = ceil(L / tile).  Outputs: out [d]; idx [T*S_tile] logical indices, tile
 * by tile (optional); wt [T] = W_t / Z (optional); tile_out [T*d] = O_t
 * (optional); cdf [L] tile-local CDF values (optional). */
void orc_flash(const double *s, const void *v, int v_f32, int64_t row_stride, int L, int d,
               int tile, int S_tile, const float *a, int32_t *idx, double *out, double *wt,
               double *tile_out, double *cdf) {
  const int T = (L + tile - 1) / tile;
  double *m = (double *)malloc(sizeof(double) * (size_t)T);
  double *l = (double *)malloc(sizeof(double) * (size_t)T);
  double *p = (double *)malloc(sizeof(double) * (size_t)tile);
  double *C = (double *)malloc(sizeof(double) * (size_t)tile);
  double *thr = (double *)malloc(sizeof(double) * (size_t)S_tile);
  int32_t *ix = (int32_t *)malloc(sizeof(int32_t) * (size_t)S_tile);
  double *ot = (double *)malloc(sizeof(double) * (size_t)d * (size_t)T);
  for (int t = 0; t < T; ++t) {
    const int j0 = t * tile, n = (L - j0 < tile) ? L - j0 : tile;
    /* tile statistics and the tile's own distribution */
    m[t] = s[j0];
    for (int j = 1; j < n; ++j)
      if (s[j0 + j] > m[t]) m[t] = s[j0 + j];
    l[t] = 0.0;
    for (int j = 0; j < n; ++j) l[t] += exp(s[j0 + j] - m[t]);
    orc_softmax(s + j0, n, p);
    orc_cdf(p, n, C);
    if (cdf)
      for (int j = 0; j < n; ++j) cdf[j0 + j] = C[j];
    /* systematic draws inside the tile and the tile estimate */
    orc_thresholds(0, a + t, S_tile, thr);
    orc_inverse_cdf(C, n, thr, S_tile, ix);
    orc_gather_mean((const char *)v + (int64_t)j0 * row_stride * (int64_t)esize(v_f32), v_f32, row_stride,
                    d, ix, S_tile, ot + (int64_t)t * d);
    if (idx)
      for (int i = 0; i < S_tile; ++i) idx[(int64_t)t * S_tile + i] = j0 + ix[i];
  }
  /* merge: tiles weighted by W_t = exp(m_t - m*) l_t */
  double ms = m[0];
  for (int t = 1; t < T; ++t)
    if (m[t] > ms) ms = m[t];
  double Z = 0.0;
  for (int t = 0; t < T; ++t) Z += exp(m[t] - ms) * l[t];
  for (int i = 0; i < d; ++i) out[i] = 0.0;
  for (int t = 0; t < T; ++t) {
    const double w = exp(m[t] - ms) * l[t] / Z;
    if (wt) wt[t] = w;
    for (int i = 0; i < d; ++i) out[i] += w * ot[(int64_t)t * d + i];
  }
  if (tile_out) memcpy(tile_out, ot, sizeof(double) * (size_t)d * (size_t)T);
  free(m);
  free(l);
  free(p);
  free(C);
  free(thr);
  free(ix);
  free(ot);
}

/* ------------------------------------------------------------------------- */
/* Batch driver                                                              */
/* ------------------------------------------------------------------------- */

typedef struct {
  int32_t B, Hq, Hkv, d, n_max;
  int32_t is_f32;        /* element type of q (and of k, v when kv_fp8 is 0) */
  const void *q;         /* [B, Hq, d] */
  const void *k;         /* logical keys: element (b, j, kv, i) at b*sb + j*sn + kv*sh + i */
  const void *v;         /* logical values, same strides */
  int64_t sb, sn, sh;
  const int32_t *ctx_len; /* [B] */
  double scale;
  int32_t kv_fp8;        /* 1: k, v hold FP8 E4M3 codes scaled by k_scale / v_scale */
  const float *k_scale;  /* [B, Hkv] */
  const float *v_scale;  /* [B, Hkv] */
} orc_problem_t;

/* The keys and values of row (b, kv) as arrays the step functions read: the
 * stored arrays themselves (kind is_f32, row stride sn), or, for an FP8
 * cache, their decoded values times the row's scales in kd / vd (float64,
 * row stride d). */
static void kv_rows(const orc_problem_t *P, int b, int kv, int L, double *kd, double *vd,
                    const void **k_out, const void **v_out, int *kind, int64_t *stride) {
  const int64_t base = (int64_t)b * P->sb + (int64_t)kv * P->sh;
  if (!P->kv_fp8) {
    const size_t esz = P->is_f32 ? 4 : 2;
    *k_out = (const char *)P->k + base * (int64_t)esz;
    *v_out = (const char *)P->v + base * (int64_t)esz;
    *kind = P->is_f32;
    *stride = P->sn;
    return;
  }
  const double ks = (double)P->k_scale[(int64_t)b * P->Hkv + kv];
  const double vs = (double)P->v_scale[(int64_t)b * P->Hkv + kv];
  const uint8_t *kc = (const uint8_t *)P->k + base, *vc = (const uint8_t *)P->v + base;
  for (int j = 0; j < L; ++j)
    for (int i = 0; i < P->d; ++i) {
      kd[(int64_t)j * P->d + i] = ks * orc_fp8_e4m3(kc[(int64_t)j * P->sn + i]);
      vd[(int64_t)j * P->d + i] = vs * orc_fp8_e4m3(vc[(int64_t)j * P->sn + i]);
    }
  *k_out = kd;
  *v_out = vd;
  *kind = 2;
  *stride = P->d;
}

enum { ORC_DENSE = 0, ORC_SYSTEMATIC = 1, ORC_STRATIFIED = 2, ORC_IID = 3, ORC_BERNOULLI_SYS = 4,
       ORC_IID_SPACINGS = 5 };

/* One decode step for the listed rows (row = b*Hq + h; rows == NULL means all):
 *   kind dense:        out = AV
 *   kind systematic:   u[b*Hq + h], thresholds (m+u)/S
 *   kind stratified:   u[(b*Hq + h)*S + m]
 *   kind iid:          u[(b*Hq + h)*S + m], sorted
 *   kind iid spacings: u[(b*Hq + h)*(S+1) + i], thresholds by exponential spacings
 *   kind bernoulli:    Bernoulli scores from u_q (mode 0: [B, Hq, d*(iid?B:1)]; mode 1:
 *                      [B, Hkv, d*(iid?B:1)]) followed by systematic sampling with u[b*Hq + h].
 * Outputs are compact over the listed rows: out[r*d], idx[r*S] (sampled kinds),
 * cdf[r*n_max] (optional), and for bernoulli w[r*d] and mask[r*d] (optional).
 * Returns the number of OpenMP threads used. */
int orc_decode(const orc_problem_t *P, int kind, int S, const float *u, const float *u_q,
               int B_draws, int mode, int iid_draws, int nrows, const int32_t *rows, double *out,
               int32_t *idx, double *cdf, double *w_out, uint8_t *mask_out) {
  const int G = P->Hq / P->Hkv;
  const int total = nrows > 0 ? nrows : P->B * P->Hq;
  int threads = 1;
#pragma omp parallel
  {
#ifdef _OPENMP
#pragma omp single
    threads = omp_get_num_threads();
#endif
    double *qd = (double *)malloc(sizeof(double) * (size_t)P->d);
    double *wg = (double *)malloc(sizeof(double) * (size_t)P->d * (size_t)G);
    uint8_t *mk = (uint8_t *)malloc((size_t)P->d);
    double *s = (double *)malloc(sizeof(double) * (size_t)(P->n_max > 0 ? P->n_max : 1));
    double *p = (double *)malloc(sizeof(double) * (size_t)(P->n_max > 0 ? P->n_max : 1));
    double *C = (double *)malloc(sizeof(double) * (size_t)(P->n_max > 0 ? P->n_max : 1));
    double *T = (double *)malloc(sizeof(double) * (size_t)(S > 0 ? S : 1));
    const size_t slab = P->kv_fp8 ? (size_t)(P->n_max > 0 ? P->n_max : 1) * (size_t)P->d : 1;
    double *kd = (double *)malloc(sizeof(double) * slab);
    double *vd = (double *)malloc(sizeof(double) * slab);
#pragma omp for schedule(dynamic, 1)
    for (int r = 0; r < total; ++r) {
      const int row = rows ? rows[r] : r;
      const int b = row / P->Hq, h = row % P->Hq, kv = h / G;
      const int L = P->ctx_len[b];
      double *o = out + (int64_t)r * P->d;
      if (L <= 0) {
        for (int i = 0; i < P->d; ++i) o[i] = 0.0;
        if (idx && kind != ORC_DENSE)
          for (int m = 0; m < S; ++m) idx[(int64_t)r * S + m] = -1;
        continue;
      }
      /* query weights */
      const double *wq = qd;
      if (kind == ORC_BERNOULLI_SYS) {
        const float *ub = mode == 0
                              ? u_q + ((int64_t)b * P->Hq + (int64_t)kv * G) * P->d * (iid_draws ? B_draws : 1)
                              : u_q + ((int64_t)b * P->Hkv + kv) * P->d * (iid_draws ? B_draws : 1);
        const size_t esz = P->is_f32 ? 4 : 2;
        const char *qg = (const char *)P->q + ((int64_t)b * P->Hq + (int64_t)kv * G) * P->d * esz;
        orc_bernoulli_weights(qg, P->is_f32, G, P->d, ub, B_draws, iid_draws, mode, wg, mk);
        wq = wg + (int64_t)(h - kv * G) * P->d;
        if (w_out)
          for (int i = 0; i < P->d; ++i) w_out[(int64_t)r * P->d + i] = wq[i];
        if (mask_out)
          for (int i = 0; i < P->d; ++i) mask_out[(int64_t)r * P->d + i] = mk[i];
      } else {
        for (int i = 0; i < P->d; ++i) qd[i] = elem(P->q, P->is_f32, ((int64_t)b * P->Hq + h) * P->d + i);
      }
      const void *kb, *vb;
      int kvk;
      int64_t rs;
      kv_rows(P, b, kv, L, kd, vd, &kb, &vb, &kvk, &rs);
      orc_scores(wq, P->d, kb, kvk, rs, L, P->scale, s);
      orc_softmax(s, L, p);
      if (kind == ORC_DENSE) {
        orc_weighted_sum(p, vb, kvk, rs, L, P->d, o);
        continue;
      }
      orc_cdf(p, L, C);
      if (cdf)
        for (int j = 0; j < L; ++j) cdf[(int64_t)r * P->n_max + j] = C[j];
      if (kind == ORC_SYSTEMATIC || kind == ORC_BERNOULLI_SYS)
        orc_thresholds(0, u + (int64_t)row, S, T);
      else if (kind == ORC_IID_SPACINGS)
        orc_thresholds(3, u + (int64_t)row * (S + 1), S, T);
      else
        orc_thresholds(kind == ORC_STRATIFIED ? 1 : 2, u + (int64_t)row * S, S, T);
      int32_t *ix = idx + (int64_t)r * S;
      orc_inverse_cdf(C, L, T, S, ix);
      orc_gather_mean(vb, kvk, rs, P->d, ix, S, o);
    }
    free(kd);
    free(vd);
    free(qd);
    free(wg);
    free(mk);
    free(s);
    free(p);
    free(C);
    free(T);
  }
  return threads;
}

/* orc_flash over the listed rows (row = b*Hq + h; rows == NULL means all):
 * u[(b*Hq + h)*T_max + t] is the uniform of tile t, T_max = ceil(n_max / tile).
 * Outputs compact over the listed rows: out[r*d]; idx[r*T_max*S_tile] (tiles at
 * or past ceil(L_b / tile) hold -1); wt[r*T_max] (optional, 0 past the row's
 * tiles); cdf[r*n_max] tile-local CDF (optional).  Returns the thread count. */
int orc_decode_flash(const orc_problem_t *P, int tile, int S_tile, const float *u, int nrows,
                     const int32_t *rows, double *out, int32_t *idx, double *wt, double *cdf) {
  const int G = P->Hq / P->Hkv;
  const int total = nrows > 0 ? nrows : P->B * P->Hq;
  const int Tm = (P->n_max + tile - 1) / tile;
  int threads = 1;
#pragma omp parallel
  {
#ifdef _OPENMP
#pragma omp single
    threads = omp_get_num_threads();
#endif
    double *qd = (double *)malloc(sizeof(double) * (size_t)P->d);
    double *s = (double *)malloc(sizeof(double) * (size_t)(P->n_max > 0 ? P->n_max : 1));
    const size_t slab = P->kv_fp8 ? (size_t)(P->n_max > 0 ? P->n_max : 1) * (size_t)P->d : 1;
    double *kd = (double *)malloc(sizeof(double) * slab);
    double *vd = (double *)malloc(sizeof(double) * slab);
#pragma omp for schedule(dynamic, 1)
    for (int r = 0; r < total; ++r) {
      const int row = rows ? rows[r] : r;
      const int b = row / P->Hq, h = row % P->Hq, kv = h / G;
      const int L = P->ctx_len[b];
      double *o = out + (int64_t)r * P->d;
      int32_t *ix = idx ? idx + (int64_t)r * Tm * S_tile : NULL;
      double *w = wt ? wt + (int64_t)r * Tm : NULL;
      if (ix)
        for (int i = 0; i < Tm * S_tile; ++i) ix[i] = -1;
      if (w)
        for (int t = 0; t < Tm; ++t) w[t] = 0.0;
      if (L <= 0) {
        for (int i = 0; i < P->d; ++i) o[i] = 0.0;
        continue;
      }
      for (int i = 0; i < P->d; ++i) qd[i] = elem(P->q, P->is_f32, ((int64_t)b * P->Hq + h) * P->d + i);
      const void *kb, *vb;
      int kvk;
      int64_t rs;
      kv_rows(P, b, kv, L, kd, vd, &kb, &vb, &kvk, &rs);
      orc_scores(qd, P->d, kb, kvk, rs, L, P->scale, s);
      orc_flash(s, vb, kvk, rs, L, P->d, tile, S_tile, u + (int64_t)row * Tm, ix, o, w, NULL,
                cdf ? cdf + (int64_t)r * P->n_max : NULL);
    }
    free(kd);
    free(vd);
    free(qd);
    free(s);
  }
  return threads;
}
