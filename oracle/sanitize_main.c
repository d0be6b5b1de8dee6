/*
 * sanitize_main.c -- drives every entry point of the CPU oracle on small
 * ragged inputs, for a build under AddressSanitizer and
 * UndefinedBehaviorSanitizer (tests/test_oracle_sanitize.py).  Test
 * infrastructure only, like the oracle itself.  Prints a checksum of the
 * outputs so that nothing is optimised away.
 */
#include <stdio.h>

#include "santa_oracle.c"

static uint32_t lcg_state = 12345u;
static float rnd01(void) {
  lcg_state = lcg_state * 1664525u + 1013904223u;
  return (float)(lcg_state >> 8) * (1.0f / 16777216.0f);
}
static float rnd_normalish(void) { return (rnd01() + rnd01() + rnd01() - 1.5f) * 2.0f; }

static uint16_t to_bf16(float x) {
  uint32_t u;
  memcpy(&u, &x, sizeof u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static double checksum = 0.0;

static void run_problem(int is_f32, const int32_t *ctx, int B, int Hq, int Hkv, int d, int n) {
  const size_t nq = (size_t)B * Hq * d, nkv = (size_t)B * n * Hkv * d;
  const size_t esz = is_f32 ? 4 : 2;
  void *q = malloc(nq * esz), *k = malloc(nkv * esz), *v = malloc(nkv * esz);
  for (size_t i = 0; i < nq; ++i) {
    const float x = rnd_normalish();
    if (is_f32) ((float *)q)[i] = x; else ((uint16_t *)q)[i] = to_bf16(x);
  }
  for (size_t i = 0; i < nkv; ++i) {
    const float x = rnd_normalish(), y = rnd_normalish();
    if (is_f32) { ((float *)k)[i] = x; ((float *)v)[i] = y; }
    else { ((uint16_t *)k)[i] = to_bf16(x); ((uint16_t *)v)[i] = to_bf16(y); }
  }
  orc_problem_t P = {B, Hq, Hkv, d, n, is_f32, q, k, v, (int64_t)n * Hkv * d, (int64_t)Hkv * d, d,
                     ctx, 0.25};
  const int rows_all = B * Hq;
  const int S = 7;
  float *u = (float *)malloc(sizeof(float) * (size_t)rows_all * (S + 1));
  for (int i = 0; i < rows_all * (S + 1); ++i) u[i] = rnd01();
  const int G = Hq / Hkv;
  const int Bd = 3;
  float *uq = (float *)malloc(sizeof(float) * (size_t)B * Hq * d * Bd);
  for (int i = 0; i < B * Hq * d * Bd; ++i) uq[i] = rnd01();
  /* outputs hold every row, or the 3 rows of the subset below */
  const int nout = rows_all > 3 ? rows_all : 3;
  double *out = (double *)malloc(sizeof(double) * (size_t)nout * d);
  int32_t *idx = (int32_t *)malloc(sizeof(int32_t) * (size_t)nout * S);
  double *cdf = (double *)malloc(sizeof(double) * (size_t)nout * n);
  double *w = (double *)malloc(sizeof(double) * (size_t)nout * d);
  uint8_t *mask = (uint8_t *)malloc((size_t)nout * d);
  const int32_t sub[3] = {rows_all - 1, 0, G};
  for (int kind = ORC_DENSE; kind <= ORC_IID_SPACINGS; ++kind) {
    for (int mode = 0; mode < (kind == ORC_BERNOULLI_SYS ? 2 : 1); ++mode)
      for (int iid = 0; iid < (kind == ORC_BERNOULLI_SYS ? 2 : 1); ++iid)
        for (int pass = 0; pass < 2; ++pass) {
          const int nr = pass ? 3 : 0;
          orc_decode(&P, kind, S, u, uq, Bd, mode, iid, nr, pass ? sub : NULL, out, idx, cdf, w,
                     mask);
          const int rows = pass ? 3 : rows_all;
          for (int i = 0; i < rows * d; ++i) checksum += out[i];
          if (kind != ORC_DENSE)
            for (int i = 0; i < rows * S; ++i) checksum += idx[i];
        }
  }
  const int tile = 8, St = 3, Tm = (n + tile - 1) / tile;
  float *ut = (float *)malloc(sizeof(float) * (size_t)rows_all * Tm);
  for (int i = 0; i < rows_all * Tm; ++i) ut[i] = rnd01();
  int32_t *fidx = (int32_t *)malloc(sizeof(int32_t) * (size_t)nout * Tm * St);
  double *wt = (double *)malloc(sizeof(double) * (size_t)nout * Tm);
  orc_decode_flash(&P, tile, St, ut, 0, NULL, out, fidx, wt, cdf);
  orc_decode_flash(&P, tile, St, ut, 3, sub, out, fidx, wt, NULL);
  for (int i = 0; i < 3 * d; ++i) checksum += out[i];
  free(q); free(k); free(v); free(u); free(uq); free(out); free(idx); free(cdf); free(w);
  free(mask); free(ut); free(fidx); free(wt);
}

int main(void) {
  /* single-row steps */
  double s[5] = {0.5, -1.0, 2.0, 2.0, 0.0}, p[5], C[5], T[4];
  orc_softmax(s, 5, p);
  orc_cdf(p, 5, C);
  const float u1[5] = {0.3f, 0.9f, 0.0f, 0.99999994f, 0.5f};
  for (int scheme = 0; scheme < 4; ++scheme) {
    int32_t ix[4];
    orc_thresholds(scheme, u1, 4, T);
    orc_inverse_cdf(C, 5, T, 4, ix);
    for (int m = 0; m < 4; ++m) checksum += ix[m];
  }
  const int32_t ctx_a[3] = {37, 1, 0};
  run_problem(0, ctx_a, 3, 4, 2, 16, 37);
  run_problem(1, ctx_a, 3, 8, 1, 8, 37);
  const int32_t ctx_b[1] = {64};
  run_problem(0, ctx_b, 1, 2, 2, 16, 64);
  printf("checksum %.17g\n", checksum);
  return 0;
}
