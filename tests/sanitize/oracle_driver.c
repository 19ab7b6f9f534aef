/*
 * Exercises the fp64 oracle (oracle/oracle.c) under AddressSanitizer and
 * UndefinedBehaviorSanitizer: full outputs and row sampling, bf16 and 8-bit
 * caches with scales, several tokens with lengths below the token count,
 * context-only samples, every error path. Checks one closed form (q = 0:
 * every output row is the mean of the rows it sees) so that the run also
 * computes something meaningful. Exit status 0 when everything holds.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_attention_kv_fp64(int b, int h, int g, int d, int m_c, int m_d_max, int n,
                             double scale, int kv_type, const uint16_t *q, const void *Kc,
                             const void *Vc, const void *Kd, const void *Vd, const int32_t *lens,
                             const float *k_scale, const float *v_scale, double *out,
                             int nthreads);
int oracle_attention_kv_rows_fp64(int b, int h, int g, int d, int m_c, int m_d_max, int n,
                                  double scale, int kv_type, const uint16_t *q, const void *Kc,
                                  const void *Vc, const void *Kd, const void *Vd,
                                  const int32_t *lens, const float *k_scale,
                                  const float *v_scale, int nrows, const int32_t *row_i,
                                  const int32_t *row_j, const int32_t *row_t, double *out,
                                  int nthreads);
double oracle_code_value(int kv_type, int code);

static uint32_t state = 12345u;
static uint32_t next(void) {
  state = state * 1664525u + 1013904223u;
  return state >> 8;
}
static uint16_t bf16_of(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  return (uint16_t)(u >> 16);
}
static float rnd(void) { return (float)(next() % 2001) / 1000.0f - 1.0f; }

static int failures = 0;
#define CHECK(c, ...)                 \
  do {                                \
    if (!(c)) {                       \
      fprintf(stderr, __VA_ARGS__);   \
      fputc('\n', stderr);            \
      ++failures;                     \
    }                                 \
  } while (0)

/* Bytes that hold n elements of cache type kv. */
static size_t cache_bytes(int kv, size_t n) { return kv == 0 ? 2 * n : (kv == 3 ? n / 2 : n); }

/* Value of element idx of a cache of type kv (int4: nibble idx % 2 of byte idx / 2). */
static double elem_value(int kv, const unsigned char *base, size_t idx) {
  if (kv == 0) return oracle_code_value(0, ((const uint16_t *)base)[idx]);
  if (kv == 3) return oracle_code_value(3, (base[idx / 2] >> (4 * (idx % 2))) & 15);
  return oracle_code_value(kv, base[idx]);
}

/* One problem: fills the inputs, runs the full and the row evaluations. */
static void run_case(int b, int h, int g, int d, int m_c, int m_d, int n, int kv, int zero_q) {
  const size_t nq = (size_t)b * h * n * d, nc = (size_t)g * m_c * d,
               nd = (size_t)b * g * m_d * d;
  const size_t bc = cache_bytes(kv, nc), bd = cache_bytes(kv, nd);
  uint16_t *q = malloc(nq * 2);
  unsigned char *Kc = malloc(bc + 1), *Vc = malloc(bc + 1);
  unsigned char *Kd = malloc(bd + 1), *Vd = malloc(bd + 1);
  int32_t *lens = malloc(sizeof(int32_t) * b);
  float *ks = malloc(sizeof(float) * g), *vs = malloc(sizeof(float) * g);
  double *out = malloc(sizeof(double) * nq);
  for (size_t i = 0; i < nq; ++i) q[i] = zero_q ? 0 : bf16_of(rnd());
  for (size_t i = 0; i < (kv == 0 ? nc : bc); ++i) {
    if (kv == 0) {
      ((uint16_t *)Kc)[i] = bf16_of(rnd());
      ((uint16_t *)Vc)[i] = bf16_of(rnd());
    } else {
      Kc[i] = (unsigned char)(next() % (kv == 3 ? 256 : 120));
      Vc[i] = (unsigned char)(next() % (kv == 3 ? 256 : 120));
    }
  }
  for (size_t i = 0; i < (kv == 0 ? nd : bd); ++i) {
    if (kv == 0) {
      ((uint16_t *)Kd)[i] = bf16_of(rnd());
      ((uint16_t *)Vd)[i] = bf16_of(rnd());
    } else {
      Kd[i] = (unsigned char)(next() % (kv == 3 ? 256 : 120));
      Vd[i] = (unsigned char)(next() % (kv == 3 ? 256 : 120));
    }
  }
  for (int i = 0; i < b; ++i) lens[i] = m_d ? (int)(next() % (m_d + 1)) : 0;
  if (b > 1) lens[1] = 0;
  for (int k = 0; k < g; ++k) {
    ks[k] = 0.5f + 0.25f * k;
    vs[k] = 2.0f - 0.25f * k;
  }
  const float *kp = kv ? ks : NULL, *vp = kv ? vs : NULL;
  int rc = oracle_attention_kv_fp64(b, h, g, d, m_c, m_d, n, 0.125, kv, q, Kc, Vc, Kd, Vd, lens,
                                    kp, vp, out, 2);
  CHECK(rc == 0, "full evaluation failed: %d", rc);
  const int p = h / g;
  if (zero_q && rc == 0) {
    /* every row: the mean of the value rows its token sees */
    for (int i = 0; i < b; ++i)
      for (int j = 0; j < h; ++j)
        for (int r = 0; r < n; ++r) {
          const int gam = j / p;
          int vis = lens[i] - n + r + 1;
          vis = vis > 0 ? vis : 0;
          for (int u = 0; u < d; ++u) {
            double s = 0.0;
            for (int t = 0; t < m_c; ++t)
              s += (vp ? vp[gam] : 1.0) * elem_value(kv, Vc, ((size_t)gam * m_c + t) * d + u);
            for (int t = 0; t < vis; ++t) {
              const size_t idx = (((size_t)i * g + gam) * m_d + t) * d + u;
              s += (vp ? vp[gam] : 1.0) * elem_value(kv, Vd, idx);
            }
            const double mean = s / (m_c + vis);
            const double got = out[(((size_t)i * h + j) * n + r) * d + u];
            CHECK(fabs(got - mean) <= 1e-12 * (1.0 + fabs(mean)), "mean pin: %g vs %g", got, mean);
          }
        }
  }
  /* rows: every (i, j, r) in reverse order; equal to the full output */
  const int nrows = b * h * n;
  int32_t *ri = malloc(sizeof(int32_t) * nrows), *rj = malloc(sizeof(int32_t) * nrows),
          *rt = malloc(sizeof(int32_t) * nrows);
  double *rows = malloc(sizeof(double) * (size_t)nrows * d);
  for (int k = 0; k < nrows; ++k) {
    const int idx = nrows - 1 - k;
    ri[k] = idx / (h * n);
    rj[k] = (idx / n) % h;
    rt[k] = idx % n;
  }
  rc = oracle_attention_kv_rows_fp64(b, h, g, d, m_c, m_d, n, 0.125, kv, q, Kc, Vc, Kd, Vd, lens,
                                     kp, vp, nrows, ri, rj, rt, rows, 3);
  CHECK(rc == 0, "row evaluation failed: %d", rc);
  for (int k = 0; rc == 0 && k < nrows; ++k) {
    const size_t idx = (((size_t)ri[k] * h + rj[k]) * n + rt[k]) * d;
    CHECK(memcmp(rows + (size_t)k * d, out + idx, sizeof(double) * d) == 0,
          "row %d differs from the full output", k);
  }
  /* error paths: a length out of range, a bad row index, h % g */
  const int32_t saved = lens[0];
  lens[0] = m_d + 1;
  CHECK(oracle_attention_kv_fp64(b, h, g, d, m_c, m_d, n, 0.125, kv, q, Kc, Vc, Kd, Vd, lens, kp,
                                 vp, out, 1) == -6, "length past m_d accepted");
  lens[0] = saved;
  ri[0] = b;
  CHECK(oracle_attention_kv_rows_fp64(b, h, g, d, m_c, m_d, n, 0.125, kv, q, Kc, Vc, Kd, Vd, lens,
                                      kp, vp, 1, ri, rj, rt, rows, 1) == -1, "bad row accepted");
  if (g > 1)
    CHECK(oracle_attention_kv_fp64(b, h + 1, g, d, m_c, m_d, n, 0.125, kv, q, Kc, Vc, Kd, Vd, lens,
                                   kp, vp, out, 1) == -1, "h %% g != 0 accepted");
  free(q); free(Kc); free(Vc); free(Kd); free(Vd); free(lens); free(ks); free(vs); free(out);
  free(ri); free(rj); free(rt); free(rows);
}

int main(void) {
  /* b, h, g, d, m_c, m_d, n, kv, zero_q */
  run_case(3, 4, 2, 8, 5, 4, 1, 0, 0);
  run_case(3, 4, 2, 8, 5, 4, 1, 0, 1);
  run_case(4, 8, 1, 16, 1, 6, 3, 0, 0);   /* single context key, several tokens, short lengths */
  run_case(2, 6, 3, 8, 7, 0, 1, 0, 1);    /* no decode cache */
  run_case(3, 4, 4, 8, 9, 5, 2, 1, 0);    /* fp8 codes with scales */
  run_case(3, 4, 2, 8, 9, 5, 2, 2, 1);    /* int8 codes with scales */
  run_case(3, 4, 2, 8, 9, 5, 2, 3, 0);    /* int4 codes with scales */
  run_case(2, 6, 3, 6, 7, 3, 1, 3, 1);    /* int4, mean pin */
  for (int c = 0; c < 256; ++c) {
    const double v = oracle_code_value(1, c);
    CHECK(isnan(v) == ((c & 0x7f) == 0x7f), "fp8 code %d", c);
  }
  if (failures) {
    fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  printf("oracle driver: all checks passed\n");
  return 0;
}
