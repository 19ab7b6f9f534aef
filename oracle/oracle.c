/*
 * CPU fp64 oracle for bifurcated decode attention -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load this library. The GPU library never links, includes or calls it, and it
 * shares no code with the GPU library.
 *
 * What it computes (paper Section 3.3, Eq. 1-2; exactness claim of Section 4.2
 * and its proof in Appendix E.1): the bifurcated method returns exactly the
 * standard multi-group attention over the full per-sample key/value cache
 * K_i = K_c (+) K_d[i]. The oracle therefore evaluates that plain definition,
 * with no bifurcation and no online softmax:
 *
 *   for each sample i and KV group gam:
 *     materialise the explicit per-sample copies (widened bf16 -> fp64)
 *         K_{i,gam} = [Kc[gam, 0:m_c, :] ; Kd[i, gam, 0:len_i, :]]   (m_c+len_i rows)
 *         V_{i,gam} likewise
 *     for each head j of the group (j = gam*p + r, r < p; group-major,
 *     matching the bgpnk index order of Eq. 1):
 *       and each of its n query tokens r (0 <= r < n):
 *         the token sees the context rows and the first
 *             vis_r = max(0, len_i - n + r + 1)
 *         decode rows (m_r = m_c + vis_r keys)
 *         s_t   = scale * sum_u q[i,j,r,u] * K_{i,gam}[t,u]      (t < m_r)
 *         mu    = max_t s_t
 *         w_t   = exp(s_t - mu)
 *         Z     = sum_t w_t
 *         o[u]  = (sum_t w_t * V_{i,gam}[t,u]) / Z
 *
 * q and the output are [b][h][n][d] (the paper's b g p n k order). With
 * n = 1 (one new token per sample, Section 3.1) the token sees all len_i
 * decode rows. With n > 1 (draft tokens verified in one step, the appendix
 * on speculative decoding, where n_g replaces n) the n new tokens are the
 * last n of the sample's len_i decode rows and each sees the rows up to and
 * including itself. All sums run sequentially in index order in fp64. Rows
 * a token does not see are never read. Outputs are fp64.
 *
 * Parity pins for this file live in tests/test_oracle_pins.py (closed forms,
 * invariants, brute force, and agreement with an independent numpy
 * evaluation of the bifurcated Eq. 3-4).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_EINVAL -1
#define ORACLE_ENOMEM -4
#define ORACLE_ELENS -6

static double widen_bf16(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* One output row (sample i, head j): the textbook two-pass softmax over the
 * materialised per-sample cache of the head's group. */
static void attend_row(int d, int m_i, double scale, const double *qrow,
                       const double *K, const double *V, double *s, double *o) {
  double mu = -INFINITY;
  for (int t = 0; t < m_i; ++t) {
    double acc = 0.0;
    for (int u = 0; u < d; ++u) acc += qrow[u] * K[(size_t)t * d + u];
    s[t] = scale * acc;
    if (s[t] > mu) mu = s[t];
  }
  double Z = 0.0;
  for (int t = 0; t < m_i; ++t) {
    s[t] = exp(s[t] - mu);
    Z += s[t];
  }
  for (int u = 0; u < d; ++u) {
    double acc = 0.0;
    for (int t = 0; t < m_i; ++t) acc += s[t] * V[(size_t)t * d + u];
    o[u] = acc / Z;
  }
}

/* Decode rows that query token r (of n) of a sample with len valid rows sees. */
static int visible(int len, int n, int r) {
  const int v = len - n + r + 1;
  return v > 0 ? v : 0;
}

static int check_dims(int b, int h, int g, int d, int m_c, int m_d_max, int n,
                      const int32_t *lens) {
  if (b < 1 || h < 1 || g < 1 || d < 1 || m_c < 0 || m_d_max < 0 || n < 1) return ORACLE_EINVAL;
  if (h % g) return ORACLE_EINVAL;
  for (int i = 0; i < b; ++i)
    if (lens[i] < 0 || lens[i] > m_d_max) return ORACLE_ELENS;
  for (int i = 0; i < b; ++i)
    if (m_c + visible(lens[i], n, 0) < 1) return ORACLE_EINVAL; /* softmax over nothing */
  return ORACLE_OK;
}

/* Rows (sample row_i[r], head row_j[r], token row_t[r]) for r < nrows,
 * written to out[r*d .. r*d+d). Rows are independent; threads split them. */
int oracle_attention_rows_fp64(int b, int h, int g, int d, int m_c, int m_d_max, int n,
                               double scale, const uint16_t *q,
                               const uint16_t *Kc, const uint16_t *Vc,
                               const uint16_t *Kd, const uint16_t *Vd,
                               const int32_t *lens, int nrows,
                               const int32_t *row_i, const int32_t *row_j,
                               const int32_t *row_t, double *out, int nthreads) {
  int rc = check_dims(b, h, g, d, m_c, m_d_max, n, lens);
  if (rc) return rc;
  for (int r = 0; r < nrows; ++r)
    if (row_i[r] < 0 || row_i[r] >= b || row_j[r] < 0 || row_j[r] >= h || row_t[r] < 0 ||
        row_t[r] >= n)
      return ORACLE_EINVAL;
  const int p = h / g;
  int failed = 0;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1) reduction(| : failed)
#endif
  for (int r = 0; r < nrows; ++r) {
    const int i = row_i[r], j = row_j[r], tok = row_t[r], gam = j / p;
    const int vis = visible(lens[i], n, tok);
    const int m_i = m_c + vis;
    double *K = malloc(sizeof(double) * (size_t)m_i * d);
    double *V = malloc(sizeof(double) * (size_t)m_i * d);
    double *s = malloc(sizeof(double) * (size_t)m_i);
    double *qrow = malloc(sizeof(double) * (size_t)d);
    if (!K || !V || !s || !qrow) {
      failed = 1;
    } else {
      for (int t = 0; t < m_c; ++t)
        for (int u = 0; u < d; ++u) {
          size_t src = ((size_t)gam * m_c + t) * d + u;
          K[(size_t)t * d + u] = widen_bf16(Kc[src]);
          V[(size_t)t * d + u] = widen_bf16(Vc[src]);
        }
      for (int t = 0; t < vis; ++t)
        for (int u = 0; u < d; ++u) {
          size_t src = (((size_t)i * g + gam) * m_d_max + t) * d + u;
          K[(size_t)(m_c + t) * d + u] = widen_bf16(Kd[src]);
          V[(size_t)(m_c + t) * d + u] = widen_bf16(Vd[src]);
        }
      for (int u = 0; u < d; ++u)
        qrow[u] = widen_bf16(q[(((size_t)i * h + j) * n + tok) * d + u]);
      attend_row(d, m_i, scale, qrow, K, V, s, out + (size_t)r * d);
    }
    free(K);
    free(V);
    free(s);
    free(qrow);
  }
  return failed ? ORACLE_ENOMEM : ORACLE_OK;
}

/* Full output [b, h, n, d]. The per-sample cache of each (i, gam) is
 * materialised once (all len_i rows) and reused by the group's p heads and
 * n tokens, each token taking its visible prefix of the decode rows. */
int oracle_attention_fp64(int b, int h, int g, int d, int m_c, int m_d_max, int n,
                          double scale, const uint16_t *q, const uint16_t *Kc,
                          const uint16_t *Vc, const uint16_t *Kd,
                          const uint16_t *Vd, const int32_t *lens, double *out,
                          int nthreads) {
  int rc = check_dims(b, h, g, d, m_c, m_d_max, n, lens);
  if (rc) return rc;
  const int p = h / g;
  int failed = 0;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1) reduction(| : failed)
#endif
  for (long unit = 0; unit < (long)b * g; ++unit) {
    const int i = (int)(unit / g), gam = (int)(unit % g);
    const int m_i = m_c + lens[i];
    double *K = malloc(sizeof(double) * (size_t)(m_i > 0 ? m_i : 1) * d);
    double *V = malloc(sizeof(double) * (size_t)(m_i > 0 ? m_i : 1) * d);
    double *s = malloc(sizeof(double) * (size_t)(m_i > 0 ? m_i : 1));
    double *qrow = malloc(sizeof(double) * (size_t)d);
    if (!K || !V || !s || !qrow) {
      failed = 1;
    } else {
      for (int t = 0; t < m_c; ++t)
        for (int u = 0; u < d; ++u) {
          size_t src = ((size_t)gam * m_c + t) * d + u;
          K[(size_t)t * d + u] = widen_bf16(Kc[src]);
          V[(size_t)t * d + u] = widen_bf16(Vc[src]);
        }
      for (int t = 0; t < lens[i]; ++t)
        for (int u = 0; u < d; ++u) {
          size_t src = (((size_t)i * g + gam) * m_d_max + t) * d + u;
          K[(size_t)(m_c + t) * d + u] = widen_bf16(Kd[src]);
          V[(size_t)(m_c + t) * d + u] = widen_bf16(Vd[src]);
        }
      for (int r = 0; r < p; ++r) {
        const int j = gam * p + r;
        for (int tok = 0; tok < n; ++tok) {
          const size_t row = ((size_t)i * h + j) * n + tok;
          for (int u = 0; u < d; ++u) qrow[u] = widen_bf16(q[row * d + u]);
          attend_row(d, m_c + visible(lens[i], n, tok), scale, qrow, K, V, s, out + row * d);
        }
      }
    }
    free(K);
    free(V);
    free(s);
    free(qrow);
  }
  return failed ? ORACLE_ENOMEM : ORACLE_OK;
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
