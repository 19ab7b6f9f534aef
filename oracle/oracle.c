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
 * Quantized caches (the FAQ on attention quantization: 8-bit KV halves the
 * KV bytes, 4-bit KV quarters them, and the method is unchanged). Reading: a
 * cache may hold 8-bit or 4-bit codes instead of bf16, with one fp32 scale
 * per KV group for keys and one for values, shared by the context and
 * decode caches of that group (the decode cache continues the context's
 * sequence, so one static scale serves both). The key (value) of a row is
 * k_scale[gam] (v_scale[gam]) times the code's value:
 *   int8      two's complement integer in [-128, 127]
 *   int4      two's complement integer in [-8, 7], two codes per byte:
 *             element u of a row is in byte u/2 of the row, even u in the
 *             low nibble (bits 0-3), odd u in the high nibble (bits 4-7);
 *             a row of d elements is d/2 bytes (d even)
 *   fp8 e4m3  OCP 8-bit float E4M3 (sign, 4-bit exponent with bias 7, 3-bit
 *             mantissa; exponent 0 is subnormal, m/8 * 2^-6; all-ones
 *             exponent and mantissa is NaN; no infinities; largest 448)
 * The scaled values are formed exactly in fp64 (a float times an 8-bit value
 * fits in 53 bits) and the attention above runs on them unchanged. bf16
 * caches take scales too (NULL means 1).
 *
 * Parity pins for this file live in tests/test_oracle_pins.py (closed forms,
 * invariants, brute force, and agreement with an independent numpy
 * evaluation of the bifurcated Eq. 3-4) and tests/test_oracle_kvquant.py
 * (code tables against torch's float8 conversion, numpy's int8 view and an
 * unpackbits table of the int4 codes; scale identities; int4 against int8 of
 * sixteen times the codes).
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

#define KV_BF16 0
#define KV_FP8_E4M3 1
#define KV_INT8 2
#define KV_INT4 3

static double widen_bf16(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* OCP E4M3: value = (-1)^s * (1 + m/8) * 2^(e-7) for e > 0, (-1)^s * m/8 *
 * 2^-6 for e = 0; e = 15 with m = 7 is NaN. */
static double fp8_e4m3_value(uint8_t c) {
  const int sgn = c >> 7, e = (c >> 3) & 15, m = c & 7;
  if (e == 15 && m == 7) return NAN;
  const double mag = e == 0 ? ldexp((double)m, -9) : ldexp(8.0 + m, e - 10);
  return sgn ? -mag : mag;
}

/* Two's complement value of a 4-bit code (its bit 3 weighs -8). */
static double int4_value(unsigned nibble) {
  const int v = (int)(nibble & 7u) - ((nibble & 8u) ? 8 : 0);
  return (double)v;
}

/* Unscaled value of element idx of a cache stored as kv_type (idx counts
 * elements; for int4 it selects a nibble of byte idx/2). */
static double code_value(int kv_type, const void *base, size_t idx) {
  switch (kv_type) {
    case KV_FP8_E4M3: return fp8_e4m3_value(((const uint8_t *)base)[idx]);
    case KV_INT8: return (double)(int8_t)((const uint8_t *)base)[idx];
    case KV_INT4: {
      const uint8_t byte = ((const uint8_t *)base)[idx >> 1];
      return int4_value((idx & 1) ? (unsigned)(byte >> 4) : (unsigned)(byte & 15u));
    }
    default: return widen_bf16(((const uint16_t *)base)[idx]);
  }
}

/* Decoded value of one code (for the pins of the code tables); an int4 code
 * is the low nibble of `code`. */
double oracle_code_value(int kv_type, int code) {
  if (kv_type == KV_BF16) return widen_bf16((uint16_t)code);
  return code_value(kv_type, &(uint8_t){(uint8_t)code}, 0);
}

/* One output row (sample i, head j): the textbook two-pass softmax over the
 * materialised per-sample cache of the head's group. Every sum runs
 * sequentially in index order: each logit over u, Z over t, and each output
 * element over t. The loops are arranged so that several independent sums
 * advance together (four keys' logits at a time; all d output elements per
 * key), which leaves each sum's order, and so its value, unchanged. */
static void attend_row(int d, int m_i, double scale, const double *qrow,
                       const double *K, const double *V, double *s, double *o) {
  double mu = -INFINITY;
  int t = 0;
  for (; t + 4 <= m_i; t += 4) {
    const double *k0 = K + (size_t)t * d;
    double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
    for (int u = 0; u < d; ++u) {
      a0 += qrow[u] * k0[u];
      a1 += qrow[u] * k0[d + u];
      a2 += qrow[u] * k0[2 * d + u];
      a3 += qrow[u] * k0[3 * d + u];
    }
    s[t] = scale * a0;
    s[t + 1] = scale * a1;
    s[t + 2] = scale * a2;
    s[t + 3] = scale * a3;
  }
  for (; t < m_i; ++t) {
    double acc = 0.0;
    for (int u = 0; u < d; ++u) acc += qrow[u] * K[(size_t)t * d + u];
    s[t] = scale * acc;
  }
  for (t = 0; t < m_i; ++t)
    if (s[t] > mu) mu = s[t];
  double Z = 0.0;
  for (t = 0; t < m_i; ++t) {
    s[t] = exp(s[t] - mu);
    Z += s[t];
  }
  for (int u = 0; u < d; ++u) o[u] = 0.0;
  for (t = 0; t < m_i; ++t) {
    const double w = s[t];
    const double *vr = V + (size_t)t * d;
    for (int u = 0; u < d; ++u) o[u] += w * vr[u];
  }
  for (int u = 0; u < d; ++u) o[u] /= Z;
}

/* Decode rows that query token r (of n) of a sample with len valid rows sees. */
static int visible(int len, int n, int r) {
  const int v = len - n + r + 1;
  return v > 0 ? v : 0;
}

static int check_dims(int b, int h, int g, int d, int m_c, int m_d_max, int n, int kv_type,
                      const int32_t *lens) {
  if (b < 1 || h < 1 || g < 1 || d < 1 || m_c < 0 || m_d_max < 0 || n < 1) return ORACLE_EINVAL;
  if (kv_type != KV_BF16 && kv_type != KV_FP8_E4M3 && kv_type != KV_INT8 && kv_type != KV_INT4)
    return ORACLE_EINVAL;
  if (kv_type == KV_INT4 && d % 2) return ORACLE_EINVAL; /* whole bytes per row */
  if (h % g) return ORACLE_EINVAL;
  for (int i = 0; i < b; ++i)
    if (lens[i] < 0 || lens[i] > m_d_max) return ORACLE_ELENS;
  for (int i = 0; i < b; ++i)
    if (m_c + visible(lens[i], n, 0) < 1) return ORACLE_EINVAL; /* softmax over nothing */
  return ORACLE_OK;
}

/* The first m_c + vis rows of the explicit per-sample cache of (i, gam):
 * context rows, then the sample's decode rows, scaled values in fp64. */
static void gather_rows(int g, int d, int m_c, int m_d_max, int kv_type, const void *Kc,
                        const void *Vc, const void *Kd, const void *Vd, const float *k_scale,
                        const float *v_scale, int i, int gam, int vis, double *K, double *V) {
  const double ks = k_scale ? (double)k_scale[gam] : 1.0;
  const double vs = v_scale ? (double)v_scale[gam] : 1.0;
  for (int t = 0; t < m_c; ++t)
    for (int u = 0; u < d; ++u) {
      size_t src = ((size_t)gam * m_c + t) * d + u;
      K[(size_t)t * d + u] = ks * code_value(kv_type, Kc, src);
      V[(size_t)t * d + u] = vs * code_value(kv_type, Vc, src);
    }
  for (int t = 0; t < vis; ++t)
    for (int u = 0; u < d; ++u) {
      size_t src = (((size_t)i * g + gam) * m_d_max + t) * d + u;
      K[(size_t)(m_c + t) * d + u] = ks * code_value(kv_type, Kd, src);
      V[(size_t)(m_c + t) * d + u] = vs * code_value(kv_type, Vd, src);
    }
}

/* Rows (sample row_i[r], head row_j[r], token row_t[r]) for r < nrows,
 * written to out[r*d .. r*d+d). Rows are independent; threads split them. */
int oracle_attention_kv_rows_fp64(int b, int h, int g, int d, int m_c, int m_d_max, int n,
                                  double scale, int kv_type, const uint16_t *q, const void *Kc,
                                  const void *Vc, const void *Kd, const void *Vd,
                                  const int32_t *lens, const float *k_scale,
                                  const float *v_scale, int nrows, const int32_t *row_i,
                                  const int32_t *row_j, const int32_t *row_t, double *out,
                                  int nthreads) {
  int rc = check_dims(b, h, g, d, m_c, m_d_max, n, kv_type, lens);
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
      gather_rows(g, d, m_c, m_d_max, kv_type, Kc, Vc, Kd, Vd, k_scale, v_scale, i, gam, vis, K,
                  V);
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
int oracle_attention_kv_fp64(int b, int h, int g, int d, int m_c, int m_d_max, int n,
                             double scale, int kv_type, const uint16_t *q, const void *Kc,
                             const void *Vc, const void *Kd, const void *Vd,
                             const int32_t *lens, const float *k_scale, const float *v_scale,
                             double *out, int nthreads) {
  int rc = check_dims(b, h, g, d, m_c, m_d_max, n, kv_type, lens);
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
      gather_rows(g, d, m_c, m_d_max, kv_type, Kc, Vc, Kd, Vd, k_scale, v_scale, i, gam, lens[i],
                  K, V);
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

/* bf16 caches, unit scales. */
int oracle_attention_fp64(int b, int h, int g, int d, int m_c, int m_d_max, int n,
                          double scale, const uint16_t *q, const uint16_t *Kc,
                          const uint16_t *Vc, const uint16_t *Kd, const uint16_t *Vd,
                          const int32_t *lens, double *out, int nthreads) {
  return oracle_attention_kv_fp64(b, h, g, d, m_c, m_d_max, n, scale, KV_BF16, q, Kc, Vc, Kd,
                                  Vd, lens, NULL, NULL, out, nthreads);
}

int oracle_attention_rows_fp64(int b, int h, int g, int d, int m_c, int m_d_max, int n,
                               double scale, const uint16_t *q, const uint16_t *Kc,
                               const uint16_t *Vc, const uint16_t *Kd, const uint16_t *Vd,
                               const int32_t *lens, int nrows, const int32_t *row_i,
                               const int32_t *row_j, const int32_t *row_t, double *out,
                               int nthreads) {
  return oracle_attention_kv_rows_fp64(b, h, g, d, m_c, m_d_max, n, scale, KV_BF16, q, Kc, Vc,
                                       Kd, Vd, lens, NULL, NULL, nrows, row_i, row_j, row_t, out,
                                       nthreads);
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
