/*
 * Plain fp64 CPU oracle for the QTEA compressed ternary GEMV.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the GPU library; both sides take their inputs
 * from the seeded generator (which holds none of the method's arithmetic).
 *
 * What is computed (paper: "Efficient Ternary Computation", Eq. 10 and
 * Eq. 11, with one quantization group spanning all K columns and beta = 0):
 *
 *   y[b][r] = alpha_r * sum_j T[r][j] * v_j * x[b][j]
 *           + sum_{s : S_s in salient columns} R[r][S_s] * x[b][S_s]
 *
 * where R is nonzero only at row 4g + idx[s][g] of each group g of four
 * consecutive output rows (one stored residual per group of four entries of
 * a salient column, same section).  The residual is scaled by neither alpha
 * nor v (Eq. 11 adds R_rj x_j as is).
 *
 * Readings of points the paper leaves open (also listed in the design notes):
 *   - a byte holds 5 consecutive columns' trits as base-3 digits d = t + 1,
 *     column 5p + i being digit i (least significant first);
 *   - K is padded to a multiple of 5 with the zero trit (digit 1);
 *   - byte values 243..255 are invalid (3^5 = 243 < 256);
 *   - fp16 inputs are IEEE binary16, converted exactly to binary64 here.
 *
 * Every function is plain nested loops in the order of the definition; the
 * only parallelism is an OpenMP loop over independent output rows.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum {
  OR_OK = 0,
  OR_ERR_ARG = -1,
  OR_ERR_TRIT = -2,  /* a trit outside {-1, 0, +1} */
  OR_ERR_CODE = -3,  /* a byte >= 243, or a nonzero trit in the K padding */
  OR_ERR_RESID = -4, /* a residual position > 3 or a bad salient list */
  OR_ERR_NOMEM = -5,
};

static const int kPow3[5] = {1, 3, 9, 27, 81};

/* IEEE 754 binary16 -> binary64, from the format's definition. */
double or_half_to_double(uint16_t h) {
  const int sign = h >> 15, e = (h >> 10) & 31, m = h & 1023;
  double mag;
  if (e == 0)
    mag = ldexp((double)m, -24); /* subnormal: m * 2^-24 */
  else if (e == 31)
    mag = m ? NAN : INFINITY;
  else
    mag = ldexp((double)(1024 + m), e - 25); /* (1 + m/1024) * 2^(e-15) */
  return sign ? -mag : mag;
}

int64_t or_num_packs(int64_t K) { return (K + 4) / 5; }

/* Base-3 code of five trits (Eq. 10 discussion: 3^5 < 2^8, five ternary
 * values per byte). Returns the code 0..242, or OR_ERR_TRIT. */
int or_encode5(const int8_t* t) {
  int c = 0;
  for (int i = 0; i < 5; ++i) {
    if (t[i] < -1 || t[i] > 1) return OR_ERR_TRIT;
    c += (t[i] + 1) * kPow3[i];
  }
  return c;
}

/* Inverse of or_encode5: digit i of the code is floor(c / 3^i) mod 3. */
int or_decode_code(int code, int8_t* t) {
  if (code < 0 || code >= 243) return OR_ERR_CODE;
  for (int i = 0; i < 5; ++i) t[i] = (int8_t)((code / kPow3[i]) % 3 - 1);
  return OR_OK;
}

/* Canonical packing: out[r][p] = code of columns 5p..5p+4 of row r, with the
 * zero trit standing in for columns >= K. */
int or_pack(const int8_t* trits, int64_t nrows, int64_t K, uint8_t* out) {
  if (nrows < 0 || K < 1) return OR_ERR_ARG;
  const int64_t Kp = or_num_packs(K);
  for (int64_t r = 0; r < nrows; ++r) {
    for (int64_t p = 0; p < Kp; ++p) {
      int8_t t[5];
      for (int i = 0; i < 5; ++i) {
        const int64_t j = 5 * p + i;
        t[i] = j < K ? trits[r * K + j] : 0;
      }
      const int c = or_encode5(t);
      if (c < 0) return c;
      out[r * Kp + p] = (uint8_t)c;
    }
  }
  return OR_OK;
}

/* Canonical unpacking; rejects invalid bytes and nonzero padding trits. */
int or_unpack(const uint8_t* bytes, int64_t nrows, int64_t K, int8_t* trits) {
  if (nrows < 0 || K < 1) return OR_ERR_ARG;
  const int64_t Kp = or_num_packs(K);
  for (int64_t r = 0; r < nrows; ++r) {
    for (int64_t p = 0; p < Kp; ++p) {
      int8_t t[5];
      const int rc = or_decode_code(bytes[r * Kp + p], t);
      if (rc != OR_OK) return rc;
      for (int i = 0; i < 5; ++i) {
        const int64_t j = 5 * p + i;
        if (j < K)
          trits[r * K + j] = t[i];
        else if (t[i] != 0)
          return OR_ERR_CODE;
      }
    }
  }
  return OR_OK;
}

/* Salient list: strictly increasing column indices in [0, K). */
int or_check_salient(const int32_t* S, int64_t nS, int64_t K) {
  if (nS < 0 || nS > K) return OR_ERR_ARG;
  for (int64_t s = 0; s < nS; ++s) {
    if (S[s] < 0 || S[s] >= K) return OR_ERR_RESID;
    if (s > 0 && S[s] <= S[s - 1]) return OR_ERR_RESID;
  }
  return OR_OK;
}

/* Output row of each stored residual: rows[s][g] = 4g + idx[s][g]. */
int or_resid_rows(const uint8_t* idx, int64_t nS, int64_t N, int32_t* rows) {
  if (nS < 0 || N < 0 || N % 4) return OR_ERR_ARG;
  const int64_t G = N / 4;
  for (int64_t s = 0; s < nS; ++s)
    for (int64_t g = 0; g < G; ++g) {
      const uint8_t q = idx[s * G + g];
      if (q > 3) return OR_ERR_RESID;
      rows[s * G + g] = (int32_t)(4 * g + q);
    }
  return OR_OK;
}

typedef struct {
  int64_t N, K, nS;
  const uint16_t* alpha; /* fp16 [N] */
  const uint16_t* v;     /* fp16 [K] */
  const int32_t* S;      /* [nS] */
  const uint16_t* R;     /* fp16 [nS][N/4] */
  const uint8_t* idx;    /* [nS][N/4] */
} or_layer;

static int check_layer(const or_layer* L) {
  if (L->N < 4 || L->N % 4 || L->K < 1 || L->nS < 0) return OR_ERR_ARG;
  int rc = or_check_salient(L->S, L->nS, L->K);
  if (rc) return rc;
  const int64_t G = L->N / 4;
  for (int64_t i = 0; i < L->nS * G; ++i)
    if (L->idx[i] > 3) return OR_ERR_RESID;
  return OR_OK;
}

/* Dequantized row r in fp64 (Eq. 10 with G = K, beta = 0, plus Eq. 11):
 * W[j] = alpha_r * v_j * T[r][j], then W[S_s] += R[s][r/4] where the stored
 * position of group r/4 is r mod 4.  `codes` is the canonical row. */
static int dense_row(const or_layer* L, int64_t r, const uint8_t* codes, double* W) {
  const int64_t K = L->K, Kp = or_num_packs(K), G = L->N / 4;
  const double a = or_half_to_double(L->alpha[r]);
  for (int64_t p = 0; p < Kp; ++p) {
    int8_t t[5];
    const int rc = or_decode_code(codes[p], t);
    if (rc) return rc;
    for (int i = 0; i < 5; ++i) {
      const int64_t j = 5 * p + i;
      if (j < K)
        W[j] = a * or_half_to_double(L->v[j]) * (double)t[i];
      else if (t[i] != 0)
        return OR_ERR_CODE;
    }
  }
  const int64_t g = r / 4;
  for (int64_t s = 0; s < L->nS; ++s)
    if (L->idx[s * G + g] == (uint8_t)(r % 4)) W[L->S[s]] += or_half_to_double(L->R[s * G + g]);
  return OR_OK;
}

static or_layer make_layer(int64_t N, int64_t K, int64_t nS, const uint16_t* alpha,
                           const uint16_t* v, const int32_t* S, const uint16_t* R,
                           const uint8_t* idx) {
  or_layer L = {N, K, nS, alpha, v, S, R, idx};
  return L;
}

/* Dense fp64 rows W[i][:] of the listed output rows. P_rows[i] is the
 * canonical byte row of output row rows[i]. */
int or_dense_rows(int64_t N, int64_t K, const uint8_t* P_rows, const int64_t* rows,
                  int64_t nrows, const uint16_t* alpha, const uint16_t* v, const int32_t* S,
                  int64_t nS, const uint16_t* R, const uint8_t* idx, double* W) {
  const or_layer L = make_layer(N, K, nS, alpha, v, S, R, idx);
  int rc = check_layer(&L);
  if (rc) return rc;
  const int64_t Kp = or_num_packs(K);
  for (int64_t i = 0; i < nrows; ++i) {
    if (rows[i] < 0 || rows[i] >= N) return OR_ERR_ARG;
    rc = dense_row(&L, rows[i], P_rows + i * Kp, W + i * K);
    if (rc) return rc;
  }
  return OR_OK;
}

/* y[b][i] = sum_j W[rows[i]][j] * x[b][j], summed in fp64 in ascending j. */
int or_gemv_rows(int64_t N, int64_t K, const uint8_t* P_rows, const int64_t* rows,
                 int64_t nrows, const uint16_t* alpha, const uint16_t* v, const int32_t* S,
                 int64_t nS, const uint16_t* R, const uint8_t* idx, const uint16_t* x,
                 int64_t B, double* y, int nthreads) {
  const or_layer L = make_layer(N, K, nS, alpha, v, S, R, idx);
  int rc = check_layer(&L);
  if (rc) return rc;
  if (B < 1) return OR_ERR_ARG;
  for (int64_t i = 0; i < nrows; ++i)
    if (rows[i] < 0 || rows[i] >= N) return OR_ERR_ARG;
  double* xd = (double*)malloc((size_t)(B * K) * sizeof(double));
  if (!xd) return OR_ERR_NOMEM;
  for (int64_t e = 0; e < B * K; ++e) xd[e] = or_half_to_double(x[e]);
  const int64_t Kp = or_num_packs(K);
  int err = OR_OK;
#pragma omp parallel num_threads(nthreads > 0 ? nthreads : 1)
  {
    double* W = (double*)malloc((size_t)K * sizeof(double));
    if (!W) {
#pragma omp atomic write
      err = OR_ERR_NOMEM;
    }
#pragma omp for schedule(dynamic, 16)
    for (int64_t i = 0; i < nrows; ++i) {
      if (!W) continue;
      const int rr = dense_row(&L, rows[i], P_rows + i * Kp, W);
      if (rr) {
#pragma omp atomic write
        err = rr;
        continue;
      }
      for (int64_t b = 0; b < B; ++b) {
        double acc = 0.0;
        for (int64_t j = 0; j < K; ++j) acc += W[j] * xd[b * K + j];
        y[b * nrows + i] = acc;
      }
    }
    free(W);
  }
  free(xd);
  return err;
}

/* The same product through per-pack lookup tables (Eq. 10 discussion):
 * a_j = v_j * x_j (zero in the K padding); for pack p and code c,
 * L_p[c] = sum_i (d_i(c) - 1) * a_{5p+i}; then
 * y[b][i] = alpha_r * sum_p L_p[P[r][p]] + sum_s [stored row] R x[S_s].
 * All in fp64; used to show the table route reaches the plain definition. */
int or_gemv_lut_rows(int64_t N, int64_t K, const uint8_t* P_rows, const int64_t* rows,
                     int64_t nrows, const uint16_t* alpha, const uint16_t* v, const int32_t* S,
                     int64_t nS, const uint16_t* R, const uint8_t* idx, const uint16_t* x,
                     int64_t B, double* y) {
  const or_layer L = make_layer(N, K, nS, alpha, v, S, R, idx);
  int rc = check_layer(&L);
  if (rc) return rc;
  if (B < 1) return OR_ERR_ARG;
  const int64_t Kp = or_num_packs(K), G = N / 4;
  double* a = (double*)calloc((size_t)(B * 5 * Kp), sizeof(double));
  double* T = (double*)malloc((size_t)(B * Kp * 243) * sizeof(double));
  if (!a || !T) {
    free(a);
    free(T);
    return OR_ERR_NOMEM;
  }
  for (int64_t b = 0; b < B; ++b)
    for (int64_t j = 0; j < K; ++j)
      a[b * 5 * Kp + j] = or_half_to_double(v[j]) * or_half_to_double(x[b * K + j]);
  for (int64_t b = 0; b < B; ++b)
    for (int64_t p = 0; p < Kp; ++p)
      for (int c = 0; c < 243; ++c) {
        int8_t t[5];
        or_decode_code(c, t);
        double e = 0.0;
        for (int i = 0; i < 5; ++i) e += (double)t[i] * a[b * 5 * Kp + 5 * p + i];
        T[(b * Kp + p) * 243 + c] = e;
      }
  for (int64_t i = 0; i < nrows; ++i) {
    const int64_t r = rows[i];
    if (r < 0 || r >= N) {
      rc = OR_ERR_ARG;
      break;
    }
    for (int64_t p = 0; p < Kp; ++p)
      if (P_rows[i * Kp + p] >= 243) rc = OR_ERR_CODE;
    if (rc) break;
    const double al = or_half_to_double(alpha[r]);
    for (int64_t b = 0; b < B; ++b) {
      double acc = 0.0;
      for (int64_t p = 0; p < Kp; ++p) acc += T[(b * Kp + p) * 243 + P_rows[i * Kp + p]];
      double res = 0.0;
      for (int64_t s = 0; s < nS; ++s)
        if (idx[s * G + r / 4] == (uint8_t)(r % 4))
          res += or_half_to_double(R[s * G + r / 4]) * or_half_to_double(x[b * K + S[s]]);
      y[b * nrows + i] = al * acc + res;
    }
  }
  free(a);
  free(T);
  return rc;
}

/* Bits per weight of the stored format, counting everything: packed trits
 * (8 bits per 5 columns, K padded to a multiple of 5), one 16-bit residual
 * value and one 2-bit position per four entries of each salient column, a
 * K-bit salient bitmap, 16-bit alpha per row and 16-bit v per column. */
double or_bpw_full(int64_t N, int64_t K, int64_t nS) {
  const double bits = 8.0 * (double)N * (double)or_num_packs(K) +
                      (double)(N / 4) * (double)nS * (16.0 + 2.0) + (double)K +
                      16.0 * (double)N + 16.0 * (double)K;
  return bits / ((double)N * (double)K);
}

/* The paper's own accounting (setup section): 8/5 bits for the ternary
 * codes plus f * b / 4 for b-bit residual values on a fraction f of the
 * columns at one value per four entries. */
double or_bpw_paper(double f, double value_bits) { return 8.0 / 5.0 + f * value_bits / 4.0; }

/* Bytes one GEMV must read for its weights: canonical packed trits, fp16
 * residual values with 2-bit positions, fp16 alpha and v, int32 salient
 * column list. */
int64_t or_algorithmic_bytes(int64_t N, int64_t K, int64_t nS) {
  const int64_t entries = (N / 4) * nS;
  return N * or_num_packs(K) + 2 * entries + (2 * entries + 7) / 8 + 2 * N + 2 * K + 4 * nS;
}

/* The paper's storage of the salient residual (its GEMV section, at its
 * evaluation setting): one FP8 E4M3 value per four entries of a salient
 * column and a bitmap over the input columns marking the salient ones. */

/* FP8 E4M3 -> binary64, from the format's definition: sign bit, 4 exponent
 * bits with bias 7, 3 mantissa bits; exponent 0 is subnormal (m/8 * 2^-6);
 * no infinities; exponent 15 with mantissa 7 is NaN. */
double or_e4m3_to_double(uint8_t c) {
  const int sign = c >> 7, e = (c >> 3) & 15, m = c & 7;
  double mag;
  if (e == 15 && m == 7)
    mag = NAN;
  else if (e == 0)
    mag = ldexp((double)m, -9); /* (m / 8) * 2^(1 - 7) */
  else
    mag = ldexp((double)(8 + m), e - 10); /* (1 + m/8) * 2^(e - 7) */
  return sign ? -mag : mag;
}

/* Salient column list from a bitmap (bit j % 32 of word j / 32 marks column
 * j), ascending.  Returns the count, or OR_ERR_RESID for a bit at or past K
 * or more than cap columns. */
int64_t or_bitmap_to_list(const uint32_t* words, int64_t K, int32_t* S, int64_t cap) {
  int64_t n = 0;
  const int64_t nw = (K + 31) / 32;
  for (int64_t j = 0; j < 32 * nw; ++j) {
    if (!((words[j / 32] >> (j % 32)) & 1u)) continue;
    if (j >= K || n >= cap) return OR_ERR_RESID;
    S[n++] = (int32_t)j;
  }
  return n;
}

/* Weight bytes of one GEMV as or_algorithmic_bytes, with value_bytes per
 * residual value (2 for fp16, 1 for E4M3). */
int64_t or_algorithmic_bytes_vb(int64_t N, int64_t K, int64_t nS, int64_t value_bytes) {
  const int64_t entries = (N / 4) * nS;
  return N * or_num_packs(K) + value_bytes * entries + (2 * entries + 7) / 8 + 2 * N + 2 * K + 4 * nS;
}

/* ------------------------------------------------------------------------
 * The paper's quantization groups (Eq. 10 in full; its setting: group size
 * 128).  Row r and 128-column group g have a scale alpha_{r,g} and a bias
 * beta_{r,g}:
 *
 *   y[b][r] = sum_g ( alpha_{r,g} sum_{j in g} T[r][j] v_j x[b][j]
 *                   + beta_{r,g}  sum_{j in g} x[b][j] )
 *           + the Eq. 11 residual, as above.
 *
 * The 128 trits of a row's group are packed into 26 bytes (the paper's
 * appendix: 1.625 bits per weight): bytes 0..24 hold columns 5p..5p+4 of
 * the group, byte 25 its last three columns and two zero trits; columns
 * past K (in the last group) are zero trits too.
 * ------------------------------------------------------------------------ */
int64_t or_num_groups128(int64_t K) { return (K + 127) / 128; }

/* out[r][26 g + p]: code of pack p of group g of row r. */
int or_pack128(const int8_t* trits, int64_t nrows, int64_t K, uint8_t* out) {
  if (nrows < 0 || K < 1) return OR_ERR_ARG;
  const int64_t ng = or_num_groups128(K);
  for (int64_t r = 0; r < nrows; ++r)
    for (int64_t g = 0; g < ng; ++g)
      for (int p = 0; p < 26; ++p) {
        int8_t t[5];
        for (int i = 0; i < 5; ++i) {
          const int64_t c = 5 * p + i;  /* column within the group */
          const int64_t j = 128 * g + c;
          t[i] = (c < 128 && j < K) ? trits[r * K + j] : 0;
        }
        const int code = or_encode5(t);
        if (code < 0) return code;
        out[(r * ng + g) * 26 + p] = (uint8_t)code;
      }
  return OR_OK;
}

/* Inverse of or_pack128; rejects invalid bytes and nonzero padding trits. */
int or_unpack128(const uint8_t* bytes, int64_t nrows, int64_t K, int8_t* trits) {
  if (nrows < 0 || K < 1) return OR_ERR_ARG;
  const int64_t ng = or_num_groups128(K);
  for (int64_t r = 0; r < nrows; ++r)
    for (int64_t g = 0; g < ng; ++g)
      for (int p = 0; p < 26; ++p) {
        int8_t t[5];
        const int rc = or_decode_code(bytes[(r * ng + g) * 26 + p], t);
        if (rc) return rc;
        for (int i = 0; i < 5; ++i) {
          const int64_t c = 5 * p + i;
          const int64_t j = 128 * g + c;
          if (c < 128 && j < K)
            trits[r * K + j] = t[i];
          else if (t[i] != 0)
            return OR_ERR_CODE;
        }
      }
  return OR_OK;
}

/* y[b][i] for output rows rows[i], from the packed groups P_rows[i] (row
 * rows[i], 26 bytes per group), the group scales and biases alpha, beta
 * ([N][ng] fp16), v [K], the residual as above, x [B][K]; fp64, each group's
 * two sums in ascending column order, groups in ascending order. */
int or_gemv128_rows(int64_t N, int64_t K, const uint8_t* P_rows, const int64_t* rows, int64_t nrows,
                    const uint16_t* alpha, const uint16_t* beta, const uint16_t* v, const int32_t* S,
                    int64_t nS, const uint16_t* R, const uint8_t* idx, const uint16_t* x, int64_t B,
                    double* y, int nthreads) {
  const or_layer L = make_layer(N, K, nS, alpha, v, S, R, idx);
  int rc = check_layer(&L);
  if (rc) return rc;
  if (B < 1) return OR_ERR_ARG;
  for (int64_t i = 0; i < nrows; ++i)
    if (rows[i] < 0 || rows[i] >= N) return OR_ERR_ARG;
  const int64_t ng = or_num_groups128(K), G = N / 4;
  double* xd = (double*)malloc((size_t)(B * K) * sizeof(double));
  if (!xd) return OR_ERR_NOMEM;
  for (int64_t e = 0; e < B * K; ++e) xd[e] = or_half_to_double(x[e]);
  int err = OR_OK;
#pragma omp parallel num_threads(nthreads > 0 ? nthreads : 1)
  {
    int8_t* T = (int8_t*)malloc((size_t)K);
    if (!T) {
#pragma omp atomic write
      err = OR_ERR_NOMEM;
    }
#pragma omp for schedule(dynamic, 16)
    for (int64_t i = 0; i < nrows; ++i) {
      if (!T) continue;
      const int64_t r = rows[i];
      const int rr = or_unpack128(P_rows + i * ng * 26, 1, K, T);
      if (rr) {
#pragma omp atomic write
        err = rr;
        continue;
      }
      for (int64_t b = 0; b < B; ++b) {
        const double* xb = xd + b * K;
        double total = 0.0;
        for (int64_t g = 0; g < ng; ++g) {
          double tv = 0.0, xs = 0.0;
          for (int64_t j = 128 * g; j < 128 * g + 128 && j < K; ++j) {
            tv += (double)T[j] * or_half_to_double(v[j]) * xb[j];
            xs += xb[j];
          }
          total += or_half_to_double(alpha[r * ng + g]) * tv + or_half_to_double(beta[r * ng + g]) * xs;
        }
        double res = 0.0;
        for (int64_t s = 0; s < nS; ++s)
          if (idx[s * G + r / 4] == (uint8_t)(r % 4)) res += or_half_to_double(R[s * G + r / 4]) * xb[S[s]];
        y[b * nrows + i] = total + res;
      }
    }
    free(T);
  }
  free(xd);
  return err;
}

/* Weight bytes of one GEMV in the grouped format: 26 bytes per row and
 * group, fp16 alpha and beta per row and group, the residual with value_bytes
 * per value and 2-bit positions, fp16 v, int32 salient list. */
int64_t or_algorithmic_bytes128(int64_t N, int64_t K, int64_t nS, int64_t value_bytes) {
  const int64_t ng = or_num_groups128(K), entries = (N / 4) * nS;
  return N * ng * 26 + 4 * N * ng + value_bytes * entries + (2 * entries + 7) / 8 + 2 * K + 4 * nS;
}
