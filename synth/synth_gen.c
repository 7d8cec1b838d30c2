/*
 * Seeded synthetic input generator for the ternary-LUT GEMV workloads.
 *
 * This file holds random-number generation and distribution sampling only:
 * no part of the compressed format (no base-3 packing, no scaling, no LUT)
 * lives here, so both the CPU oracle and the GPU path can consume its output
 * without sharing any of the method's arithmetic.
 *
 * Generator: SplitMix64 (Steele, Lea and Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014), used in counter mode:
 *   draw(key, i) = mix64(key + (i + 1) * GAMMA)
 * so element i of any stream can be produced independently of the others
 * (a row subset of a 57344 x 8192 trit matrix costs only that subset).
 *
 * Stream keys are derived from (seed, layer, matrix, field) by chaining the
 * same mixer; see synth_key().
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define SM64_GAMMA 0x9E3779B97F4A7C15ULL

static inline uint64_t sm64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

/* Element i of the counter-mode stream keyed by `key`. With key = s this is
 * the (i+1)-th output of a sequential SplitMix64 seeded with s. */
static inline uint64_t sm64_at(uint64_t key, uint64_t i) {
  return sm64_mix(key + (i + 1) * SM64_GAMMA);
}

uint64_t synth_sm64_at(uint64_t key, uint64_t i) { return sm64_at(key, i); }

uint64_t synth_key(uint64_t seed, uint64_t layer, uint64_t mat, uint64_t field) {
  uint64_t k = sm64_mix(seed + SM64_GAMMA);
  k = sm64_mix(k + (layer + 1) * SM64_GAMMA);
  k = sm64_mix(k + (mat + 1) * SM64_GAMMA);
  k = sm64_mix(k + (field + 1) * SM64_GAMMA);
  return k;
}

/* Ternary draws: element (r, j) uses counter r*K + j; the top 32 bits u of
 * the draw give -1 if u < thr_neg, 0 if u < thr_zero, else +1. */
static inline int8_t trit_of(uint64_t z, uint32_t thr_neg, uint32_t thr_zero) {
  uint32_t u = (uint32_t)(z >> 32);
  return (int8_t)(u < thr_neg ? -1 : (u < thr_zero ? 0 : 1));
}

void synth_trits(uint64_t key, int64_t N, int64_t K, uint32_t thr_neg,
                 uint32_t thr_zero, int8_t* out, int nthreads) {
#pragma omp parallel for schedule(static) num_threads(nthreads)
  for (int64_t r = 0; r < N; ++r) {
    const uint64_t base = (uint64_t)r * (uint64_t)K;
    int8_t* o = out + r * K;
    for (int64_t j = 0; j < K; ++j)
      o[j] = trit_of(sm64_at(key, base + (uint64_t)j), thr_neg, thr_zero);
  }
}

void synth_trits_rows(uint64_t key, int64_t K, const int64_t* rows,
                      int64_t nrows, uint32_t thr_neg, uint32_t thr_zero,
                      int8_t* out, int nthreads) {
#pragma omp parallel for schedule(static) num_threads(nthreads)
  for (int64_t i = 0; i < nrows; ++i) {
    const uint64_t base = (uint64_t)rows[i] * (uint64_t)K;
    int8_t* o = out + i * K;
    for (int64_t j = 0; j < K; ++j)
      o[j] = trit_of(sm64_at(key, base + (uint64_t)j), thr_neg, thr_zero);
  }
}

/* Uniform doubles in [lo, hi): lo + (hi - lo) * (top 53 bits) * 2^-53. */
void synth_uniform(uint64_t key, int64_t n, double lo, double hi, double* out) {
  for (int64_t i = 0; i < n; ++i) {
    const double u = (double)(sm64_at(key, (uint64_t)i) >> 11) * 0x1p-53;
    out[i] = lo + (hi - lo) * u;
  }
}

/* Normal doubles by the Box-Muller transform (cosine branch only): element i
 * uses counters 2i (u1 in (0,1]) and 2i+1 (u2 in [0,1)). */
void synth_normal(uint64_t key, int64_t n, double mu, double sigma, double* out) {
  const double two_pi = 6.283185307179586476925286766559;
  for (int64_t i = 0; i < n; ++i) {
    const double u1 =
        (double)((sm64_at(key, 2 * (uint64_t)i) >> 11) + 1) * 0x1p-53;
    const double u2 =
        (double)(sm64_at(key, 2 * (uint64_t)i + 1) >> 11) * 0x1p-53;
    out[i] = mu + sigma * sqrt(-2.0 * log(u1)) * cos(two_pi * u2);
  }
}

/* 2-bit uniform draws (top two bits of each draw), values 0..3. */
void synth_uint2(uint64_t key, int64_t n, uint8_t* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = (uint8_t)(sm64_at(key, (uint64_t)i) >> 62);
}

static int cmp_i32(const void* a, const void* b) {
  const int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
  return (x > y) - (x < y);
}

/* n distinct values from [0, K) chosen uniformly without replacement by a
 * partial Fisher-Yates shuffle, returned sorted ascending. Draw i picks the
 * swap partner i + floor(z * (K - i) / 2^64) (Lemire's multiply-high; its
 * bias is below (K - i) / 2^64). Returns 0, or -1 on bad arguments. */
int synth_choose_sorted(uint64_t key, int64_t K, int64_t n, int32_t* out) {
  if (K < 0 || n < 0 || n > K || K > 0x7fffffff) return -1;
  if (n == 0) return 0;
  int32_t* perm = (int32_t*)malloc((size_t)K * sizeof(int32_t));
  if (!perm) return -1;
  for (int64_t i = 0; i < K; ++i) perm[i] = (int32_t)i;
  for (int64_t i = 0; i < n; ++i) {
    const uint64_t z = sm64_at(key, (uint64_t)i);
    const uint64_t span = (uint64_t)(K - i);
    const int64_t j = i + (int64_t)(((unsigned __int128)z * span) >> 64);
    const int32_t t = perm[i];
    perm[i] = perm[j];
    perm[j] = t;
  }
  memcpy(out, perm, (size_t)n * sizeof(int32_t));
  free(perm);
  qsort(out, (size_t)n, sizeof(int32_t), cmp_i32);
  return 0;
}
