// Internal definitions shared by the library's translation units: layout
// constants, the device layout arithmetic (layout versions 2 and 3) and
// small device helpers.  Not part of the public ABI.
#ifndef QTEA_INTERNAL_H_
#define QTEA_INTERNAL_H_

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "qtea.h"

namespace qtea_detail {

constexpr int kGroupPacks = 16;
constexpr int kGroupCols = 80;   // 16 packs x 5 columns
constexpr int kTileRows = 64;    // one row per lane of a wavefront
constexpr int kCodes = 243;      // 3^5
constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr uint32_t kZeroCode4 = 0x79797979u;  // four copies of code 121 (all-zero trits)
constexpr int kLayout = 2;      // residual values fp16
constexpr int kLayoutE4M3 = 3;  // residual values FP8 E4M3 (one byte each)
// The paper's format: per row and 128-column group a scale alpha and a bias
// beta, the group's 128 trits in 26 one-byte packs, E4M3 residual values.
// On the device a group takes 32 pack slots (two 16-pack groups), slots
// 26..31 holding the all-zero code.
constexpr int kLayoutG128 = 4;
constexpr int kScaleCols = 128;  // columns per quantization group
constexpr int kScalePacks = 26;  // packs per quantization group (25 of five columns, one of three)
constexpr int64_t kAlign = 256;
constexpr int64_t kHeaderBytes = 256;
constexpr int kFlagOffset = 128;

constexpr uint32_t kFlagBadTrit = 1u;
constexpr uint32_t kFlagBadResid = 2u;

// FP8 E4M3 (sign, 4 exponent bits with bias 7, 3 mantissa bits, no
// infinities; exponent and mantissa all ones is NaN) to the fp16 bits of the
// same value.  Every finite E4M3 value is an fp16 value: normal values keep
// their mantissa and move the exponent bias from 7 to 15; a subnormal m 2^-9
// (m = 1..7) is normal in fp16.
__host__ __device__ __forceinline__ uint16_t e4m3_to_half_bits(uint32_t b) {
  const uint32_t s = (b & 0x80u) << 8, e = (b >> 3) & 15u, m = b & 7u;
  if (e) return uint16_t(s | ((e + 8u) << 10) | (m << 7));
  if (!m) return uint16_t(s);
  const uint32_t p = m >= 4u ? 2u : (m >= 2u ? 1u : 0u);  // floor(log2 m)
  return uint16_t(s | ((p + 6u) << 10) | ((m << (10u - p)) & 0x3ffu));
}
__host__ __device__ __forceinline__ bool e4m3_is_nan(uint32_t b) { return (b & 0x7fu) == 0x7fu; }
// The same value as fp32: a normal code moves its exponent bias from 7 to
// 127; a subnormal one is m 2^-9 (exact).
__device__ __forceinline__ float e4m3_to_float(uint32_t b) {
  const uint32_t sgn = (b & 0x80u) << 24, e = (b >> 3) & 15u, m = b & 7u;
  const float nrm = __uint_as_float(sgn | ((e + 120u) << 23) | (m << 20));
  const float sub = __uint_as_float(sgn | __float_as_uint(float(m) * 0x1p-9f));
  return e ? nrm : sub;
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) float lds_float;

inline int64_t align_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

// Residual values are stored tile-major: [n_pad/64 tiles][n_salient][16], the
// sixteen four-row groups of a 64-row tile contiguous for each salient
// column, so the residual of one tile over a run of salient columns is one
// contiguous run of 32 bytes per column.  Index of group g, column s:
__host__ __device__ __forceinline__ int64_t rval_index(int64_t g, int64_t s, int64_t nS) {
  return ((g >> 4) * nS + s) * 16 + (g & 15);
}
inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

__device__ __forceinline__ float h2f(uint16_t h) {
  _Float16 v;
  __builtin_memcpy(&v, &h, 2);
  return (float)v;
}

// ---------------------------------------------------------------------------
// Layout arithmetic shared by the host entry points.
// ---------------------------------------------------------------------------
struct Layout {
  int64_t value_bytes;  // bytes per residual value: 2 (fp16, layout 2) or 1 (E4M3, layouts 3 and 4)
  int64_t n_packs, n_groups, n_pad, n_tiles;
  int64_t off_trits, off_alpha, off_v, off_salient, off_spos, off_rval, off_ridx;
  int64_t off_vs;  // u32 per device column: v | (1 + rank in its slice's salient run) << 16
  int64_t total;
};

// Layout 4 differs in three regions: trits hold two 16-pack groups per
// 128-column group; "alpha" holds u32 (alpha | beta << 16) per row and group
// as [n_pad/64][n_groups/2][64]; v is in device column order (80 per
// 16-pack group, zero in the padding slots).  n_packs is the paper's count
// (26 per group).
inline bool make_layout(int64_t N, int64_t K, int64_t nS, Layout* L, int layout = kLayout) {
  if (N < 4 || N % 4 != 0 || K < 1 || nS < 0 || nS > K) return false;
  if (layout != kLayout && layout != kLayoutE4M3 && layout != kLayoutG128) return false;
  L->value_bytes = layout == kLayout ? 2 : 1;
  const bool g128 = layout == kLayoutG128;
  if (N > (int64_t(1) << 31) - 64 || K > (int64_t(1) << 31) - 160) return false;
  L->n_packs = g128 ? kScalePacks * cdiv(K, kScaleCols) : cdiv(K, 5);
  L->n_groups = g128 ? 2 * cdiv(K, kScaleCols) : cdiv(L->n_packs, kGroupPacks);
  L->n_pad = align_up(N, kTileRows);
  L->n_tiles = L->n_pad / kTileRows;
  int64_t o = kHeaderBytes;
  L->off_trits = o;
  o = align_up(o + L->n_pad * L->n_groups * kGroupPacks, kAlign);
  L->off_alpha = o;
  o = align_up(o + (g128 ? 2 * L->n_pad * L->n_groups : 2 * L->n_pad), kAlign);
  L->off_v = o;
  o = align_up(o + 2 * L->n_groups * kGroupCols, kAlign);
  L->off_salient = o;
  o = align_up(o + 4 * nS, kAlign);
  L->off_spos = o;
  o = align_up(o + 4 * (L->n_groups + 1), kAlign);
  L->off_rval = o;
  o = align_up(o + L->value_bytes * nS * (L->n_pad / 4), kAlign);
  L->off_ridx = o;
  o = align_up(o + 4 * nS * (L->n_pad / 64), kAlign);
  // The v bits again, with each salient column's rank among the salient
  // columns of its 320-column slice (0: not salient): the matrix-core kernel
  // gathers the activations of salient columns as it stages a slice.
  L->off_vs = o;
  o = align_up(o + 4 * L->n_groups * kGroupCols, kAlign);
  L->total = o;
  return true;
}

inline bool desc_ok(const qtea_desc* d) {
  if (!d || d->magic != QTEA_DESC_MAGIC) return false;
  Layout L;
  if (!make_layout(d->N, d->K, d->n_salient, &L, int(d->layout))) return false;
  return L.total == d->bytes_total && L.off_trits == d->off_trits && L.off_alpha == d->off_alpha &&
         L.off_v == d->off_v && L.off_salient == d->off_salient && L.off_spos == d->off_spos &&
         L.off_rval == d->off_rval && L.off_ridx == d->off_ridx && L.n_pad == d->n_pad &&
         L.n_groups == d->n_groups && L.n_packs == d->n_packs;
}

__device__ __forceinline__ void store_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_coherent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace qtea_detail

#endif  // QTEA_INTERNAL_H_
