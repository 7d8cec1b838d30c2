// Internal definitions shared by the library's translation units: device
// helpers on top of the host layout arithmetic (layout.h).  Not part of the
// public ABI.
#ifndef QTEA_INTERNAL_H_
#define QTEA_INTERNAL_H_

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "layout.h"
#include "qtea.h"

namespace qtea_detail {

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


// Residual values are stored tile-major: [n_pad/64 tiles][n_salient][16], the
// sixteen four-row groups of a 64-row tile contiguous for each salient
// column, so the residual of one tile over a run of salient columns is one
// contiguous run of 32 bytes per column.  Index of group g, column s:
__host__ __device__ __forceinline__ int64_t rval_index(int64_t g, int64_t s, int64_t nS) {
  return ((g >> 4) * nS + s) * 16 + (g & 15);
}

__device__ __forceinline__ float h2f(uint16_t h) {
  _Float16 v;
  __builtin_memcpy(&v, &h, 2);
  return (float)v;
}

__device__ __forceinline__ void store_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_coherent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace qtea_detail

#endif  // QTEA_INTERNAL_H_
