// Plan of a grouped GEMV (many independent problems in one persistent
// launch): the records the host planner writes and the kernels read, shared
// by the batch-1 table kernel (grouped.hip) and the low-batch matrix-core
// kernel (grouped_mma.hip).  Internal to the library.
#ifndef QTEA_GROUPED_PLAN_H_
#define QTEA_GROUPED_PLAN_H_

#include "plan_host.h"
#include "qtea_internal.h"

namespace qtea_grouped {

using namespace qtea_detail;

// Coherent 16-byte load from the workspace (device scope: sc1), for parts
// written by other workgroups with device-scope stores.
constexpr int kAuxSC1 = 16;

// The last workgroup of a split panel sums its parts in run order:
// out[e] = sum over k = ga..gb of part[slot(k) * S + e] (slot(k) = 2k, or
// 2ga + 1 for the first part when odd0), for the S floats of a slot (S a
// multiple of 4), and hands each float4 of sums to store(e, value).  The T
// threads split the vectors and, when there are fewer vectors than
// threads, the parts too (Q groups of threads take every Q-th part), with
// up to 8 loads in flight per thread; the groups' sums are added in group
// order through `tmp` (LDS, T float4).  Fixed order: deterministic.
template <int T, class Store>
__device__ __forceinline__ void sum_parts(const float* part, int64_t S, int ga, int gb, int odd0, float4* tmp,
                                          Store store) {
  const int tid = threadIdx.x;
  const int V4 = int(S / 4);
  const int Q = V4 < T ? T / V4 : 1;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(part), 0, 0x7fffffff, 0x00020000);
  auto ld = [&](int k, int v) -> float4 {
    const int64_t slot = 2 * int64_t(k) + (k == ga ? odd0 : 0);
    const int64_t off = (slot * S + 4 * int64_t(v)) * 4;
    return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, int(off), 0, kAuxSC1));
  };
  if (Q > 1) {
    const int v = tid % V4, qg = tid / V4;
    float4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    if (qg < Q) {
      for (int k0 = ga + qg; k0 <= gb; k0 += 8 * Q) {
        float4 t8[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) t8[j] = ld(min(k0 + j * Q, gb), v);
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (k0 + j * Q <= gb) acc += t8[j];
      }
      tmp[qg * V4 + v] = acc;
    }
    __syncthreads();
    if (tid < V4) {
      float4 tot = tmp[tid];
      for (int j = 1; j < Q; ++j) tot += tmp[j * V4 + tid];
      store(4 * tid, tot);
    }
    __syncthreads();  // tmp is free again
  } else {
    for (int v0 = tid; v0 < V4; v0 += 4 * T) {
      float4 acc[4] = {};
      for (int k0 = ga; k0 <= gb; k0 += 4) {
        float4 t16[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) t16[i][j] = ld(min(k0 + j, gb), min(v0 + i * T, V4 - 1));
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (k0 + j <= gb) acc[i] += t16[i][j];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (v0 + i * T < V4) store(4 * (v0 + i * T), acc[i]);
    }
  }
}

typedef __attribute__((address_space(1))) const uint8_t gu8;
typedef __attribute__((address_space(1))) const uint16_t gu16;
typedef __attribute__((address_space(1))) const uint32_t gu32;
typedef __attribute__((address_space(1))) const int32_t gi32;
typedef __attribute__((address_space(1))) const u32x4 gu32x4;
typedef __attribute__((address_space(1))) float gf32;

// Pointers read from the plan are generic; loads through them would be flat
// loads (which also hold the LDS wait counter).  They all point to global
// memory, so they are cast to the global address space.
__device__ __forceinline__ gu8* gptr(const uint8_t* p) { return (gu8*)p; }
__device__ __forceinline__ gu16* gptr(const uint16_t* p) { return (gu16*)p; }
__device__ __forceinline__ gu32* gptr(const uint32_t* p) { return (gu32*)p; }
__device__ __forceinline__ gi32* gptr(const int32_t* p) { return (gi32*)p; }
// Read-only and read with a uniform index: the constant address space lets
// the compiler use scalar loads, which do not wait behind the vector loads.
typedef __attribute__((address_space(4))) const int32_t ci32;
__device__ __forceinline__ ci32* cptr(const int32_t* p) { return (ci32*)p; }

struct Cursor {
  int m, panel, slice;
};

__device__ __forceinline__ Cursor advance(Cursor c, const GProblem* P) {
  if (++c.slice == P[c.m].n_slices) {
    c.slice = 0;
    if (++c.panel == P[c.m].n_panels) {
      c.panel = 0;
      ++c.m;
    }
  }
  return c;
}

// Buffer resources (gfx9 family): word 3 of the descriptor for raw byte
// buffers, and the non-temporal bit of a buffer load's cache policy.
constexpr int kBufferWord3 = 0x00020000;
constexpr int kAuxNT = 2;

// Device-side launches of the low-batch kernels (grouped_mma.hip): the
// persistent matrix-core kernel for 2 <= batch <= 16 over `grid`
// workgroups, and its static shared-memory size.
hipError_t launch_grouped_mma(const uint8_t* plan, int grid, int batch, bool f8, float* part, hipStream_t st);
// The same kernel on one problem (one.batch rows), `grid` workgroups, split
// panels finished by their last workgroup (counters: one word per panel).
hipError_t launch_one_mma(const GOne& one, int grid, bool f8, float* part, uint32_t* counters, hipStream_t st);
// Rows per panel of the matrix-core kernel at `batch` (2..16): grouped
// launches, and one matrix on its own.
int grouped_mma_rows_per_panel(int batch);
int one_mma_rows_per_panel(int batch);

}  // namespace qtea_grouped

#endif  // QTEA_GROUPED_PLAN_H_
