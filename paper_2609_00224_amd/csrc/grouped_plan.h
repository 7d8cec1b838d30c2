// Plan of a grouped GEMV (many independent problems in one persistent
// launch): the records the host planner writes and the kernels read, shared
// by the batch-1 table kernel (grouped.hip) and the low-batch matrix-core
// kernel (grouped_mma.hip).  Internal to the library.
#ifndef QTEA_GROUPED_PLAN_H_
#define QTEA_GROUPED_PLAN_H_

#include "qtea_internal.h"

namespace qtea_grouped {

using namespace qtea_detail;

constexpr int kSliceGroups = 4;                           // groups per K slice (one per quarter-wave)
constexpr int kSlicePacks = kSliceGroups * kGroupPacks;   // 64
constexpr int kSliceCols = kSliceGroups * kGroupCols;     // 320
constexpr uint32_t kGPlanMagic = 0x51475250u;            // "QGRP"
constexpr int64_t kPlanProblemsOff = 256;

struct GProblem {
  const uint8_t* trits;
  const uint16_t* alpha;
  const uint16_t* v;
  const int32_t* S;
  const int32_t* spos;
  const uint16_t* rval;  // fp16, or E4M3 bytes when the plan's f8 is set
  const uint32_t* ridx;
  const uint16_t* x;
  float* y;
  int64_t N, K, n_pad;
  int32_t n_groups, nS, n_slices, n_panels;
  int64_t unit_base;
  const uint32_t* vs;  // v | (1 + rank in the slice's salient run) << 16, per device column
};
static_assert(sizeof(GProblem) == 128, "plan record size");

// One problem run on its own (qtea_gemv, qtea_gemm_lowbatch): its record
// is a kernel argument, and workgroup g of G takes the contiguous run of
// units [g U / G, (g + 1) U / G) of the U = n_panels * n_slices units.  A
// panel whose units fall in more than one run is finished by the last of
// its workgroups to arrive (a counter per panel in the workspace), which
// sums the parts in run order.
struct GOne {
  GProblem pr;
  int32_t n_units;
  int32_t batch;
  int32_t reserved[2];
};

// Workgroup whose run holds unit x, for U units over G runs: the largest g
// with floor(g U / G) <= x.
__host__ __device__ __forceinline__ int one_owner(int64_t x, int64_t U, int64_t G) {
  return int(((x + 1) * G - 1) / U);
}
__host__ __device__ __forceinline__ int64_t one_first(int64_t g, int64_t U, int64_t G) { return (g * U) / G; }

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

struct GPlanHeader {
  uint32_t magic, version;
  int32_t n_problems, n_wg, rows_per_panel, max_parts, batch, n_chunks;
  int64_t n_units, off_chunks, n_grabs, off_splits, n_splits;
  int32_t f8, reserved;  // residual values are E4M3 bytes (layout 3) in every problem
};

// A chunk: units [ub, ue), the first of them at (problem m, panel, slice).
struct GChunk {
  int32_t ub, ue, m, panel, slice, reserved[3];
};
static_assert(sizeof(GChunk) == 32, "one scalar load per chunk record");

// A panel whose slices fall in more than one chunk: its parts are in the
// partial slots of chunks ga..gb (slot 2k, except 2ga + 1 when the part in
// chunk ga starts after that chunk's first unit).
struct GSplit {
  int32_t m, panel, ga, gb, ga_odd, reserved[3];
};

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
int grouped_mma_rows_per_panel();

}  // namespace qtea_grouped

#endif  // QTEA_GROUPED_PLAN_H_
