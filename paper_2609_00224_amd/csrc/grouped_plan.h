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
int grouped_mma_rows_per_panel();

}  // namespace qtea_grouped

#endif  // QTEA_GROUPED_PLAN_H_
