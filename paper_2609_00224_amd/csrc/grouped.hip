// Grouped GEMV: y_m = W_m x_m for a list of independent problems in one
// persistent launch (Eq. 10 with one group and zero bias, plus the Eq. 11
// residual, for every problem of the list).
//
// Work unit = (problem, panel of RP rows, K slice of 4 sixteen-pack groups =
// 64 packs = 320 columns).  Units are ordered (problem, panel, slice) with
// the slice fastest.  Two 512-thread workgroups share each CU (about 79 KB of
// LDS each): while one builds its tables the other streams and looks up, so
// the phases of one workgroup's units hide behind the other's.  Per unit a
// workgroup:
//
//   - stages a_j = v_j x_j and x_j of the slice in LDS;
//   - builds the full 243-entry table of each of the slice's 64 packs
//     (62,208 bytes of LDS, one fp32 entry per code and pack);
//   - adds one table entry per packed byte of the panel's rows, the entry
//     address formed from the byte by a single v_perm_b32;
//   - adds the slice's salient residual;
//   - at the panel's last slice, writes y = alpha * acc + residual.
//
// While a unit is processed, the next unit's packed bytes, activations,
// residual and row scales are already in flight: each 16-byte register of
// packed bytes is refilled with the next unit's bytes as soon as its lookups
// have been issued, so the weight stream does not stop at unit, panel,
// problem or chunk boundaries.
//
// Scheduling.  The two workgroups of a CU do not progress at the same rate
// (the older one's waves win instruction issue), so equal static shares
// leave half of the CUs' workgroups idle long before the launch ends.  The
// unit list is therefore cut into chunks whose sizes shrink from large to a
// single unit (guided self-scheduling, planned on the host), and after its
// first two chunks a workgroup takes the next chunk from a queue counter in
// the workspace, one chunk ahead of need.  A panel whose slices fall in
// more than one chunk is split: each part stores its partial rows in the
// workspace and grouped_reduce_kernel, launched right after, sums the parts
// in chunk order (fixed order: deterministic whichever workgroup ran which
// chunk).  No workgroup ever waits for another one.
#include <stdlib.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "grouped_plan.h"

namespace {

using namespace qtea_detail;
using namespace qtea_grouped;

constexpr int kGT = 512;                                  // threads per workgroup
constexpr int kGW = kGT / 64;                             // waves per workgroup
constexpr int kWgPerCu = 2;                               // workgroups sharing a CU
// Table rows: one per code (code row = 64 packs x 4 bytes, 62,208 bytes).
// The debug build (QTEA_DEBUG) also gives the unused byte values 243..255
// rows, filled with NaN: a packed byte that is no base-3 code then turns
// its output row into NaN instead of reading other LDS data.
#ifdef QTEA_DEBUG
constexpr int kTabRows = 256;
#else
constexpr int kTabRows = kCodes;
#endif
constexpr int kTabBytes = kTabRows * 256;
// salient columns of a slice staged per wave (more: direct loads): fp16
// values fill the wave's 1 KiB value area at 16 columns, E4M3 values at 32
constexpr int kResCols = 16;
constexpr int kResCols8 = 32;
static_assert(kSlicePacks * 4 == 256, "one table row of 256 bytes per code");

static_assert(kSliceCols % 64 == 0, "staging by whole waves");
static_assert(kSlicePacks == 64 && kSlicePacks * 8 == kGT,
              "one 27-code build task per thread, codes 0..215, one wave per pair of leading trits");
static_assert(kSliceCols <= kGT, "one staged column per thread");


template <int RB>
struct GLds {
  static constexpr int RP = kGW * 16 * RB;   // rows per panel
  static constexpr int TPW = RP / 64 / kGW;  // 64-row tiles per wave in the residual phase
  static constexpr int GPW = 16 * TPW;       // four-row groups per wave
  static constexpr int QR = 64 / GPW;        // residual lanes per group
  static constexpr int ST = kTabBytes;                    // two buffers: a_j fp32 [320], x_j fp32 [320]
  static constexpr int STB = 8 * kSliceCols;              // bytes of one buffer
  static constexpr int RR = ST + 2 * STB;                 // residual row sums, fp32 [RP]
  static constexpr int RV = RR + 4 * RP;                  // per wave: values [TPW][16 fp16 or 32 E4M3 columns][16]
  static constexpr int RI = RV + kGW * 1024;              // per wave: u32 positions [2][16], fp32 x [32]
  static constexpr int FLAG = RI + kGW * 256;             // one int
  static constexpr int XS = FLAG + 16;                    // layout 4: [2 buffers][5 waves][2] fp32 group sums of x
  static constexpr int BYTES = XS + 128;
};
static_assert(GLds<4>::TPW == 1 && GLds<8>::TPW == 2, "one or two tiles per wave");
static_assert(2 * kResCols * 32 == 1024 && 2 * kResCols8 * 16 == 1024,
              "one 16-byte load per lane stages two tiles' values");
#ifndef QTEA_DEBUG
static_assert(kWgPerCu * GLds<8>::BYTES <= 160 * 1024, "two workgroups per CU");
#endif



// The chunk queue's words in the first bytes of the workspace: word 0 the
// take counter, word 1 error flags (sticky until the workspace is
// zero-filled again), words 2-3 a 64-bit exit word: the count of finished
// workgroups (top 16 bits) and the sum of the tags (chunk_tag) of the
// chunks they ran (low 48 bits).  The workgroup whose exit completes a
// multiple of the grid checks that the launch ran every chunk once (the
// plan's exit_sum) and took exactly the plan's count, and leaves the take
// counter and the exit word at zero for the next launch.  A take past the
// plan's count yields no chunk, so every index stays in range, and sets
// kQueueStale.  A launch that starts from words a completed launch does not
// leave runs every chunk once or raises a flag, unless the left-over words
// cancel the tags of the chunks it skipped: the tags are hashed, so that
// takes some 2^-32 luck rather than a small left-over count.
constexpr uint32_t kQueueStale = 1u;  // a take found the counter past the plan's count
constexpr uint32_t kQueueCount = 2u;  // the launch's chunks or takes did not add up to the plan's
constexpr uint64_t kExitSumMask = (uint64_t(1) << 48) - 1;

__device__ __forceinline__ void queue_exit(uint32_t* counters, uint32_t n_grabs, uint64_t exit_sum,
                                           uint64_t my_sum) {
  if (threadIdx.x != 0) return;
  // Relaxed: every queue word is read and written only by device-scope
  // atomics, which the device performs at one coherence point, and each
  // workgroup's takes have returned before it issues its exit, so the exit
  // that completes the count comes after every take of the launch.  (An
  // acquire-release here would write back and invalidate the L2 of the
  // workgroup's XCD at every exit, under the other workgroups' loads.)
  uint64_t* ew = reinterpret_cast<uint64_t*>(counters + 2);
  const uint64_t old = __hip_atomic_fetch_add(ew, (uint64_t(1) << 48) + my_sum, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT);
  if ((uint32_t(old >> 48) + 1u) % gridDim.x != 0u) return;
  const uint64_t ran = (old + my_sum) & kExitSumMask;
  const uint32_t taken = __hip_atomic_load(counters, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (ran != exit_sum || taken != n_grabs)
    __hip_atomic_fetch_or(counters + 1, kQueueCount, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(counters, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(ew, uint64_t(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

// Selector of v_perm_b32 that forms (byte k of src1) << 8 | (byte k of src0).
__device__ __forceinline__ constexpr uint32_t perm_sel(int k) {
  return 0x0C0C0000u | (uint32_t(k) << 8) | uint32_t(4 + k);
}

// F8: residual values are E4M3 bytes (layouts 3, 4), else fp16 (layout 2).
// G128: the paper's 128-column groups (layout 4): a slice is two groups, a
// group two 16-pack slots of 13 packs (65 columns each, device columns
// 160 g + 80 h + c, c < 65); a lane's 13 bytes of a slot row are 13 bytes
// apart from the next row's, loaded as the 16 bytes from the dword below
// them and shifted into place (one v_alignbyte per dword), and looked up 13
// at a time; each slot row's sum is scaled by its row's alpha[r][g] as it is
// added, and the quarter holding the group's first slot adds beta[r][g]
// times the group's sum of x.
//
// ONE: a single problem launched on its own (GOne): no plan and no queue;
// workgroup g takes the contiguous run of units [g U / G, (g + 1) U / G), and
// a panel split between runs is summed by the last of its workgroups to
// arrive (counters[panel] in the workspace, partial rows in `part`).
template <int RB, bool F8, bool G128 = false, bool ONE = false>
__global__ __launch_bounds__(kGT) void grouped_gemv_kernel(const uint8_t* __restrict__ plan,
                                                           float* __restrict__ part,
                                                           uint32_t* __restrict__ counters, const GOne one) {
  using L = GLds<RB>;
  constexpr int RP = L::RP, TPW = L::TPW, GPW = L::GPW, QR = L::QR;
  constexpr int TPP = RP / 64;  // tiles per panel
  extern __shared__ float smem[];
  char* lds = reinterpret_cast<char*>(smem);
  float* rres = reinterpret_cast<float*>(lds + L::RR);
#ifdef QTEA_DEBUG
  // rows of the byte values 243..255: NaN, never overwritten (ordered before
  // the first lookups by the first table build's barrier)
  for (int i = threadIdx.x; i < (256 - kCodes) * 64; i += kGT)
    reinterpret_cast<uint32_t*>(lds + kCodes * 256)[i] = 0x7fc00000u;
#endif
  int* flag = reinterpret_cast<int*>(lds + L::FLAG);

  const GPlanHeader* H = reinterpret_cast<const GPlanHeader*>(plan);
  const GProblem* P = reinterpret_cast<const GProblem*>(plan + kPlanProblemsOff);
  const GChunk* CR = reinterpret_cast<const GChunk*>(plan + (ONE ? 0 : H->off_chunks));
  auto PR = [&](int m) -> const GProblem& {
    if constexpr (ONE) return one.pr;
    else return P[m];
  };
  // the unit after c within its problem list (ONE: within the problem)
  auto adv = [&](Cursor c) -> Cursor {
    if constexpr (ONE) {
      if (++c.slice == one.pr.n_slices) {
        c.slice = 0;
        ++c.panel;
      }
      return c;
    } else {
      return advance(c, P);
    }
  };
  const int g = blockIdx.x;
  const int G = ONE ? int(gridDim.x) : H->n_wg, NC = ONE ? int(gridDim.x) : H->n_chunks;
  // Chunks g and g + G are this workgroup's first two; every later chunk is
  // taken from the queue counters[0] (2G + the count before the increment)
  // while the current chunk runs, for the chunk after the next one, as late
  // as the prefetch allows: each unit loads the next unit's operands, so the
  // chunk after chunk c must be known at the top of c's last unit, and a take
  // is issued at the top of a unit and published at its last barrier.  The
  // take is made at the current chunk's second-to-last unit (at its only unit
  // for a one-unit chunk): taking at a chunk's first unit instead fixes the
  // large early chunks to workgroups at the start, and the launch ends less
  // evenly.  The next chunk's record is loaded at the top of every unit and
  // first used after the table build's barrier, so a chunk switch does not
  // wait for it.  (ONE: one run per workgroup, nothing taken.)
  const uint32_t n_grabs = ONE ? 0u : uint32_t(H->n_grabs);
  const uint64_t exit_sum = ONE ? 0u : H->exit_sum;
  if (!ONE && g >= NC) {
    queue_exit(counters, n_grabs, exit_sum, 0u);
    return;
  }
  int c = g, cn = ONE ? NC : g + G;
  uint64_t my_sum = chunk_tag(uint32_t(g));  // tags of the chunks this workgroup has started
  int* cnext_lds = flag + 1;  // chunk taken from the queue, published at the unit's last barrier

  const int tid = threadIdx.x, lane = tid & 63, q = lane >> 4, l16 = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wt = w >> 2, wr = w & 3;  // tile of the wave's first row block, block in its tile
  // residual lane mapping: wave w takes the TPW tiles w*TPW.. of the panel,
  // one four-row group per lane (gw), the QR lanes of a group (rq) taking its
  // salient columns round-robin
  const int gw = lane & (GPW - 1), rq = lane / GPW;
  const int gi = w * GPW + gw;  // group in the panel
  const int rtile = gw >> 4, g16 = gw & 15;

  // table slot bytes of this lane: byte k of slotreg[d] = 4 * (16 q + ((4 d +
  // k + l16) mod 16)), layout 4: mod 13 (the packs of a slot row are stored
  // rotated by the row the same way)
  constexpr int NLK = G128 ? kG128SlotPacks : kGroupPacks;  // lookups per 16-byte load
  uint32_t slotreg[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    uint32_t r = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) r |= uint32_t(4 * (16 * q + (4 * d + k + l16) % NLK)) << (8 * k);
    slotreg[d] = r;
  }
  // layout 4: this lane's slot rows start (row mod 4) bytes into their 16-byte loads
  const uint32_t g128_sh = uint32_t((wr * 16 + l16) & 3);

  int u, ue;
  Cursor cur;
  if constexpr (ONE) {
    u = int(one_first(g, one.n_units, G));
    ue = int(one_first(g + 1, one.n_units, G));
    cur = Cursor{0, u / one.pr.n_slices, u % one.pr.n_slices};
  } else {
    const GChunk rec_c = CR[c];
    u = rec_c.ub;
    ue = rec_c.ue;
    cur = Cursor{rec_c.m, rec_c.panel, rec_c.slice};
  }

  // Loads.  Every load is unconditional, from an index clamped into its
  // array (groups past the matrix read a real group whose table entries are
  // zero since a_j = 0 past the last column; rows past n_pad feed only rows
  // that are never stored; values past a range are ignored after the load),
  // so that every path through the unit loop issues the same loads and the
  // compiler's wait counts stay exact: a wait for one value then never also
  // waits for the next unit's weights, which are the youngest loads.

  // activations: this thread stages slice column tid (kept as loaded, checked when staged)
  // real column of device column tid of slice s (layout 4: 160 device
  // columns per 128-column group, 80 per slot, the last 15 of a slot unused)
  const int g128_h = (tid % 160) / kGroupCols, g128_c = (tid % 160) % kGroupCols;
  const bool g128_in = g128_c < kG128SlotCols && kG128SlotCols * g128_h + g128_c < kScaleCols;
  auto real_col = [&](int s) -> uint32_t {
    return G128 ? uint32_t(s * 2 * kScaleCols + kScaleCols * (tid / 160) + kG128SlotCols * g128_h + g128_c)
                : uint32_t(s * kSliceCols + tid);
  };
  auto load_xv = [&](const Cursor c, uint16_t& xr, uint16_t& vr) {
    const GProblem& pr = PR(c.m);
    const uint32_t kx = uint32_t(pr.K), kv = uint32_t(pr.n_groups * kGroupCols);
    const uint32_t col = real_col(c.slice), dcol = uint32_t(c.slice * kSliceCols + tid);
    xr = gptr(pr.x)[col < kx ? col : kx - 1];
    vr = gptr(pr.v)[dcol < kv ? dcol : kv - 1];  // v is in device column order
  };
  // row scales of the row blocks this lane finalizes: t = q + 4 i
  constexpr int RF = RB / 4;
  static_assert(RB % 4 == 0, "row blocks in multiples of the quarters");
  auto load_alpha = [&](const Cursor c, uint16_t (&al)[RF]) {
    const GProblem& pr = PR(c.m);
    const uint32_t np = uint32_t(pr.n_pad);
#pragma unroll
    for (int i = 0; i < RF; ++i) {
      const uint32_t rowq = uint32_t(c.panel * RP + (w + kGW * (q + 4 * i)) * 16 + l16);
      al[i] = gptr(pr.alpha)[rowq < np ? rowq : np - 1];
    }
  };
  // salient residual of unit c: this wave's tiles over the slice's first RC
  // salient columns, fetched as two loads per lane (three for E4M3) and
  // staged in the wave's LDS area in the residual phase.  rvq: 16 bytes of a
  // tile's value run (lanes 0..31 the first tile, 32..63 the second; fp16:
  // 32 bytes per column, 16 columns; E4M3: 16 bytes per column, 32 columns);
  // ris: lanes 0..31 the position words of the tiles (16 columns per tile),
  // lanes 32..63 the salient column indices; ris2 (E4M3): the same for
  // columns 16..31.  Indices are clamped into their regions (without salient
  // columns all read the row scales).
  constexpr int RC = F8 ? kResCols8 : kResCols;
  u32x4 rvq;
  uint32_t ris, ris2 = 0;
  auto load_res = [&](const Cursor c, const int s_lo, const int s_hi) {
    const GProblem& pr = PR(c.m);
    const bool any = pr.nS > 0;
    const uint32_t nS = uint32_t(pr.nS), n_tiles = uint32_t(pr.n_pad >> 6);
    const uint32_t tile0 = uint32_t(c.panel * TPP + w * TPW);
    constexpr uint32_t VB = F8 ? 16u : 32u;  // value bytes per (tile, salient column)
    const uint32_t Tv = min(tile0 + (TPW == 2 ? uint32_t(lane >> 5) : 0u), n_tiles - 1u);
    const uint32_t ncs = uint32_t(min(s_hi - s_lo, RC));
    const uint32_t len = ncs * VB;
    const uint32_t lofs = min(uint32_t(lane & 31) * 16u, len >= 16u ? len - 16u : 0u);
    const uint32_t vofs = any ? min((Tv * nS + uint32_t(s_lo)) * VB + lofs, n_tiles * nS * VB - 16u) : 0u;
    rvq = *reinterpret_cast<const gu32x4*>(
        (any ? reinterpret_cast<gu8*>(gptr(pr.rval)) : reinterpret_cast<gu8*>(gptr(pr.alpha))) + vofs);
    const uint32_t Ti = min(tile0 + (TPW == 2 ? uint32_t((lane >> 4) & 1) : 0u), n_tiles - 1u);
    const uint32_t sc = any ? min(uint32_t(s_lo) + uint32_t(lane & 15), nS - 1u) : 0u;
    gu32* ib = !any ? reinterpret_cast<gu32*>(gptr(pr.alpha))
                    : (lane < 32 ? gptr(pr.ridx) + Ti * nS : reinterpret_cast<gu32*>(gptr(pr.S)));
    ris = ib[sc];
    if constexpr (F8) ris2 = ib[any ? min(uint32_t(s_lo) + 16u + uint32_t(lane & 15), nS - 1u) : 0u];
  };
  // salient range [spos[g0], spos[g1]) of unit c's groups, as a vector load
  // (lane 0 reads the first bound, the other lanes the second): a scalar load
  // here would be waited for at once, and the salient list is read from HBM
  auto load_spos = [&](const Cursor c) -> int {
    const GProblem& pr = PR(c.m);
    const int g0 = c.slice * kSliceGroups;
    const int g1 = g0 + kSliceGroups < pr.n_groups ? g0 + kSliceGroups : pr.n_groups;
    return gptr(pr.spos)[lane == 0 ? g0 : g1];
  };
  // byte offset of the 16-byte unit (row block t, group of the quarter) of unit c
  auto w_off = [&](const Cursor c, int t) -> uint32_t {
    const GProblem& pr = PR(c.m);
    const int ng = pr.n_groups, n_tiles = int(pr.n_pad >> 6);
    const int grp = min(c.slice * kSliceGroups + q, ng - 1);
    const int tl = min(c.panel * TPP + wt + (kGW / 4) * t, n_tiles - 1);
    const uint32_t row = uint32_t(wr * 16 + l16);
    return G128 ? (uint32_t(tl * ng + grp) * kTileRows + row) * kG128SlotPacks - g128_sh
                : (uint32_t(tl * ng + grp) * kTileRows + row) * kGroupPacks;
  };
  // Table entry at LDS byte address `a`.  The kernel has no static LDS, so
  // the dynamic allocation (the tables first) starts at address 0.
  auto tab_at = [](uint32_t a) -> float { return *(const lds_float*)(size_t(a)); };

  u32x4 W[RB];
  uint16_t xr, vr;
  load_xv(cur, xr, vr);
  {
    // (a buffer load: a layout-4 slot row's load is dword- but not 16-byte-aligned)
    const GProblem& pc = PR(cur.m);
    const __amdgpu_buffer_rsrc_t wres0 = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(pc.trits), 0,
        int(uint32_t(pc.n_pad >> 6) * uint32_t(pc.n_groups) * (kTileRows * (G128 ? kG128SlotPacks : kGroupPacks))),
        kBufferWord3);
#pragma unroll
    for (int t = 0; t < RB; ++t) {
      W[t] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(wres0, int(w_off(cur, t)), 0, kAuxNT));
      __builtin_amdgcn_sched_barrier(0);  // the loop's order of the weight loads
    }
  }
  int s_lo_c, s_hi_c;  // salient range of the current unit
  {
    const GProblem& pr = PR(cur.m);
    const int g0 = cur.slice * kSliceGroups;
    const int g1 = g0 + kSliceGroups < pr.n_groups ? g0 + kSliceGroups : pr.n_groups;
    s_lo_c = cptr(pr.spos)[g0];
    s_hi_c = cptr(pr.spos)[g1];
  }
  load_res(cur, s_lo_c, s_hi_c);
  uint16_t al[RF];
  if (!G128) load_alpha(cur, al);
  // layout 4: (alpha | beta << 16) of row block t's row in the quarter's group, one unit ahead
  uint32_t AB[G128 ? RB : 1];
  // through a buffer resource over the problem's scale words: the lane's
  // part of the offset (group and row) in a register, the row block's tile
  // (uniform) in the scalar offset, so a row block's load costs no address
  // arithmetic per lane
  auto ab_at = [&](const Cursor c, int t) -> uint32_t {
    const GProblem& pr = PR(c.m);
    const int n_sg = pr.n_groups >> 1, n_tiles = int(pr.n_pad >> 6);
    const int sg = min(2 * c.slice + (q >> 1), n_sg - 1);
    const int tl = min(c.panel * TPP + wt + (kGW / 4) * t, n_tiles - 1);
    const __amdgpu_buffer_rsrc_t ares = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(pr.alpha), 0, int(uint32_t(n_tiles) * uint32_t(n_sg) * 256u), kBufferWord3);
    return __builtin_amdgcn_raw_buffer_load_b32(ares, int((uint32_t(sg) * 64u + uint32_t(wr * 16 + l16)) * 4u),
                                                int(uint32_t(tl) * uint32_t(n_sg) * 256u), 0);
  };
  if constexpr (G128) {
#pragma unroll
    for (int t = 0; t < RB; ++t) AB[t] = ab_at(cur, t);
  }

  // stage a slice's activations in buffer b: a_j = v_j x_j (exact in fp32) and x_j
  auto stage = [&](const Cursor c, int b) {
    if (w * 64 < kSliceCols) {  // whole waves (kSliceCols is a multiple of 64)
      const GProblem& pr = PR(c.m);
      const int gcol = int(real_col(c.slice)), dcol = c.slice * kSliceCols + tid;
      const bool xin = gcol < pr.K && (!G128 || g128_in);
      const float xf = xin ? h2f(xr) : 0.0f;
      const float vf = dcol < pr.n_groups * kGroupCols ? h2f(vr) : 0.0f;
      float* st = reinterpret_cast<float*>(lds + L::ST + b * L::STB);
      st[tid] = vf * xf;
      st[kSliceCols + tid] = xf;
      if constexpr (G128) {
        // the slice's two groups' sums of x: per wave (butterfly, fixed
        // order), the five waves' parts summed by their readers
        float s0 = tid < 160 ? xf : 0.0f, s1 = tid < 160 ? 0.0f : xf;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
          s0 += __shfl_xor(s0, off);
          s1 += __shfl_xor(s1, off);
        }
        if (lane == 0) {
          float* xs = reinterpret_cast<float*>(lds + L::XS + 64 * b) + 2 * w;
          xs[0] = s0;
          xs[1] = s1;
        }
      }
    }
  };
  stage(cur, 0);
  __syncthreads();

  float acc[RB], racc[4];
#pragma unroll
  for (int t = 0; t < RB; ++t) acc[t] = 0.0f;
#pragma unroll
  for (int k = 0; k < 4; ++k) racc[k] = 0.0f;
  int pstart_slice = cur.slice;     // first slice of the open panel part
  bool part_at_chunk_start = true;  // the open panel part began at its chunk's first unit
  bool chunk_first = true;
  int ctaken = NC;  // chunk after the next one, taken while the current chunk runs (NC: none)

  for (int it = 0;; ++it) {
    const GProblem& pr = PR(cur.m);
    const bool chunk_last = u + 1 == ue;
    const bool has_next = !chunk_last || cn < NC;
    GChunk rec_cn{};
    if constexpr (!ONE) rec_cn = CR[min(cn, NC - 1)];
    const Cursor nxt = !chunk_last ? adv(cur) : (has_next ? Cursor{rec_cn.m, rec_cn.panel, rec_cn.slice} : cur);
    const bool pstart = (cur.slice == 0) || chunk_first;
    const bool pend = (cur.slice == pr.n_slices - 1) || chunk_last;
    if (pstart) {
      pstart_slice = cur.slice;
      part_at_chunk_start = chunk_first;
    }
    // at the chunk's second-to-last unit (its only unit for a one-unit
    // chunk), take the chunk after the next one from the queue
    const bool take = !ONE && cn < NC && (ue - u == 2 || (chunk_first && ue - u == 1));
    uint32_t taken = 0;
    if (take && tid == 0) taken = __hip_atomic_fetch_add(counters, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int col0 = cur.slice * kSliceCols;
    // device column of real column j of this slice, if it is one
    const int rcol0 = G128 ? cur.slice * 2 * kScaleCols : col0;
    auto xcol = [&](int j) -> int {
      const int jl = j - rcol0;
      return G128 ? (jl >= 0 && jl < 2 * kScaleCols ? int(g128_dcol(jl)) : -1) : jl;
    };
    const int sb = it & 1;  // staging buffer of this unit
    const float* a_lds = reinterpret_cast<const float*>(lds + L::ST + sb * L::STB);
    const float* xr_lds = a_lds + kSliceCols;

    // 1. tables (the slice's activations were staged before the last barrier).
    // The 243 codes of a pack are (d4 d3 d2 d1 d0); pass 0: task (pack,
    // d4 d3) for d4 d3 < 22 writes 27 codes; pass 1: task (pack, d2) writes
    // the nine codes 22 d2 d1 d0, so that no wave does two 27-code tasks.
    {
      const int p = lane;
      const float a0 = a_lds[5 * p], a1 = a_lds[5 * p + 1], a2 = a_lds[5 * p + 2];
      const float a3 = a_lds[5 * p + 3], a4 = a_lds[5 * p + 4];
      // the wave's task: d4 d3 = w in base 3 (wave-uniform), so the two
      // leading trits are uniform signs and their part is one product and
      // one fused multiply-add (both exact but the last rounding, as t4 + t3)
      const int d4 = (w * 11) >> 5;
      const int d3 = w - 3 * d4;
      const float base = __builtin_fmaf(float(d3 - 1), a3, float(d4 - 1) * a4);
      lds_char* dst = (lds_char*)smem + p * 4 + (27 * d3 + 81 * d4) * 256;
#pragma unroll
      for (int e2 = 0; e2 < 3; ++e2) {
        const float u2 = e2 == 0 ? base - a2 : (e2 == 1 ? base : base + a2);
#pragma unroll
        for (int e1 = 0; e1 < 3; ++e1) {
          const float u1 = e1 == 0 ? u2 - a1 : (e1 == 1 ? u2 : u2 + a1);
#pragma unroll
          for (int e0 = 0; e0 < 3; ++e0) {
            const float u0 = e0 == 0 ? u1 - a0 : (e0 == 1 ? u1 : u1 + a0);
            *(lds_float*)(dst + (9 * e2 + 3 * e1 + e0) * 256) = u0;
          }
        }
        __builtin_amdgcn_sched_barrier(0);  // nine entries at a time (register pressure)
      }
      if (w < 3) {  // codes 216..242 (d4 = d3 = 2): whole waves, task (pack, d2 = w)
        const float u2 = a4 + a3 + (w == 0 ? -a2 : (w == 1 ? 0.0f : a2));
        lds_char* dst2 = (lds_char*)smem + p * 4 + (216 + 9 * w) * 256;
#pragma unroll
        for (int e1 = 0; e1 < 3; ++e1) {
          const float u1 = e1 == 0 ? u2 - a1 : (e1 == 1 ? u2 : u2 + a1);
#pragma unroll
          for (int e0 = 0; e0 < 3; ++e0) {
            const float u0 = e0 == 0 ? u1 - a0 : (e0 == 1 ? u1 : u1 + a0);
            *(lds_float*)(dst2 + (3 * e1 + e0) * 256) = u0;
          }
        }
      }
    }
    __syncthreads();

    // 2. the next unit's activations and salient range (nxt == cur after the
    // run's last unit: harmless reloads)
    // (ONE: a workgroup's last unit loads nothing more; its last waits are
    // on the critical path of the launch)
    int spv = 0;
    if (!ONE || has_next) {
      load_xv(nxt, xr, vr);
      spv = load_spos(nxt);
    }

    // 3. lookups; each 16-byte unit, once read, is refilled with the next
    // unit's bytes (after the run's last unit all lanes read one 16-byte unit)
    // Next unit's byte offsets: a uniform per-tile part (scalar offset) plus
    // this lane's part (group and row within the tile, one vector offset for
    // all refills), through a buffer resource over the next matrix's packed
    // bytes (loads past its end would return zeros).  After the run's last
    // unit every lane reads the first 16 bytes of the matrix.
    const GProblem& pn = PR(nxt.m);
    const int n_ng = pn.n_groups, n_nt = int(pn.n_pad >> 6);
    const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(pn.trits), 0, int(uint32_t(n_nt) * uint32_t(n_ng) * (kTileRows * NLK)), kBufferWord3);
    const int n_grp = min(nxt.slice * kSliceGroups + q, n_ng - 1), n_t0 = nxt.panel * TPP + wt;
    const uint32_t smask = has_next ? 0xffffffffu : 0u;
    const uint32_t lane_off = ((uint32_t(n_grp) * kTileRows + uint32_t(wr * 16 + l16)) * NLK - (G128 ? g128_sh : 0u)) & smask;
    // (the sums restart after every panel end: a part starts right after one)
    // layout 4: the sum of x over this quarter's group, for the first
    // quarter of each group (the other adds no bias)
    float xq = 0.0f;
    if constexpr (G128) {
      const float* xs = reinterpret_cast<const float*>(lds + L::XS + 64 * sb) + (q >> 1);
      const float xg = (((xs[0] + xs[2]) + xs[4]) + xs[6]) + xs[8];
      xq = (q & 1) ? 0.0f : xg;
    }
#pragma unroll
    for (int t = 0; t < RB; ++t) {
      u32x4 wv = W[t];
      if constexpr (G128) {  // the slot row's 13 bytes to bytes 0..12
        const u32x4 w0 = W[t];
        wv = u32x4{__builtin_amdgcn_alignbyte(w0[1], w0[0], g128_sh), __builtin_amdgcn_alignbyte(w0[2], w0[1], g128_sh),
                   __builtin_amdgcn_alignbyte(w0[3], w0[2], g128_sh), __builtin_amdgcn_alignbyte(w0[3], w0[3], g128_sh)};
      }
      float e[16];
#pragma unroll
      for (int d = 0; d < 4; ++d) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          e[4 * d + k] = 4 * d + k < NLK ? tab_at(__builtin_amdgcn_perm(slotreg[d], wv[d], perm_sel(k))) : 0.0f;
      }
      // all the table reads in flight before the first add
      __builtin_amdgcn_sched_group_barrier(0x002, NLK, 0);  // VALU: addresses
      __builtin_amdgcn_sched_group_barrier(0x100, NLK, 0);  // DS reads
      __builtin_amdgcn_sched_group_barrier(0x002, NLK, 0);  // VALU: sums
      if constexpr (G128) {
        float su = e[0];
#pragma unroll
        for (int i = 1; i < NLK; ++i) su += e[i];
        const float al4 = h2f(uint16_t(AB[t] & 0xffffu)), be4 = h2f(uint16_t(AB[t] >> 16));
        acc[t] = __builtin_fmaf(be4, xq, __builtin_fmaf(al4, su, acc[t]));
        AB[t] = ab_at(nxt, t);  // the next unit's, after the last use
      } else {
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[t] += e[i];
      }
      // keep the sums here: without a use in this block the compiler sinks
      // a unit's adds below the residual and holds every entry in registers
      asm volatile("" : "+v"(acc[t]));
      __builtin_amdgcn_sched_barrier(0);
      // refill after the last read of the old bytes, into the same registers
      // (a load issued earlier would need other registers and a copy at the
      // loop edge, and the copy would wait for the load)
      const uint32_t tile_off = (uint32_t(min(n_t0 + (kGW / 4) * t, n_nt - 1)) * uint32_t(n_ng) * (kTileRows * NLK)) & smask;
      if (!ONE || has_next)
        W[t] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(wres, int(lane_off), int(tile_off), kAuxNT));
      __builtin_amdgcn_sched_barrier(0);
    }

    // 4. residual of this slice: each lane's four rows accumulate in registers
    // over the panel's slices (fixed order: deterministic).  A product goes
    // to the row its 2-bit position names without a compare per row: x's
    // fp16 bits shifted left by 16 * position put x in that row's 16-bit
    // lane of a 64-bit word and zeros in the other three, and each row adds
    // R times its lane in one mixed-precision multiply-add (fp16 operands,
    // fp32 sum; R x is exact in fp32, so each sum is rounded once, as R x
    // added to it).  E4M3 values enter as fp16 bits of value * 2^-8 (the
    // seven magnitude bits at bits 7..13; exact, subnormal codes included)
    // and the sums are scaled back by 2^8 at the panel end: bit for bit the
    // unscaled sums, since no product or sum comes near fp32's limits.
    const int s_lo = s_lo_c, s_hi = s_hi_c;
    const int ncol = s_hi - s_lo;
    const int grow = cur.panel * (RP / 4) + gi;  // global four-row group
    const bool grow_ok = grow * 4 < pr.n_pad;
    const uint32_t gsh = 2u * uint32_t(g16);
#pragma unroll
    for (int k = 0; k < 4; ++k) racc[k] = pstart ? 0.0f : racc[k];
    // R (fp16 bits, or an E4M3 byte) times x (fp16 bits) into row `pos` of the group
    auto radd = [&](uint32_t rbits, uint32_t pos, uint32_t xbits) {
      const uint32_t rh = F8 ? ((rbits & 0x7fu) << 7) | ((rbits & 0x80u) << 8) : rbits;
      const _Float16 r = __builtin_bit_cast(_Float16, uint16_t(rh));
      const uint64_t x4 = uint64_t(xbits) << (pos << 4);  // xbits: zero above bit 15
      const half2_t xl = __builtin_bit_cast(half2_t, uint32_t(x4)), xh = __builtin_bit_cast(half2_t, uint32_t(x4 >> 32));
      racc[0] = __builtin_fmaf(float(r), float(xl.x), racc[0]);
      racc[1] = __builtin_fmaf(float(r), float(xl.y), racc[1]);
      racc[2] = __builtin_fmaf(float(r), float(xh.x), racc[2]);
      racc[3] = __builtin_fmaf(float(r), float(xh.y), racc[3]);
    };
    {
      // stage in this wave's own LDS area: only this wave reads it back, and a
      // wave's LDS accesses complete in order, so no barrier is needed.  The
      // column indices are replaced by the fp16 bits of the columns' activations.
      char* rv_w = lds + L::RV + w * 1024;
      uint32_t* ri_w = reinterpret_cast<uint32_t*>(lds + L::RI + w * 256);
      *reinterpret_cast<u32x4*>(rv_w + 16 * lane) = rvq;
      auto xbits_at = [&](uint32_t col) -> uint32_t {
        const int xc = xcol(int(col));
        const float xf = xr_lds[xc >= 0 && xc < kSliceCols ? xc : 0];
        return uint32_t(__builtin_bit_cast(uint16_t, (_Float16)xf));  // exact: x is an fp16 value
      };
      ri_w[lane] = lane < 32 ? ris : xbits_at(ris);
      asm volatile("" ::: "memory");
      const int nc = grow_ok ? (ncol < RC ? ncol : RC) : 0;
      // columns [c0, min(c1, c0 + 16)) with their position words and activations
      // at ri_w (value rows of 512 bytes per tile: 32 bytes per fp16 column,
      // 16 per E4M3 one); the lane's columns c0 + rq + QR i
      auto columns = [&](int c0, int c1) {
        const int ce = (c1 < c0 + 16 ? c1 : c0 + 16) - c0;
        for (int cl = rq; cl < ce; cl += QR) {  // column within the batch of 16
          const uint32_t rb = F8 ? uint32_t(reinterpret_cast<const uint8_t*>(rv_w)[512 * rtile + 16 * (c0 + cl) + g16])
                                 : uint32_t(reinterpret_cast<const uint16_t*>(rv_w)[256 * rtile + 16 * cl + g16]);
          radd(rb, (ri_w[16 * rtile + cl] >> gsh) & 3u, ri_w[32 + cl]);
        }
      };
      columns(0, nc);
      if (F8 && ncol > 16) {  // uniform: columns 16..31 through the same words area
        asm volatile("" ::: "memory");  // after the reads above (same wave: in order)
        ri_w[lane] = lane < 32 ? ris2 : xbits_at(ris2);
        asm volatile("" ::: "memory");
        columns(16, nc);
      }
    }
    if (ncol > RC) {  // a slice with many salient columns (uniform branch)
      const int64_t T = int64_t(grow >> 4);
      for (int s = s_lo + RC + rq; s < s_hi; s += QR) {
        if (grow_ok) {
          const int64_t vi = rval_index(grow, s, pr.nS);
          const uint32_t rb = F8 ? uint32_t(reinterpret_cast<gu8*>(gptr(pr.rval))[vi]) : uint32_t(gptr(pr.rval)[vi]);
          const float xf = xr_lds[xcol(gptr(pr.S)[s])];
          const uint32_t xb = uint32_t(__builtin_bit_cast(uint16_t, (_Float16)xf));
          radd(rb, (gptr(pr.ridx)[T * pr.nS + s] >> gsh) & 3u, xb);
        }
      }
    }
    // the next unit's activations into the other buffer (its last readers,
    // the previous unit's build and residual, are behind the last barrier)
    if (!ONE || has_next) stage(nxt, sb ^ 1);
    if (take && tid == 0) {
      // a take past the plan's count (a queue counter left over from a call
      // that did not complete) yields no chunk and is reported
      const bool ok = taken < n_grabs;
      *cnext_lds = ok ? 2 * G + int(taken) : NC;
      if (!ok) __hip_atomic_fetch_or(counters + 1, kQueueStale, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (pend) {
      // the group's four row sums over its QR lanes (shuffles, fixed order)
      float r4[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        float h = racc[k];
        if (QR == 4) h += __shfl_xor(h, 16);
        h += __shfl_xor(h, 32);
        r4[k] = F8 ? h * 256.0f : h;  // E4M3 sums were taken at 2^-8
      }
      if (rq == 0) {
#pragma unroll
        for (int k = 0; k < 4; ++k) rres[4 * gi + k] = r4[k];
      }
    }
    __syncthreads();

    // 5. panel end: y = alpha * acc + residual (or a partial of a split panel)
    if (pend) {
      float tot[RB];
#pragma unroll
      for (int t = 0; t < RB; ++t) {
        const float s2 = acc[t] + __shfl_xor(acc[t], 16);
        tot[t] = s2 + __shfl_xor(s2, 32);
        acc[t] = 0.0f;
      }
      float val[RF];
      int prow[RF];
#pragma unroll
      for (int i = 0; i < RF; ++i) {
        const int tq = q + 4 * i;
        float mine = tot[0];
#pragma unroll
        for (int t = 1; t < RB; ++t)
          if (tq == t) mine = tot[t];
        prow[i] = (w + kGW * tq) * 16 + l16;
        val[i] = (G128 ? mine : h2f(al[i]) * mine) + rres[prow[i]];  // layout 4: scaled per unit
      }
      gf32* y = (gf32*)pr.y;
      const int64_t row0 = int64_t(cur.panel) * RP;
      const bool owned = pstart_slice == 0 && cur.slice == pr.n_slices - 1;
      if (owned) {
#pragma unroll
        for (int i = 0; i < RF; ++i)
          if (row0 + prow[i] < pr.N) y[row0 + prow[i]] = val[i];
      } else if constexpr (ONE) {
        // split panel of a single problem: this run's part goes to its slot
        // (2g, or 2g + 1 for a part starting after the run's first unit) with
        // device-coherent stores, and the last of the panel's workgroups to
        // arrive sums the parts in run order
        // (one row per lane: device-scope stores that write through, which
        // measured faster here than plain stores and a release at the
        // arrival, whose write-back of the XCD's L2 dominates so few bytes)
        float* dst = part + (2 * int64_t(g) + (part_at_chunk_start ? 0 : 1)) * RP;
#pragma unroll
        for (int i = 0; i < RF; ++i) store_coherent(dst + prow[i], val[i]);
        const int64_t ns = one.pr.n_slices, p0 = int64_t(cur.panel) * ns;
        const int ga = one_owner(p0, one.n_units, G), gb = one_owner(p0 + ns - 1, one.n_units, G);
        __builtin_amdgcn_s_waitcnt(0);  // the part is complete before its arrival is counted
        __syncthreads();
        if (tid == 0) {
          const uint32_t before = __hip_atomic_fetch_add(counters + cur.panel, 1u, __ATOMIC_RELAXED,
                                                         __HIP_MEMORY_SCOPE_AGENT);
          const bool last = before == uint32_t(gb - ga);
          if (last) __hip_atomic_store(counters + cur.panel, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          flag[2] = last;
        }
        __syncthreads();
        if (flag[2]) {
          const int odd0 = one_first(ga, one.n_units, G) < p0 ? 1 : 0;
          // LDS scratch: the table region, free until the next unit's build
          sum_parts<kGT>(part, RP, ga, gb, odd0, reinterpret_cast<float4*>(lds), [&](int e, float4 v) {
            if (row0 + e < pr.N) {  // N % 4 == 0: four rows all in or all out
#pragma unroll
              for (int i = 0; i < 4; ++i) y[row0 + e + i] = v[i];
            }
          });
        }
      } else {
        // split panel: this chunk's part goes to its partial slot (2c for a
        // part holding the chunk's first unit, 2c + 1 for a part starting
        // later in the chunk); grouped_reduce_kernel sums the parts after
        // the launch, in chunk order
        gf32* dst = (gf32*)(part + (2 * int64_t(c) + (part_at_chunk_start ? 0 : 1)) * RP);
#pragma unroll
        for (int i = 0; i < RF; ++i) dst[prow[i]] = val[i];
      }
    }
    if (!has_next) break;
    if (take) ctaken = __builtin_amdgcn_readfirstlane(*cnext_lds);  // written before the last barrier
    chunk_first = chunk_last;
    if (chunk_last) {
      my_sum += chunk_tag(uint32_t(cn));
      c = cn;
      u = rec_cn.ub;
      ue = rec_cn.ue;
      cn = ctaken;
      ctaken = NC;
    } else {
      ++u;
    }
    s_lo_c = __builtin_amdgcn_readlane(spv, 0);
    s_hi_c = __builtin_amdgcn_readlane(spv, 1);
    load_res(nxt, s_lo_c, s_hi_c);  // after the last use of this unit's residual values
    if (!G128) load_alpha(nxt, al);  // and of its row scales
    cur = nxt;
  }
  if constexpr (!ONE) queue_exit(counters, n_grabs, exit_sum, my_sum);
}

// Sums the parts of every split panel in chunk order (deterministic) and
// writes its rows of y: one workgroup per split panel, four consecutive
// rows per thread and batch row (16-byte loads of every part), kRedBatch
// parts' loads in flight at a time.
constexpr int kRedBatch = 8;

template <int RP>
__global__ __launch_bounds__(RP / 4) void grouped_reduce_kernel(const GSplit* __restrict__ splits, const int B,
                                                                const float* __restrict__ part) {
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  // the split record is the only load before the parts' (it names y)
  const GSplit sd = splits[blockIdx.x];
  if (sd.y == nullptr) return;  // no record (a launch wider than the plan's split count)
  const int row = 4 * threadIdx.x;
  for (int b = 0; b < B; ++b) {  // a part's partial rows: [batch row][RP]
    f32x4 sum = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int k0 = sd.ga; k0 <= sd.gb; k0 += kRedBatch) {
      f32x4 t[kRedBatch];
#pragma unroll
      for (int j = 0; j < kRedBatch; ++j) {
        const int k = min(k0 + j, sd.gb);
        const int64_t slot = 2 * int64_t(k) + (k == sd.ga ? sd.ga_odd : 0);
        t[j] = *reinterpret_cast<const f32x4*>(part + (slot * B + b) * RP + row);
      }
#pragma unroll
      for (int j = 0; j < kRedBatch; ++j)
        if (k0 + j <= sd.gb) sum += t[j];
    }
    float* y = sd.y + int64_t(b) * sd.ystride;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (row + i < sd.rows) y[row + i] = sum[i];
  }
}

// ---------------------------------------------------------------------------
// Host planning.
// ---------------------------------------------------------------------------
template <int RB, bool F8, bool G128 = false, bool ONE = false>
hipError_t set_lds_attr() {
  static bool done = false;
  if (!done) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&grouped_gemv_kernel<RB, F8, G128, ONE>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, GLds<RB>::BYTES);
    if (e != hipSuccess) return e;
    done = true;
  }
  return hipSuccess;
}

int cu_count() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return n;
}

// Workgroups of the launch: kWgPerCu per CU when that many fit (they do on
// gfx950: 160 KB of LDS, 16 waves of at most 128 VGPRs), else one per CU.
// The kernel never waits for another workgroup, so any grid is correct.
int grid_size() {
  int dev = 0, n = 0, per = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (set_lds_attr<kMaxRB, false>() != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, reinterpret_cast<const void*>(&grouped_gemv_kernel<kMaxRB, false>),
                                                   kGT, GLds<kMaxRB>::BYTES) != hipSuccess)
    return 0;
  return n * std::max(1, std::min(per, kWgPerCu));
}

template <int RB, bool F8, bool G128 = false>
hipError_t launch_grouped(const uint8_t* plan, int grid, const GSplit* splits, int n_splits, float* part,
                          uint32_t* counters, hipStream_t st) {
  const hipError_t e = set_lds_attr<RB, F8, G128>();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((grouped_gemv_kernel<RB, F8, G128>), dim3(grid), dim3(kGT), GLds<RB>::BYTES, st, plan,
                     part, counters, GOne{});
  if (n_splits > 0) {
    constexpr int RP = GLds<RB>::RP;
    hipLaunchKernelGGL(grouped_reduce_kernel<RP>, dim3(n_splits), dim3(RP / 4), 0, st, splits, 1, part);
  }
  return hipGetLastError();
}

// Launch shape of one matrix on its own: batch 1 runs the table kernel on
// 512-row panels, two workgroups per CU at most; batch 2..16 the matrix-core
// kernel on 512-row panels, one workgroup per CU at most.
constexpr int kOneRB = 4;
static_assert(GLds<kOneRB>::RP == kRowsPerRB * kOneRB && GLds<kMaxRB>::RP == kRowsPerRB * kMaxRB,
              "panel heights of the planner");
bool one_shape(const qtea_desc& d, int batch, OneShape* o) {
  return one_shape_for(d, batch, batch == 1 ? grid_size() : cu_count(),
                       batch == 1 ? GLds<kOneRB>::RP : one_mma_rows_per_panel(batch), o);
}

template <bool F8, bool G128>
hipError_t launch_one_b1(const GOne& one, int grid, float* part, uint32_t* counters, hipStream_t st) {
  const hipError_t e = set_lds_attr<kOneRB, F8, G128, true>();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((grouped_gemv_kernel<kOneRB, F8, G128, true>), dim3(grid), dim3(kGT), GLds<kOneRB>::BYTES, st,
                     nullptr, part, counters, one);
  return hipGetLastError();
}

// One matrix on its own (arguments checked by the caller): the panels'
// arrival counters at `counters` (zero on entry, left at zero), the partial
// rows of split panels at `part` (2 grid slots of rp x batch floats).
int one_launch(const qtea_desc& d, const void* packed, const uint16_t* X, int batch, float* Y, const OneShape& o,
               uint32_t* counters, float* part, hipStream_t st) {
  const bool f8 = d.layout != kLayout, g128 = d.layout == kLayoutG128;
  GOne one{};
  fill_problem(d, packed, X, Y, o.rp, one.pr);
  one.n_units = int32_t(o.n_units);
  one.batch = batch;
  hipError_t e;
  if (batch > 1)
    e = launch_one_mma(one, o.grid, f8, part, counters, st);
  else if (g128)
    e = launch_one_b1<true, true>(one, o.grid, part, counters, st);
  else
    e = f8 ? launch_one_b1<true, false>(one, o.grid, part, counters, st)
           : launch_one_b1<false, false>(one, o.grid, part, counters, st);
  return e == hipSuccess ? QTEA_OK : QTEA_ERR_HIP;
}

// The allocation-free variant's workspace: a file-scope device array, one
// copy per GPU, held until the process ends.  Host code never passes the
// array's name to a kernel (on the host it is only a stand-in for the
// symbol): the device address comes from hipGetSymbolAddress, once per
// device with that device current, and is kept per device.  Layout: the
// panels' arrival counters in the first kNoallocCounterBytes (zero-filled
// once, at the first call on the device, and left at zero by every call that
// completes), then the partial rows.
constexpr int64_t kNoallocCounterBytes = 65536;
static __device__ __align__(256) uint8_t scratch[QTEA_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_on_current_device(void** out, hipStream_t st) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return QTEA_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return QTEA_ERR_HIP;
    // a fill kernel (not a memset node) on the caller's stream, ordered
    // before this call's kernels
    const int rc = qtea_workspace_init(p, kNoallocCounterBytes, st);
    if (rc != QTEA_OK) return rc;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return QTEA_OK;
}

}  // namespace

extern "C" {

int qtea_grouped_plan_bytes(int n_problems, int64_t* out_bytes) {
  if (!out_bytes || n_problems < 1 || n_problems > (1 << 24)) return QTEA_ERR_INVALID_ARG;
  const int G = grid_size();
  if (G < 1) return QTEA_ERR_HIP;
  // room for the grouped format at any batch: one batch-1 problem per row
  *out_bytes = plan_bytes_for(n_problems * QTEA_MAX_BATCH, G);
  return QTEA_OK;
}

int qtea_grouped_plan(const qtea_desc* descs, const void* const* packed, const uint16_t* const* x,
                      float* const* y, int n_problems, int batch, void* plan, int64_t plan_bytes,
                      qtea_grouped_info* info, void* stream) {
  if (!descs || !packed || !x || !y || !plan || !info || n_problems < 1) return QTEA_ERR_INVALID_ARG;
  info->magic = 0;
  if (batch < 1 || batch > QTEA_MAX_BATCH) return QTEA_ERR_BATCH;
  int64_t cap = 0;
  const int st_plan = qtea_grouped_plan_bytes(n_problems, &cap);
  if (st_plan != QTEA_OK) return st_plan;
  if (plan_bytes < cap) return QTEA_ERR_WORKSPACE;
  // The grouped format at batch B: one batch-1 problem per activation row
  // (row b of problem m reads x_m + b K_m and writes y_m + b N_m), so that
  // its per-group scales and biases stay in the table kernel.
  std::vector<qtea_desc> d_rows;
  std::vector<const void*> p_rows;
  std::vector<const uint16_t*> x_rows;
  std::vector<float*> y_rows;
  if (descs[0].layout == kLayoutG128 && batch > 1) {
    for (int m = 0; m < n_problems; ++m) {
      if (!x[m] || !y[m]) return QTEA_ERR_INVALID_ARG;
      for (int b = 0; b < batch; ++b) {
        d_rows.push_back(descs[m]);
        p_rows.push_back(packed[m]);
        x_rows.push_back(x[m] + int64_t(b) * descs[m].K);
        y_rows.push_back(y[m] + int64_t(b) * descs[m].N);
      }
    }
    descs = d_rows.data();
    packed = p_rows.data();
    x = x_rows.data();
    y = y_rows.data();
    n_problems *= batch;
    batch = 1;
  }
  // batch 1: the table kernel, two workgroups per CU and the chunk queue;
  // batch 2..16: the matrix-core kernel, one workgroup per CU and one
  // static run of units each
  const int G = batch > 1 ? cu_count() : grid_size();
  if (G < 1) return QTEA_ERR_HIP;
  const int64_t need = plan_bytes_for(n_problems, G);
  if (need > cap) return QTEA_ERR_WORKSPACE;
  uint8_t* hbuf = static_cast<uint8_t*>(malloc(size_t(need)));
  if (!hbuf) return QTEA_ERR_INVALID_ARG;
  const int rc = plan_write(descs, packed, x, y, n_problems, batch, G, grouped_mma_rows_per_panel(batch), hbuf, need,
                            info);
  if (rc != QTEA_OK) {
    free(hbuf);
    return rc;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(plan, hbuf, size_t(need), hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  free(hbuf);
  if (e != hipSuccess) return QTEA_ERR_HIP;
  info->magic = kGPlanMagic;
  return QTEA_OK;
}

int qtea_workspace_bytes(const qtea_desc* desc, int batch, int64_t* out_bytes) {
  if (!out_bytes || !desc_ok(desc)) return QTEA_ERR_INVALID_ARG;
  if (batch < 1 || batch > QTEA_MAX_BATCH) return QTEA_ERR_BATCH;
  // the grouped format runs its batch rows one after another through the
  // batch-1 kernel: the batch-1 workspace serves every batch
  OneShape o;
  if (!one_shape(*desc, desc->layout == kLayoutG128 ? 1 : batch, &o)) return QTEA_ERR_HIP;
  *out_bytes = o.ws_bytes;
  return QTEA_OK;
}

int qtea_gemm_lowbatch(const qtea_desc* desc, const void* packed, const uint16_t* X, int batch,
                       float* Y, void* workspace, int64_t workspace_bytes, void* stream) {
  if (!desc_ok(desc) || !packed || !X || !Y || !offsets_fit(*desc)) return QTEA_ERR_INVALID_ARG;
  if (batch < 1 || batch > QTEA_MAX_BATCH) return QTEA_ERR_BATCH;
  const bool rows = desc->layout == kLayoutG128;  // grouped format: one batch-1 launch per row
  OneShape o;
  if (!one_shape(*desc, rows ? 1 : batch, &o)) return QTEA_ERR_HIP;
  if (!workspace || workspace_bytes < o.ws_bytes) return QTEA_ERR_WORKSPACE;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  for (int b = 0; b < (rows ? batch : 1); ++b) {
    const int rc = one_launch(*desc, packed, X + b * desc->K, rows ? 1 : batch, Y + b * desc->N, o,
                              reinterpret_cast<uint32_t*>(ws), reinterpret_cast<float*>(ws + o.off_part),
                              static_cast<hipStream_t>(stream));
    if (rc != QTEA_OK) return rc;
  }
  return QTEA_OK;
}

int qtea_gemv(const qtea_desc* desc, const void* packed, const uint16_t* x, float* y, void* workspace,
              int64_t workspace_bytes, void* stream) {
  return qtea_gemm_lowbatch(desc, packed, x, 1, y, workspace, workspace_bytes, stream);
}

int qtea_gemm_lowbatch_noalloc(const qtea_desc* desc, const void* packed, const uint16_t* X, int batch, float* Y,
                               void* stream) {
  if (!desc_ok(desc) || !packed || !X || !Y || !offsets_fit(*desc)) return QTEA_ERR_INVALID_ARG;
  if (batch < 1 || batch > QTEA_MAX_BATCH) return QTEA_ERR_BATCH;
  const bool rows = desc->layout == kLayoutG128;  // grouped format: one batch-1 launch per row
  OneShape o;
  if (!one_shape(*desc, rows ? 1 : batch, &o)) return QTEA_ERR_HIP;
  const int64_t part_bytes = o.ws_bytes - o.off_part;
  if (4 * int64_t(o.n_panels) > kNoallocCounterBytes || part_bytes > QTEA_NOALLOC_SCRATCH_BYTES - kNoallocCounterBytes)
    return QTEA_ERR_WORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  void* p = nullptr;
  const int rc = scratch_on_current_device(&p, st);
  if (rc != QTEA_OK) return rc;
  uint8_t* ws = static_cast<uint8_t*>(p);
  for (int b = 0; b < (rows ? batch : 1); ++b) {
    const int rc2 = one_launch(*desc, packed, X + b * desc->K, rows ? 1 : batch, Y + b * desc->N, o,
                               reinterpret_cast<uint32_t*>(ws), reinterpret_cast<float*>(ws + kNoallocCounterBytes), st);
    if (rc2 != QTEA_OK) return rc2;
  }
  return QTEA_OK;
}

int qtea_grouped_status(const void* workspace, uint32_t* flags, void* stream) {
  if (!workspace || !flags) return QTEA_ERR_INVALID_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint32_t h = 0;
  if (hipMemcpyAsync(&h, static_cast<const uint32_t*>(workspace) + 1, 4, hipMemcpyDeviceToHost, st) != hipSuccess)
    return QTEA_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return QTEA_ERR_HIP;
  *flags = h;
  return QTEA_OK;
}

int qtea_grouped_gemv(const qtea_grouped_info* info, const void* plan, void* workspace,
                      int64_t workspace_bytes, void* stream) {
  if (!info || info->magic != kGPlanMagic || !plan) return QTEA_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < info->workspace_bytes) return QTEA_ERR_WORKSPACE;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  uint32_t* counters = reinterpret_cast<uint32_t*>(ws);
  float* part = reinterpret_cast<float*>(ws + kAlign);
  const uint8_t* pl = static_cast<const uint8_t*>(plan);
  if (info->n_problems < 1 || info->grid < 1 || info->grid > kMaxPlanGrid || info->n_split_panels < 0 ||
      info->n_split_panels > kMaxChunksPerWg * info->grid)
    return QTEA_ERR_INVALID_ARG;
  // the split records, where the planner put them for this plan's shape
  const GSplit* splits = reinterpret_cast<const GSplit*>(pl + plan_off_splits(info->n_problems, info->grid));
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (info->layout != kLayout && info->layout != kLayoutE4M3 && info->layout != kLayoutG128)
    return QTEA_ERR_INVALID_ARG;
  const bool f8 = info->layout != kLayout, g128 = info->layout == kLayoutG128;
  if (g128 && info->batch != 1) return QTEA_ERR_INVALID_ARG;
  hipError_t e;
  if (info->batch > 1) {
    const int rp = grouped_mma_rows_per_panel(info->batch);
    if (info->rows_per_panel != rp || (rp != 1024 && rp != 768)) return QTEA_ERR_INVALID_ARG;
    e = launch_grouped_mma(pl, info->grid, info->batch, f8, part, st);
    if (e == hipSuccess && info->n_split_panels > 0) {
      if (rp == 1024)
        hipLaunchKernelGGL(grouped_reduce_kernel<1024>, dim3(info->n_split_panels), dim3(1024 / 4), 0, st, splits,
                           info->batch, part);
      else
        hipLaunchKernelGGL(grouped_reduce_kernel<768>, dim3(info->n_split_panels), dim3(768 / 4), 0, st, splits,
                           info->batch, part);
      e = hipGetLastError();
    }
    return e == hipSuccess ? QTEA_OK : QTEA_ERR_HIP;
  }
  if (g128) {
    switch (info->rows_per_panel) {
      case GLds<4>::RP: e = launch_grouped<4, true, true>(pl, info->grid, splits, info->n_split_panels, part, counters, st); break;
      case GLds<8>::RP: e = launch_grouped<8, true, true>(pl, info->grid, splits, info->n_split_panels, part, counters, st); break;
      default: return QTEA_ERR_INVALID_ARG;
    }
    return e == hipSuccess ? QTEA_OK : QTEA_ERR_HIP;
  }
  switch (info->rows_per_panel * (f8 ? -1 : 1)) {
    case GLds<4>::RP: e = launch_grouped<4, false>(pl, info->grid, splits, info->n_split_panels, part, counters, st); break;
    case GLds<8>::RP: e = launch_grouped<8, false>(pl, info->grid, splits, info->n_split_panels, part, counters, st); break;
    case -GLds<4>::RP: e = launch_grouped<4, true>(pl, info->grid, splits, info->n_split_panels, part, counters, st); break;
    case -GLds<8>::RP: e = launch_grouped<8, true>(pl, info->grid, splits, info->n_split_panels, part, counters, st); break;
    default: return QTEA_ERR_INVALID_ARG;
  }
  return e == hipSuccess ? QTEA_OK : QTEA_ERR_HIP;
}

}  // extern "C"
