// Plan records of the grouped GEMV and the host planner that writes them:
// plain C++ with no device code and no runtime calls, so that the planner
// runs unchanged in host-only programs (the plan checks, built with the host
// address and undefined-behaviour sanitizers) and in the library, which
// passes in the grid size it queried from the device.  Internal to the
// library.
//
// Work is cut into units: one unit is one panel of rows (a multiple of 64)
// times one K slice of four 80-column groups (320 device columns), the
// share of the product y = W x (Eq. 10 / Eq. 11) that one workgroup computes
// with one lookup table (the batch-1 kernel) or one set of decode images
// (the matrix-core kernel).  A problem's units are numbered panel-major, its
// slices innermost.
#ifndef QTEA_PLAN_HOST_H_
#define QTEA_PLAN_HOST_H_

#include <stdint.h>
#include <stdlib.h>

#include <algorithm>
#include <vector>

#include "layout.h"
#include "qtea.h"

#ifdef __HIP__
#define QTEA_HD __attribute__((host, device, always_inline)) inline
#else
#define QTEA_HD inline
#endif

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
// panel whose units fall in more than one run is summed in run order: at
// batch 1 by the last of its workgroups to arrive (a counter per panel in
// the workspace), at batch 2..16 by a small reduce kernel after the launch.
struct GOne {
  GProblem pr;
  int32_t n_units;
  int32_t batch;
  int32_t reserved[2];
};

// Workgroup whose run holds unit x, for U units over G runs: the largest g
// with floor(g U / G) <= x.
QTEA_HD int one_owner(int64_t x, int64_t U, int64_t G) { return int(((x + 1) * G - 1) / U); }
QTEA_HD int64_t one_first(int64_t g, int64_t U, int64_t G) { return (g * U) / G; }

struct GPlanHeader {
  uint32_t magic, version;
  int32_t n_problems, n_wg, rows_per_panel, max_parts, batch, n_chunks;
  int64_t n_units, off_chunks, n_grabs, off_splits, n_splits;
  int32_t f8, reserved;  // f8: residual values are E4M3 bytes (layout 3) in every problem
  uint64_t exit_sum;     // sum of chunk_tag(c) over the chunks: what one complete launch adds up
};
static_assert(sizeof(GPlanHeader) <= kPlanProblemsOff, "plan header");

// The tag a chunk adds to the batch-1 kernel's exit word: the MurmurHash3
// 32-bit finalizer of its index + 1, so that left-over queue words cancel
// the tags of skipped chunks only by a coincidence of hashes.
QTEA_HD uint32_t chunk_tag(uint32_t c) {
  uint32_t h = c + 1u;
  h ^= h >> 16;
  h *= 0x85ebca6bu;
  h ^= h >> 13;
  h *= 0xc2b2ae35u;
  h ^= h >> 16;
  return h;
}

// A chunk: units [ub, ue), the first of them at (problem m, panel, slice).
struct GChunk {
  int32_t ub, ue, m, panel, slice, reserved[3];
};
static_assert(sizeof(GChunk) == 32, "one scalar load per chunk record");

// A panel whose slices fall in more than one chunk: its parts are in the
// partial slots of chunks ga..gb (slot 2k, except 2ga + 1 when the part in
// chunk ga starts after that chunk's first unit).  y is the panel's first
// output row of batch row 0, rows the panel's rows that are rows of y, and
// ystride the batch-row stride of y (N): the reduce kernel needs no other
// record.  m is the problem's index in the plan.
struct GSplit {
  float* y;
  int32_t rows, ystride, ga, gb, ga_odd, m;
};
static_assert(sizeof(GSplit) == 32, "one scalar load per split record");

// Rows per panel of the batch-1 kernel are kRowsPerRB times its row blocks
// per wave (4 or 8); the matrix-core kernel's panel height is its own.
constexpr int kMaxRB = 8;
constexpr int kRowsPerRB = 128;
// Chunks: the unit list is cut into chunks whose sizes shrink from about
// kGuideDen/(kGuideNum G) of the remaining work to a single unit (guided
// self-scheduling), at most kMaxChunksPerWg per workgroup on average.
// Measured on the 8B, 14B and 70B stacks at batch 1 (with takes at a
// chunk's second-to-last unit): 5/2 is best or within 0.5% on the 8B and
// 14B stacks and the grouped format; 3 is 1.7% faster on the 70B stack;
// 2 is within noise of 5/2 on the 8B stack; 3/2 and 1 are 3 to 4% slower.
constexpr int kGuideNum = 5, kGuideDen = 2;
constexpr int kMaxChunksPerWg = 16;
constexpr int kMaxPlanGrid = 4096;

inline int units_for(const qtea_desc& d, int RP, int* n_slices, int* n_panels) {
  *n_slices = int(cdiv(d.n_groups, kSliceGroups));
  *n_panels = int(cdiv(d.n_pad, RP));
  return *n_slices * *n_panels;
}

// The problem record of one packed matrix with its activations and outputs
// (the descriptor passed desc_ok).
inline void fill_problem(const qtea_desc& d, const void* packed, const uint16_t* x, float* y, int RP,
                         GProblem& pr) {
  const uint8_t* pk = static_cast<const uint8_t*>(packed);
  pr = GProblem{};
  pr.trits = pk + d.off_trits;
  pr.alpha = reinterpret_cast<const uint16_t*>(pk + d.off_alpha);
  pr.v = reinterpret_cast<const uint16_t*>(pk + d.off_v);
  pr.S = reinterpret_cast<const int32_t*>(pk + d.off_salient);
  pr.spos = reinterpret_cast<const int32_t*>(pk + d.off_spos);
  pr.rval = reinterpret_cast<const uint16_t*>(pk + d.off_rval);
  pr.ridx = reinterpret_cast<const uint32_t*>(pk + d.off_ridx);
  Layout lm;  // regions the descriptor does not list
  make_layout(d.N, d.K, d.n_salient, &lm, int(d.layout));  // succeeds: desc_ok checked it
  pr.vs = reinterpret_cast<const uint32_t*>(pk + lm.off_vs);
  pr.x = x;
  pr.y = y;
  pr.N = d.N;
  pr.K = d.K;
  pr.n_pad = d.n_pad;
  pr.n_groups = int32_t(d.n_groups);
  pr.nS = int32_t(d.n_salient);
  int ns, np;
  units_for(d, RP, &ns, &np);
  pr.n_slices = ns;
  pr.n_panels = np;
  pr.unit_base = 0;
}

// The kernels address the packed bytes and the residual with 32-bit offsets.
inline bool offsets_fit(const qtea_desc& d) {
  const int64_t trit_bytes = d.n_pad * d.n_groups * kGroupPacks;
  const int64_t resid_bytes = (d.n_pad / 4) * d.n_salient * (d.layout == kLayout ? 2 : 1);
  return trit_bytes < (int64_t(1) << 31) && resid_bytes < (int64_t(1) << 31);
}

// Launch shape of one matrix on its own (qtea_gemv, qtea_gemm_lowbatch) over
// at most max_wg workgroups of rp-row panels.  Every workgroup takes the
// same number of units (the least that fits the grid), so no workgroup
// carries more than the others.  The workspace holds one arrival counter
// per panel (used at batch 1), then two partial-row slots per workgroup.
struct OneShape {
  int rp, n_panels, n_slices, grid;
  int64_t n_units, off_part, ws_bytes;
};
inline bool one_shape_for(const qtea_desc& d, int batch, int max_wg, int rp, OneShape* o) {
  if (max_wg < 1 || rp < 64 || rp % 64 != 0) return false;
  o->rp = rp;
  o->n_units = units_for(d, o->rp, &o->n_slices, &o->n_panels);
  const int64_t per = cdiv(o->n_units, max_wg);
  o->grid = int(cdiv(o->n_units, per));
  o->off_part = align_up(4 * int64_t(o->n_panels), kAlign);
  o->ws_bytes = o->off_part + 2 * int64_t(o->grid) * o->rp * batch * 4;
  return true;
}

// Layout of the plan of n_problems problems for a launch of G workgroups:
// header, problem records, chunk records from plan_off_chunks, split
// records from plan_off_splits, plan_bytes_for bytes in all.
inline int64_t plan_off_chunks(int n_problems) {
  return align_up(kPlanProblemsOff + int64_t(sizeof(GProblem)) * n_problems, kAlign);
}
inline int64_t plan_off_splits(int n_problems, int G) {
  return plan_off_chunks(n_problems) + align_up(int64_t(sizeof(GChunk)) * kMaxChunksPerWg * G, kAlign);
}
inline int64_t plan_bytes_for(int n_problems, int G) {
  return plan_off_splits(n_problems, G) + int64_t(sizeof(GSplit)) * kMaxChunksPerWg * G;
}

// The plan of a grouped launch, written into hbuf (hbytes bytes, at least
// plan_bytes_for(n_problems, G)): G workgroups (two per CU for the batch-1
// kernel, one per CU for the matrix-core kernel at batch 2..16), mma_rows
// the matrix-core kernel's panel height.  Fills every field of *info but
// the magic, which the caller sets once the plan is on the device.
// Returns QTEA_OK, or the status of the first argument found wrong.
inline int plan_write(const qtea_desc* descs, const void* const* packed, const uint16_t* const* x,
                      float* const* y, int n_problems, int batch, int G, int mma_rows, uint8_t* hbuf,
                      int64_t hbytes, qtea_grouped_info* info) {
  if (!descs || !packed || !x || !y || !hbuf || !info || n_problems < 1) return QTEA_ERR_INVALID_ARG;
  if (batch < 1 || batch > QTEA_MAX_BATCH) return QTEA_ERR_BATCH;
  // at most 16 G chunks: the batch-1 kernel's exit word holds the count of
  // workgroups in 16 bits and the sum of at most 16 G 32-bit tags in 48
  if (G < 1 || G > kMaxPlanGrid) return QTEA_ERR_INVALID_ARG;
  const int64_t need = plan_bytes_for(n_problems, G);
  if (hbytes < need) return QTEA_ERR_WORKSPACE;
  const bool mma = batch > 1;
  const uint32_t layout = descs[0].layout;
  if (layout == kLayoutG128 && batch != 1) return QTEA_ERR_BATCH;  // the grouped format runs at batch 1
  for (int m = 0; m < n_problems; ++m) {
    if (!desc_ok(&descs[m]) || !packed[m] || !x[m] || !y[m]) return QTEA_ERR_INVALID_ARG;
    if (descs[m].layout != layout) return QTEA_ERR_INVALID_ARG;  // one residual format per plan
    if (!offsets_fit(descs[m])) return QTEA_ERR_INVALID_ARG;
  }
  std::fill(hbuf, hbuf + need, uint8_t(0));

  // rows per panel: the largest that still gives every workgroup several units
  int RB = kMaxRB;
  for (; !mma && RB > 4; RB /= 2) {
    int64_t units = 0;
    for (int m = 0; m < n_problems; ++m) {
      int ns, np;
      units += units_for(descs[m], kRowsPerRB * RB, &ns, &np);
    }
    if (units >= 4 * int64_t(G)) break;
  }
  const int RP = mma ? mma_rows : kRowsPerRB * RB;

  const int64_t max_chunks = int64_t(kMaxChunksPerWg) * G;
  const int64_t off_chunks = plan_off_chunks(n_problems), off_splits = plan_off_splits(n_problems, G);
  GPlanHeader* H = reinterpret_cast<GPlanHeader*>(hbuf);
  GProblem* P = reinterpret_cast<GProblem*>(hbuf + kPlanProblemsOff);
  GChunk* chunks = reinterpret_cast<GChunk*>(hbuf + off_chunks);
  std::vector<int64_t> ranges(size_t(max_chunks) + 1, 0);  // chunk k holds units [ranges[k], ranges[k + 1])
  GSplit* splits = reinterpret_cast<GSplit*>(hbuf + off_splits);

  // unit costs: packed bytes of the unit plus a fixed table-build share;
  // prefix sums of the costs, and the end (exclusive) of each unit's panel
  std::vector<int64_t> prefix(1, 0), panel_end;
  std::vector<GChunk> ucur;
  int64_t total_units = 0;
  // Problems are laid out with the most K slices per panel first (stable),
  // so that the small chunks at the end of the unit list split panels of
  // few slices.  The kernel only needs each problem's units to be
  // contiguous; outputs are addressed through each problem's own record.
  std::vector<int> order(static_cast<size_t>(n_problems));
  for (int m = 0; m < n_problems; ++m) order[size_t(m)] = m;
  std::stable_sort(order.begin(), order.end(),
                   [&](int a, int b) { return descs[a].n_groups > descs[b].n_groups; });
  for (int m = 0; m < n_problems; ++m) {
    const int src = order[size_t(m)];
    const qtea_desc& d = descs[src];
    int ns, np;
    units_for(d, RP, &ns, &np);
    GProblem& pr = P[m];
    fill_problem(d, packed[src], x[src], y[src], RP, pr);
    pr.unit_base = total_units;
    for (int p = 0; p < np; ++p) {
      const int64_t rows = std::min<int64_t>(RP, d.n_pad - int64_t(p) * RP);
      const int64_t pe = total_units + int64_t(p + 1) * ns;
      for (int s = 0; s < ns; ++s) {
        const int64_t groups = std::min<int64_t>(kSliceGroups, d.n_groups - int64_t(s) * kSliceGroups);
        prefix.push_back(prefix.back() + rows * groups * kGroupPacks + 8192);
        panel_end.push_back(pe);
        ucur.push_back(GChunk{0, 0, m, p, s, {0, 0, 0}});
      }
    }
    total_units += int64_t(ns) * np;
    if (total_units >= (int64_t(1) << 31)) return QTEA_ERR_INVALID_ARG;  // unit indices are 32-bit on the device
  }
  // chunks: guided sizes, a chunk that reaches the end of its panel (or
  // several panels) within half a target taking them whole, so that most
  // small panels are not split
  int64_t n_chunks = 0;
  if (mma) {
    // one contiguous run of balanced cost per workgroup
    const int64_t total_cost = prefix.back();
    int64_t u = 0;
    ranges[0] = 0;
    for (int k = 1; k <= G && u < total_units; ++k) {
      int64_t e = k == G ? total_units
                         : int64_t(std::lower_bound(prefix.begin(), prefix.end(), (total_cost * k) / G) - prefix.begin());
      e = std::min(total_units, std::max(e, u + 1));
      chunks[n_chunks] = ucur[size_t(u)];
      chunks[n_chunks].ub = int32_t(u);
      chunks[n_chunks].ue = int32_t(e);
      ranges[size_t(++n_chunks)] = e;
      u = e;
    }
  } else {
    const int64_t total_cost = prefix.back();
    const int64_t unit_min = prefix[1] - prefix[0];
    int64_t u = 0;
    ranges[0] = 0;
    while (u < total_units) {
      const int64_t rem = total_cost - prefix[size_t(u)];
      // every chunk but the last covers at least half its target, so a
      // target of twice the remaining cost per remaining chunk of the budget
      // finishes within the budget with chunks of equal cost, instead of
      // leaving the whole rest to one workgroup
      const int64_t left = max_chunks - n_chunks;
      const int64_t target = std::max({unit_min, rem * kGuideDen / (int64_t(kGuideNum) * G), 2 * rem / left});
      int64_t e = u;
      if (n_chunks + 1 == max_chunks) {
        e = total_units;  // chunk budget spent: the rest is one chunk
      } else {
        while (e < total_units) {
          const int64_t pe = panel_end[size_t(e)];
          const int64_t have = prefix[size_t(e)] - prefix[size_t(u)];
          if (have + prefix[size_t(pe)] - prefix[size_t(e)] <= target + target / 2) {
            e = pe;  // the rest of this panel fits
            if (prefix[size_t(e)] - prefix[size_t(u)] >= target) break;
            continue;
          }
          if (e > u && have >= target / 2) break;  // cut at the panel boundary
          while (e < pe && prefix[size_t(e)] - prefix[size_t(u)] < target) ++e;
          break;
        }
      }
      chunks[n_chunks] = ucur[size_t(u)];
      chunks[n_chunks].ub = int32_t(u);
      chunks[n_chunks].ue = int32_t(e);
      ranges[size_t(++n_chunks)] = e;
      u = e;
    }
  }
  // split panels (a chunk is the first chunk of at most one of them, so
  // there are at most n_chunks), and the largest number of parts of one
  int max_parts = 1;
  int64_t n_splits = 0;
  for (int m = 0; m < n_problems; ++m) {
    for (int p = 0; p < P[m].n_panels; ++p) {
      const int64_t p0 = P[m].unit_base + int64_t(p) * P[m].n_slices, p1 = p0 + P[m].n_slices;
      const auto rb = ranges.begin(), re = ranges.begin() + n_chunks + 1;
      const int ga = int(std::upper_bound(rb, re, p0) - rb) - 1;
      const int gb = int(std::lower_bound(rb, re, p1) - rb) - 1;
      if (gb > ga) {
        const int64_t row0 = int64_t(p) * RP;
        splits[n_splits++] = GSplit{P[m].y + row0, int32_t(std::min<int64_t>(RP, P[m].N - row0)), int32_t(P[m].N),
                                    ga, gb, p0 > ranges[size_t(ga)] ? 1 : 0, m};
      }
      max_parts = std::max(max_parts, gb - ga + 1);
    }
  }
  // queue takes of one launch: every chunk past the first 2G, plus one
  // final take by each workgroup that has a second chunk
  const int64_t n_grabs = mma ? 0
                              : std::max<int64_t>(0, n_chunks - 2 * int64_t(G)) +
                                    std::min<int64_t>(G, std::max<int64_t>(0, n_chunks - G));
  H->magic = kGPlanMagic;
  H->version = 2;
  H->n_problems = n_problems;
  H->n_wg = G;
  H->rows_per_panel = RP;
  H->max_parts = max_parts;
  H->batch = batch;
  H->n_chunks = int32_t(n_chunks);
  H->n_units = total_units;
  H->off_chunks = off_chunks;
  H->n_grabs = n_grabs;
  H->off_splits = off_splits;
  H->n_splits = n_splits;
  H->f8 = layout != kLayout;
  uint64_t exit_sum = 0;
  for (int64_t c = 0; c < n_chunks; ++c) exit_sum += chunk_tag(uint32_t(c));
  H->exit_sum = exit_sum;

  info->magic = 0;
  info->n_problems = n_problems;
  info->batch = batch;
  info->grid = G;
  info->rows_per_panel = RP;
  info->max_parts = max_parts;
  info->n_chunks = int32_t(n_chunks);
  info->n_split_panels = int32_t(n_splits);
  info->layout = int32_t(layout);
  info->reserved = 0;
  info->n_units = total_units;
  info->plan_bytes = need;
  info->workspace_bytes = kAlign + 2 * n_chunks * RP * int64_t(batch) * 4;
  return QTEA_OK;
}

}  // namespace qtea_grouped

#endif  // QTEA_PLAN_HOST_H_
