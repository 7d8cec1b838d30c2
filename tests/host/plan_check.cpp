// Host checks of the grouped GEMV's plan records, the packed layout's
// regions and the chunk queue's protocol, on the planner code the library
// itself compiles (plan_host.h, layout.h).  Built with the host address and
// undefined-behaviour sanitizers by tests/test_host_plan.py; no device and
// no runtime library.  Prints one line per passed group and exits non-zero
// at the first failed check.
//
// What is checked (every matrix shape of the 8B, 14B and 70B stacks, the
// paper's 128-column format, and edge shapes; grids of 1 to 1024
// workgroups; batch 1 and 2..16):
//   * layout: each region the kernels read (trits, row scales, v, salient
//     list, slice offsets spos[0..n_groups], residual values and positions,
//     the vs words of 4 n_groups 80 bytes) lies inside bytes_total, aligned,
//     and no two overlap; the descriptor the pack entry points return passes
//     desc_ok, and one changed field fails it;
//   * plan records: every pointer of every problem record is its matrix's
//     base plus that region's offset (vs included), x and y are the
//     caller's, each problem's units are contiguous, the chunks cover the
//     unit list once in order and name their first unit, the split records
//     are exactly the panels that span chunks, no two parts share a partial
//     slot and the workspace holds every slot;
//   * the chunk queue (a step-by-step model of the batch-1 kernel's takes
//     and exits under random interleavings): from clean words every chunk
//     runs once, the take count is the plan's n_grabs, no flag is raised and
//     the words are left clean; from left-over words (listed cases and
//     random ones) every chunk index stays in range, and a launch whose
//     chunks did not each run once raises a flag;
//   * one matrix on its own: the workgroup runs partition the units, none
//     empty, one_owner inverts one_first, and the split panels' parts have
//     distinct slots inside the workspace.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <random>
#include <string>
#include <utility>
#include <vector>

#include "plan_host.h"

using namespace qtea_grouped;

namespace {

int g_checks = 0;
#define CHECK(cond, ...)                                                   \
  do {                                                                     \
    ++g_checks;                                                            \
    if (!(cond)) {                                                         \
      fprintf(stderr, "FAIL %s:%d: %s: ", __FILE__, __LINE__, #cond);      \
      fprintf(stderr, __VA_ARGS__);                                        \
      fprintf(stderr, "\n");                                               \
      exit(1);                                                             \
    }                                                                      \
  } while (0)

struct Mat {
  int64_t N, K, nS;
  int layout;
};

struct Region {
  const char* name;
  int64_t off, bytes;
};

// The regions the kernels read, with the sizes the format gives them (one
// byte per pack slot, fp16 row scales or u32 scale-and-bias words per
// 128-column group, fp16 v per device column, i32 salient list, i32 slice
// offsets for groups 0..n_groups, residual values per four-row group and
// salient column, u32 positions per 64-row tile and salient column, u32 vs
// per device column).
std::vector<Region> regions(const qtea_desc& d, const Layout& L) {
  const bool g128 = d.layout == uint32_t(kLayoutG128);
  const int64_t vb = d.layout == uint32_t(kLayout) ? 2 : 1;
  return {
      {"trits", d.off_trits, d.n_pad * d.n_groups * (g128 ? kG128SlotPacks : 16)},
      {"alpha", d.off_alpha, g128 ? 4 * d.n_pad * (d.n_groups / 2) : 2 * d.n_pad},
      {"v", d.off_v, 2 * d.n_groups * 80},
      {"S", d.off_salient, 4 * d.n_salient},
      {"spos", d.off_spos, 4 * (d.n_groups + 1)},
      {"rval", d.off_rval, vb * d.n_salient * (d.n_pad / 4)},
      {"ridx", d.off_ridx, 4 * d.n_salient * (d.n_pad / 64)},
      {"vs", L.off_vs, 4 * d.n_groups * 80},
  };
}

qtea_desc make_desc(const Mat& m, Layout* L) {
  const bool ok = make_layout(m.N, m.K, m.nS, L, m.layout);
  CHECK(ok, "make_layout N=%lld K=%lld nS=%lld layout=%d", (long long)m.N, (long long)m.K, (long long)m.nS,
        m.layout);
  return desc_from_layout(*L, m.N, m.K, m.nS, m.layout);
}

void check_layout(const Mat& m) {
  Layout L;
  const qtea_desc d = make_desc(m, &L);
  CHECK(desc_ok(&d), "desc_ok on the pack's descriptor");
  CHECK(d.n_pad % 64 == 0 && d.n_pad >= d.N && d.n_pad < d.N + 64, "n_pad %lld", (long long)d.n_pad);
  if (m.layout == kLayoutG128) {
    CHECK(d.n_groups == 2 * cdiv(m.K, 128) && d.n_packs == 26 * cdiv(m.K, 128), "g128 groups");
  } else {
    CHECK(d.n_packs == cdiv(m.K, 5) && d.n_groups == cdiv(d.n_packs, 16), "groups");
  }
  std::vector<Region> R = regions(d, L);
  for (const Region& r : R) {
    CHECK(r.off >= kHeaderBytes && r.off % kAlign == 0, "%s offset %lld", r.name, (long long)r.off);
    CHECK(r.off + r.bytes <= d.bytes_total, "%s [%lld, +%lld) past bytes_total %lld", r.name, (long long)r.off,
          (long long)r.bytes, (long long)d.bytes_total);
  }
  for (size_t i = 0; i < R.size(); ++i)
    for (size_t j = i + 1; j < R.size(); ++j) {
      const bool apart = R[i].off + R[i].bytes <= R[j].off || R[j].off + R[j].bytes <= R[i].off;
      CHECK(apart || R[i].bytes == 0 || R[j].bytes == 0, "%s and %s overlap", R[i].name, R[j].name);
    }
  CHECK(d.bytes_total % kAlign == 0, "bytes_total alignment");
  // one changed field and the descriptor is refused
  int64_t qtea_desc::*fields[] = {&qtea_desc::N,         &qtea_desc::K,         &qtea_desc::n_salient,
                                        &qtea_desc::n_packs,   &qtea_desc::n_groups,  &qtea_desc::n_pad,
                                        &qtea_desc::bytes_total, &qtea_desc::off_trits, &qtea_desc::off_alpha,
                                        &qtea_desc::off_v,     &qtea_desc::off_salient, &qtea_desc::off_spos,
                                        &qtea_desc::off_rval,  &qtea_desc::off_ridx};
  for (auto f : fields) {
    qtea_desc e = d;
    e.*f += 256;
    CHECK(!desc_ok(&e), "a descriptor with one field moved was accepted");
  }
  qtea_desc e = d;
  e.magic ^= 1u;
  CHECK(!desc_ok(&e), "bad magic accepted");
  e = d;
  e.layout = 5;
  CHECK(!desc_ok(&e), "an unknown layout version accepted");
}

// Fake device addresses: each matrix, activation and output buffer at its own
// 2^40-byte-aligned base, never dereferenced.
uintptr_t base_of(int kind, int m) { return (uintptr_t(1) << 44) + (uintptr_t(kind) << 42) + (uintptr_t(m) << 32); }

uint64_t tag_sum(int NC) {
  uint64_t t = 0;
  for (int c = 0; c < NC; ++c) t += chunk_tag(uint32_t(c));
  return t;
}

struct PlanOut {
  std::vector<uint8_t> buf;
  qtea_grouped_info info;
  std::vector<qtea_desc> descs;
  std::vector<Layout> layouts;
};

int plan(const std::vector<Mat>& mats, int batch, int G, int mma_rows, PlanOut* out) {
  const int n = int(mats.size());
  out->descs.resize(size_t(n));
  out->layouts.resize(size_t(n));
  std::vector<const void*> packed(static_cast<size_t>(n));
  std::vector<const uint16_t*> x(static_cast<size_t>(n));
  std::vector<float*> y(static_cast<size_t>(n));
  for (int m = 0; m < n; ++m) {
    out->descs[size_t(m)] = make_desc(mats[size_t(m)], &out->layouts[size_t(m)]);
    packed[size_t(m)] = reinterpret_cast<const void*>(base_of(0, m));
    x[size_t(m)] = reinterpret_cast<const uint16_t*>(base_of(1, m));
    y[size_t(m)] = reinterpret_cast<float*>(base_of(2, m));
  }
  out->buf.assign(size_t(plan_bytes_for(n, G)), uint8_t(0xa5));  // not zero: the planner clears it
  return plan_write(out->descs.data(), packed.data(), x.data(), y.data(), n, batch, G, mma_rows, out->buf.data(),
                    int64_t(out->buf.size()), &out->info);
}

struct Part {
  int64_t chunk, slot;
};

// rows per panel of the matrix-core kernel at batch 2..16 in a grouped
// launch (its workgroup shape: 1024 threads up to batch 8, 768 above); one
// matrix on its own runs 512-row panels
int mma_rows_for(int batch) { return batch <= 8 ? 1024 : 768; }
constexpr int kOneMmaRows = 512;

void check_plan(const std::vector<Mat>& mats, int batch, int G, const char* what) {
  const int mma_rows = mma_rows_for(batch);
  PlanOut po;
  const int rc = plan(mats, batch, G, mma_rows, &po);
  CHECK(rc == QTEA_OK, "%s: plan_write status %d", what, rc);
  const uint8_t* hb = po.buf.data();
  GPlanHeader H;
  memcpy(&H, hb, sizeof(H));
  const int n = int(mats.size());
  CHECK(H.magic == kGPlanMagic && H.n_problems == n && H.n_wg == G && H.batch == batch, "%s: header", what);
  const int RP = H.rows_per_panel;
  CHECK(batch > 1 ? RP == mma_rows : (RP == 512 || RP == 1024), "%s: rows per panel %d", what, RP);
  CHECK(H.n_chunks >= 1 && H.n_chunks <= int64_t(kMaxChunksPerWg) * G, "%s: n_chunks %d", what, H.n_chunks);
  CHECK(H.off_chunks >= kPlanProblemsOff + int64_t(sizeof(GProblem)) * n && H.off_chunks % kAlign == 0, "off_chunks");
  CHECK(H.off_splits >= H.off_chunks + int64_t(sizeof(GChunk)) * H.n_chunks, "off_splits");
  CHECK(H.off_splits == plan_off_splits(n, G) && H.off_chunks == plan_off_chunks(n), "%s: record offsets", what);
  CHECK(H.off_splits + int64_t(sizeof(GSplit)) * H.n_splits <= int64_t(po.buf.size()), "%s: splits past the plan",
        what);
  CHECK(H.f8 == (mats[0].layout != kLayout ? 1 : 0), "f8");
  CHECK(H.exit_sum == tag_sum(H.n_chunks) && H.exit_sum < (uint64_t(1) << 48), "%s: exit_sum", what);
  CHECK(po.info.n_chunks == H.n_chunks && po.info.n_units == H.n_units && po.info.grid == G &&
            po.info.rows_per_panel == RP && po.info.n_split_panels == H.n_splits && po.info.magic == 0,
        "%s: info mirrors the header", what);

  // problem records: the planner orders problems by K slices (most first,
  // stable); map each record back to its matrix through its base address
  std::vector<GProblem> P(static_cast<size_t>(n));
  memcpy(P.data(), hb + kPlanProblemsOff, sizeof(GProblem) * size_t(n));
  std::vector<int> src(static_cast<size_t>(n), -1), seen(static_cast<size_t>(n), 0);
  int64_t units = 0;
  for (int k = 0; k < n; ++k) {
    const GProblem& pr = P[size_t(k)];
    const uintptr_t b = reinterpret_cast<uintptr_t>(pr.trits) & ~((uintptr_t(1) << 32) - 1);
    const int m = int((b - base_of(0, 0)) >> 32);
    CHECK(m >= 0 && m < n && !seen[size_t(m)], "%s: record %d names no matrix", what, k);
    seen[size_t(m)] = 1;
    src[size_t(k)] = m;
    const qtea_desc& d = po.descs[size_t(m)];
    const Layout& L = po.layouts[size_t(m)];
    if (k > 0) {
      const qtea_desc& dp = po.descs[size_t(src[size_t(k - 1)])];
      CHECK(dp.n_groups > d.n_groups || (dp.n_groups == d.n_groups && src[size_t(k - 1)] < m),
            "%s: problem order", what);
    }
    const uintptr_t base = base_of(0, m);
    auto at = [&](const void* p) { return int64_t(reinterpret_cast<uintptr_t>(p) - base); };
    CHECK(pr.vs != nullptr, "%s: vs unset in record %d", what, k);
    const std::pair<const void*, const char*> ptrs[] = {
        {pr.trits, "trits"}, {pr.alpha, "alpha"}, {pr.v, "v"},   {pr.S, "S"},
        {pr.spos, "spos"},   {pr.rval, "rval"},   {pr.ridx, "ridx"}, {pr.vs, "vs"}};
    const std::vector<Region> R = regions(d, L);
    for (size_t i = 0; i < R.size(); ++i) {
      CHECK(at(ptrs[i].first) == R[i].off, "%s: record %d %s at %lld, region at %lld", what, k, ptrs[i].second,
            (long long)at(ptrs[i].first), (long long)R[i].off);
      CHECK(R[i].off + R[i].bytes <= d.bytes_total, "%s: %s past bytes_total", what, R[i].name);
    }
    CHECK(reinterpret_cast<uintptr_t>(pr.x) == base_of(1, m) && reinterpret_cast<uintptr_t>(pr.y) == base_of(2, m),
          "%s: x or y of record %d", what, k);
    CHECK(pr.N == d.N && pr.K == d.K && pr.n_pad == d.n_pad && pr.n_groups == d.n_groups && pr.nS == d.n_salient,
          "%s: sizes of record %d", what, k);
    CHECK(pr.n_slices == cdiv(d.n_groups, kSliceGroups) && pr.n_panels == cdiv(d.n_pad, RP), "%s: units of %d", what,
          k);
    // a unit's groups 4 s .. 4 s + 3 (clipped) and the slice offsets the
    // kernels read, spos[4 s] and spos[min(4 s + 4, n_groups)], exist
    CHECK(int64_t(kSliceGroups) * (pr.n_slices - 1) < d.n_groups, "%s: last slice starts past the groups", what);
    CHECK(int64_t(pr.n_panels - 1) * RP < d.n_pad, "%s: last panel starts past the rows", what);
    CHECK(pr.unit_base == units, "%s: record %d unit_base", what, k);
    units += int64_t(pr.n_slices) * pr.n_panels;
  }
  CHECK(units == H.n_units, "%s: unit count", what);

  // chunks cover [0, n_units) once, in order, and name their first unit
  std::vector<GChunk> C(size_t(H.n_chunks));
  memcpy(C.data(), hb + H.off_chunks, sizeof(GChunk) * C.size());
  int64_t u = 0;
  for (int c = 0; c < H.n_chunks; ++c) {
    const GChunk& ch = C[size_t(c)];
    CHECK(ch.ub == u && ch.ue > ch.ub && ch.ue <= H.n_units, "%s: chunk %d [%d, %d) after %lld", what, c, ch.ub, ch.ue,
          (long long)u);
    CHECK(ch.m >= 0 && ch.m < n, "%s: chunk %d problem", what, c);
    const GProblem& pr = P[size_t(ch.m)];
    const int64_t local = ch.ub - pr.unit_base;
    CHECK(local >= 0 && local < int64_t(pr.n_slices) * pr.n_panels, "%s: chunk %d outside its problem", what, c);
    CHECK(ch.panel == local / pr.n_slices && ch.slice == local % pr.n_slices, "%s: chunk %d cursor", what, c);
    u = ch.ue;
  }
  CHECK(u == H.n_units, "%s: chunks end at %lld of %lld units", what, (long long)u, (long long)H.n_units);
  if (batch > 1) CHECK(H.n_chunks <= G && H.n_grabs == 0, "%s: one run per workgroup", what);

  // split panels: exactly those spanning chunks, with their first and last
  // chunk and whether the first part starts inside its chunk
  std::vector<int64_t> chunk_of(size_t(H.n_units));
  for (int c = 0; c < H.n_chunks; ++c)
    for (int64_t x = C[size_t(c)].ub; x < C[size_t(c)].ue; ++x) chunk_of[size_t(x)] = c;
  std::vector<GSplit> S(size_t(H.n_splits));
  if (!S.empty()) memcpy(S.data(), hb + H.off_splits, sizeof(GSplit) * S.size());
  int64_t si = 0;
  int max_parts = 1;
  std::vector<char> slot_used(size_t(2 * H.n_chunks), 0);
  for (int m = 0; m < n; ++m) {
    const GProblem& pr = P[size_t(m)];
    for (int p = 0; p < pr.n_panels; ++p) {
      const int64_t p0 = pr.unit_base + int64_t(p) * pr.n_slices, p1 = p0 + pr.n_slices;
      const int ga = int(chunk_of[size_t(p0)]), gb = int(chunk_of[size_t(p1 - 1)]);
      max_parts = std::max(max_parts, gb - ga + 1);
      if (gb == ga) continue;
      CHECK(si < H.n_splits, "%s: a split panel has no record", what);
      const GSplit& s = S[size_t(si++)];
      const int odd = p0 > C[size_t(ga)].ub ? 1 : 0;
      const int64_t row0 = int64_t(p) * RP;
      CHECK(s.m == m && s.y == pr.y + row0 && s.rows == std::min<int64_t>(RP, pr.N - row0) && s.rows > 0 &&
                s.ystride == pr.N && s.ga == ga && s.gb == gb && s.ga_odd == odd,
            "%s: split record of (%d, %d)", what, m, p);
      // partial slots of the parts: 2k, or 2k + 1 for a part that starts
      // after its chunk's first unit; each slot holds one part
      for (int k = ga; k <= gb; ++k) {
        const int64_t slot = 2 * int64_t(k) + (k == ga ? odd : 0);
        CHECK(!slot_used[size_t(slot)], "%s: partial slot %lld used twice", what, (long long)slot);
        slot_used[size_t(slot)] = 1;
      }
    }
  }
  CHECK(si == H.n_splits && H.n_splits <= H.n_chunks, "%s: %lld split records, %lld found", what,
        (long long)H.n_splits, (long long)si);
  CHECK(max_parts == H.max_parts, "%s: max_parts %d, found %d", what, H.max_parts, max_parts);
  CHECK(po.info.workspace_bytes >= kAlign + 2 * int64_t(H.n_chunks) * RP * batch * 4, "%s: workspace", what);
}

// ---------------------------------------------------------------------------
// The chunk queue of the batch-1 kernel, step by step.  Workgroup g starts
// chunk g and has chunk g + G next; once during every chunk that has a next
// one (in the kernel: at its second-to-last unit) it takes a ticket t
// from word 0 (chunk 2G + t if t is below
// the plan's count, else none, and a stale flag); when it has no next chunk
// it adds (1 << 48) + (the tags of the chunks it ran) to the exit word, and
// the exit that makes the count (top 16 bits) a multiple of G checks the
// totals (the low 48 bits against the plan's exit_sum, word 0 against its
// take count), raises the count flag if they are off, and clears word 0 and
// the exit word.
// ---------------------------------------------------------------------------
struct Words {
  uint32_t take = 0, flags = 0;
  uint64_t exitw = 0;
};
constexpr uint32_t kStale = 1u, kCount = 2u;

struct Wg {
  int c, cn, ctaken;
  uint64_t my_sum;
  int state;  // 0: before the chunk's first unit, 1: chunk in progress, 2: exited
};

// Runs one launch of G workgroups over NC chunks with n_grabs tickets;
// returns how many times each chunk ran.
std::vector<int> run_queue(int G, int NC, uint32_t n_grabs, uint64_t exit_sum, Words& w, std::mt19937& rng) {
  const uint64_t mask = (uint64_t(1) << 48) - 1;
  std::vector<int> runs(size_t(NC), 0);
  std::vector<Wg> wg(static_cast<size_t>(G));
  auto do_exit = [&](Wg& s) {
    const uint64_t old = w.exitw;
    w.exitw += (uint64_t(1) << 48) + s.my_sum;
    if ((uint32_t(old >> 48) + 1u) % uint32_t(G) == 0u) {
      const uint64_t ran = (old + s.my_sum) & mask;
      if (ran != exit_sum || w.take != n_grabs) w.flags |= kCount;
      w.take = 0;
      w.exitw = 0;
    }
    s.state = 2;
  };
  for (int g = 0; g < G; ++g) {
    wg[size_t(g)] = Wg{g, g + G, NC, g < NC ? uint64_t(chunk_tag(uint32_t(g))) : 0u, 0};
    if (g >= NC) do_exit(wg[size_t(g)]);
  }
  for (;;) {
    std::vector<int> live;
    for (int g = 0; g < G; ++g)
      if (wg[size_t(g)].state != 2) live.push_back(g);
    if (live.empty()) break;
    Wg& s = wg[size_t(live[rng() % live.size()])];
    if (s.state == 0) {
      CHECK(s.c >= 0 && s.c < NC, "queue: chunk index %d of %d", s.c, NC);
      ++runs[size_t(s.c)];
      if (s.cn < NC) {
        const uint32_t t = w.take++;
        const bool ok = t < n_grabs;
        s.ctaken = ok ? 2 * G + int(t) : NC;
        if (!ok) w.flags |= kStale;
      }
      s.state = 1;
    } else {
      if (s.cn < NC) {
        s.my_sum += chunk_tag(uint32_t(s.cn));
        s.c = s.cn;
        s.cn = s.ctaken;
        s.ctaken = NC;
        s.state = 0;
      } else {
        do_exit(s);
      }
    }
  }
  return runs;
}

void check_queue(int G, int NC, std::mt19937& rng) {
  const uint32_t n_grabs = uint32_t(std::max(0, NC - 2 * G) + std::min(G, std::max(0, NC - G)));
  const uint64_t exit_sum = tag_sum(NC);
  Words w;
  for (int launch = 0; launch < 3; ++launch) {
    const std::vector<int> runs = run_queue(G, NC, n_grabs, exit_sum, w, rng);
    for (int c = 0; c < NC; ++c) CHECK(runs[size_t(c)] == 1, "queue G=%d NC=%d: chunk %d ran %d times", G, NC, c,
                                       runs[size_t(c)]);
    CHECK(w.flags == 0 && w.take == 0 && w.exitw == 0, "queue G=%d NC=%d: words after a clean launch", G, NC);
  }
  // left-over words (an interrupted launch, a workspace never cleared):
  // every chunk index stays in range (checked inside), and a launch whose
  // chunks did not each run once raises a flag
  const Words starts[] = {{5, 0, 0}, {0x80000000u, 0, 0}, {0xffffffffu, 0, 0}, {0, 0, uint64_t(3) << 48},
                          {0, 0, 7}, {n_grabs + 1, 0, 0}, {1, 0, (uint64_t(1) << 48) | 1}, {1, 0, 5}};
  std::vector<Words> all(std::begin(starts), std::end(starts));
  std::uniform_int_distribution<uint32_t> any;
  for (int i = 0; i < 16; ++i) {
    // words never zero-filled, and small left-overs of an interrupted launch
    all.push_back(Words{any(rng), 0, (uint64_t(any(rng)) << 32) | any(rng)});
    const uint32_t t = any(rng) % (n_grabs + 2), e = any(rng) % uint32_t(G), r = any(rng) % uint32_t(16 * NC + 1);
    if (t | e | r) all.push_back(Words{t, 0, (uint64_t(e) << 48) | r});
  }
  for (const Words& s0 : all) {
    Words ws = s0;
    for (int launch = 0; launch < 2; ++launch) {
      const uint32_t flags_before = ws.flags;
      const std::vector<int> runs = run_queue(G, NC, n_grabs, exit_sum, ws, rng);
      const bool once = std::all_of(runs.begin(), runs.end(), [](int r) { return r == 1; });
      CHECK(once || ws.flags != flags_before || flags_before != 0,
            "queue G=%d NC=%d: left-over words (%u, %llx): a chunk ran other than once, no flag", G, NC, s0.take,
            (unsigned long long)s0.exitw);
    }
  }
}

// ---------------------------------------------------------------------------
// One matrix on its own.
// ---------------------------------------------------------------------------
void check_one(const Mat& m, int batch, int max_wg, int rp) {
  Layout L;
  const qtea_desc d = make_desc(m, &L);
  OneShape o;
  CHECK(one_shape_for(d, batch, max_wg, rp, &o), "one_shape_for");
  const int64_t U = o.n_units, G = o.grid;
  CHECK(G >= 1 && G <= max_wg && G <= U, "one: grid %lld for %lld units", (long long)G, (long long)U);
  CHECK(U == int64_t(o.n_panels) * o.n_slices && o.n_panels == cdiv(d.n_pad, rp), "one: units");
  const int64_t per = cdiv(U, max_wg);
  for (int64_t g = 0; g < G; ++g) {
    const int64_t a = one_first(g, U, G), b = one_first(g + 1, U, G);
    CHECK(b > a && b - a <= per, "one: run %lld is [%lld, %lld)", (long long)g, (long long)a, (long long)b);
    CHECK(one_owner(a, U, G) == g && one_owner(b - 1, U, G) == g, "one_owner at the ends of run %lld", (long long)g);
  }
  CHECK(one_first(0, U, G) == 0 && one_first(G, U, G) == U, "one: runs cover the units");
  // parts of split panels: slot 2g for the part at run g's first unit, 2g + 1
  // for a part that starts later in the run
  std::vector<char> used(size_t(2 * G), 0);
  for (int64_t p = 0; p < o.n_panels; ++p) {
    const int64_t p0 = p * o.n_slices, p1 = p0 + o.n_slices;
    const int ga = one_owner(p0, U, G), gb = one_owner(p1 - 1, U, G);
    if (ga == gb) continue;
    for (int g = ga; g <= gb; ++g) {
      const int64_t slot = 2 * int64_t(g) + (g == ga && p0 > one_first(g, U, G) ? 1 : 0);
      CHECK(!used[size_t(slot)], "one: slot %lld twice", (long long)slot);
      used[size_t(slot)] = 1;
      CHECK((slot + 1) * rp * batch * 4 <= o.ws_bytes - o.off_part, "one: slot past the workspace");
    }
  }
  CHECK(o.off_part >= 4 * int64_t(o.n_panels) && o.off_part % kAlign == 0, "one: counters overlap the parts");
}

std::vector<Mat> stack(const int64_t (*shapes)[2], int n_shapes, int layers, double frac, int layout) {
  std::vector<Mat> v;
  for (int l = 0; l < layers; ++l)
    for (int i = 0; i < n_shapes; ++i) {
      const int64_t K = shapes[i][1];
      v.push_back(Mat{shapes[i][0], K, int64_t(frac * double(K) + 0.5), layout});
    }
  return v;
}

}  // namespace

int main() {
  setvbuf(stdout, nullptr, _IOLBF, 0);
  const int64_t s8b[4][2] = {{6144, 4096}, {4096, 4096}, {28672, 4096}, {4096, 14336}};
  const int64_t s14b[4][2] = {{7168, 5120}, {5120, 5120}, {34816, 5120}, {5120, 17408}};
  const int64_t s70b[4][2] = {{10240, 8192}, {8192, 8192}, {57344, 8192}, {8192, 28672}};
  std::vector<Mat> edge = {{4, 1, 0, kLayout},        {4, 1, 1, kLayout},         {64, 5, 5, kLayoutE4M3},
                           {100, 37, 3, kLayout},     {12, 300, 15, kLayoutG128}, {4, 1, 1, kLayoutG128},
                           {65536, 5, 0, kLayout},    {8, 65536, 100, kLayoutE4M3}, {1000, 321, 321, kLayout},
                           {68, 1279, 64, kLayoutG128}};

  // layouts
  for (const Mat& m : edge) check_layout(m);
  for (int layout : {kLayout, kLayoutE4M3, kLayoutG128})
    for (const auto* sh : {s8b, s14b, s70b})
      for (int i = 0; i < 4; ++i) check_layout(Mat{sh[i][0], sh[i][1], sh[i][1] / 20, layout});
  printf("ok layout regions (%d checks)\n", g_checks);

  // plans: the stacks at the launch shapes of the library (two workgroups
  // per CU at batch 1, one at 2..16) and odd grids
  struct Case {
    const char* name;
    std::vector<Mat> mats;
  };
  std::vector<Case> cases = {
      {"8b stack", stack(s8b, 4, 32, 0.02, kLayout)},
      {"14b stack", stack(s14b, 4, 40, 0.03, kLayout)},
      {"70b stack", stack(s70b, 4, 80, 0.02, kLayout)},
      {"8b e4m3", stack(s8b, 4, 32, 0.05, kLayoutE4M3)},
      {"8b g128", stack(s8b, 4, 32, 0.05, kLayoutG128)},
      {"8b layer", stack(s8b, 4, 1, 0.02, kLayout)},
      {"one 4096", {{4096, 4096, 82, kLayout}}},
      {"tiny", {{4, 1, 0, kLayout}}},
      {"edge mix", {{4, 1, 1, kLayout}, {100, 37, 3, kLayout}, {1000, 321, 321, kLayout}, {64, 5, 5, kLayout}}},
  };
  std::vector<Mat> many;
  for (int i = 0; i < 300; ++i) many.push_back(Mat{4 + 4 * (i % 40), 1 + 37 * (i % 23), std::min<int64_t>(i % 7, 1 + 37 * (i % 23)), kLayoutE4M3});
  cases.push_back({"300 small", many});
  for (const Case& c : cases) {
    const bool g128 = c.mats[0].layout == kLayoutG128;
    for (int G : {512, 1, 2, 3, 7, 64, 1024}) {
      check_plan(c.mats, 1, G, c.name);
      if (!g128) {
        check_plan(c.mats, 4, G / 2 > 0 ? G / 2 : 1, c.name);
        check_plan(c.mats, 16, G, c.name);
      }
    }
  }
  printf("ok plan records (%d checks)\n", g_checks);

  // argument checks of the planner
  {
    PlanOut po;
    std::vector<Mat> mixed = {{64, 64, 2, kLayout}, {64, 64, 2, kLayoutE4M3}};
    CHECK(plan(mixed, 1, 8, 1024, &po) == QTEA_ERR_INVALID_ARG, "two residual formats in one plan");
    std::vector<Mat> one = {{64, 64, 2, kLayout}};
    CHECK(plan(one, 0, 8, 1024, &po) == QTEA_ERR_BATCH && plan(one, 17, 8, 1024, &po) == QTEA_ERR_BATCH, "batch");
    std::vector<Mat> g = {{64, 300, 2, kLayoutG128}};
    CHECK(plan(g, 2, 8, 1024, &po) == QTEA_ERR_BATCH, "the grouped format above batch 1");
    Layout L;
    qtea_desc d = make_desc(one[0], &L);
    const void* pk = reinterpret_cast<const void*>(base_of(0, 0));
    const uint16_t* xp = reinterpret_cast<const uint16_t*>(base_of(1, 0));
    float* yp = reinterpret_cast<float*>(base_of(2, 0));
    std::vector<uint8_t> buf(size_t(plan_bytes_for(1, 8)));
    qtea_grouped_info info;
    CHECK(plan_write(&d, &pk, &xp, &yp, 1, 1, 8, 1024, buf.data(), int64_t(buf.size()) - 1, &info) ==
              QTEA_ERR_WORKSPACE,
          "short plan buffer");
    const uint16_t* xnull = nullptr;
    CHECK(plan_write(&d, &pk, &xnull, &yp, 1, 1, 8, 1024, buf.data(), int64_t(buf.size()), &info) ==
              QTEA_ERR_INVALID_ARG,
          "null activations");
    d.off_rval += 256;
    CHECK(plan_write(&d, &pk, &xp, &yp, 1, 1, 8, 1024, buf.data(), int64_t(buf.size()), &info) ==
              QTEA_ERR_INVALID_ARG,
          "a descriptor that does not match its layout");
  }
  printf("ok planner argument checks (%d checks)\n", g_checks);

  // the chunk queue under random interleavings, from clean and left-over words
  std::mt19937 rng(12345);
  for (int G : {1, 2, 3, 8, 64, 512})
    for (int NC : {1, 2, 3, 5, 8, 16, 17, 100, 1000, 8192}) {
      if (NC > 16 * G) continue;
      check_queue(G, NC, rng);
    }
  // the plans' own counts against the model
  for (const Case& c : cases) {
    if (c.mats.size() > 200) continue;
    PlanOut po;
    CHECK(plan(c.mats, 1, 512, 1024, &po) == QTEA_OK, "plan");
    GPlanHeader H;
    memcpy(&H, po.buf.data(), sizeof(H));
    Words w;
    const std::vector<int> runs = run_queue(512, H.n_chunks, uint32_t(H.n_grabs), H.exit_sum, w, rng);
    for (int r : runs) CHECK(r == 1, "%s: a chunk ran %d times", c.name, r);
    CHECK(w.flags == 0 && w.take == 0 && w.exitw == 0, "%s: the plan's n_grabs", c.name);
  }
  printf("ok chunk queue model (%d checks)\n", g_checks);

  // one matrix on its own at the library's shapes (512-row panels over up
  // to 512 workgroups at batch 1, over up to 256 at 2..16)
  for (const auto* sh : {s8b, s14b, s70b})
    for (int i = 0; i < 4; ++i)
      for (int layout : {kLayout, kLayoutE4M3, kLayoutG128}) {
        const Mat m{sh[i][0], sh[i][1], sh[i][1] / 20, layout};
        check_one(m, 1, 512, 512);
        for (int b : {2, 4, 8, 9, 16}) check_one(m, b, 256, kOneMmaRows);
        for (int wgs : {1, 3, 7, 100}) check_one(m, 1, wgs, 512);
      }
  for (const Mat& m : edge) {
    check_one(m, 1, 512, 512);
    check_one(m, 16, 256, kOneMmaRows);
  }
  printf("ok one-matrix runs (%d checks)\n", g_checks);
  return 0;
}
