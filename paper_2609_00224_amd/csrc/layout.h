// Layout constants and the layout arithmetic of a packed matrix (layout
// versions 2, 3 and 4): plain C++, no device code, so that host-only
// programs (the planner checks, built with the host sanitizers) compile it
// as the library does.  Internal to the library.
#ifndef QTEA_LAYOUT_H_
#define QTEA_LAYOUT_H_

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
// On the device a group takes two 16-pack groups ("slots"), each holding 13
// of its packs (65 of its columns: packs 0..12, then 13..25) densely: a
// slot's rows are 13 bytes apart, so a row and group take the paper's 26
// bytes.  A slot still spans 80 device columns (16 x 5), the last 15 zero.
constexpr int kLayoutG128 = 4;
constexpr int kScaleCols = 128;  // columns per quantization group
constexpr int kScalePacks = 26;  // packs per quantization group (25 of five columns, one of three)
constexpr int kG128SlotPacks = 13;  // packs per 16-pack slot in layout 4
constexpr int kG128SlotCols = 65;   // their columns
// Layout 4: the device column of real column j (group j / 128, slot of its
// column c = j mod 128: c / 65, column within the slot c mod 65).
constexpr int64_t g128_dcol(int64_t j) {
  return 2 * kGroupCols * (j / kScaleCols) + kGroupCols * ((j % kScaleCols) / kG128SlotCols) +
         (j % kScaleCols) % kG128SlotCols;
}
// Layout 4: the first real column of 16-pack slot dg.
constexpr int64_t g128_slot_col0(int64_t dg) { return kScaleCols * (dg >> 1) + kG128SlotCols * (dg & 1); }
constexpr int64_t kAlign = 256;
constexpr int64_t kHeaderBytes = 256;
constexpr int kFlagOffset = 128;

inline int64_t align_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }
inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

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

// Layout 4 differs in three regions: trits hold two 16-pack slots of 13
// bytes per row and 128-column group ([n_pad/64][n_groups][64][13]);
// "alpha" holds u32 (alpha | beta << 16) per row and group as
// [n_pad/64][n_groups/2][64]; v is in device column order (80 per 16-pack
// slot, zero in the unused columns).  n_packs is the paper's count (26 per
// group).
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
  o = align_up(o + L->n_pad * L->n_groups * (g128 ? kG128SlotPacks : kGroupPacks), kAlign);
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

// The descriptor of a packed matrix with layout L (what the pack entry
// points return and desc_ok accepts).
inline qtea_desc desc_from_layout(const Layout& L, int64_t N, int64_t K, int64_t nS, int layout) {
  qtea_desc d;
  d.magic = QTEA_DESC_MAGIC;
  d.layout = uint32_t(layout);
  d.N = N;
  d.K = K;
  d.n_salient = nS;
  d.n_packs = L.n_packs;
  d.n_groups = L.n_groups;
  d.n_pad = L.n_pad;
  d.bytes_total = L.total;
  d.off_trits = L.off_trits;
  d.off_alpha = L.off_alpha;
  d.off_v = L.off_v;
  d.off_salient = L.off_salient;
  d.off_spos = L.off_spos;
  d.off_rval = L.off_rval;
  d.off_ridx = L.off_ridx;
  return d;
}

}  // namespace qtea_detail

#endif  // QTEA_LAYOUT_H_
