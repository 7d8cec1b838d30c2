// Compressed ternary GEMV for gfx950: packing, the lookup-table GEMV and
// the C ABI declared in include/qtea.h.
//
// Device layout (layout versions 2 and 3), all regions 256-byte aligned:
//   header   256 B: magic, layout, sizes; a validation flag word at +128.
//   trits    [n_pad/64 tiles][n_groups][64 rows][16 bytes]
//            One 16-byte unit holds the sixteen packs of one 16-pack group
//            for one row; a wavefront (64 lanes = 64 rows of a tile) reads
//            1 KiB contiguous per 128-bit load.  Byte i of the unit of row r
//            holds pack 16*g + ((i + r) mod 16): rows are rotated so that at
//            step i the 16 lanes of a quarter-wave address 16 different
//            packs' table columns (distinct LDS banks).
//   alpha    fp16 [n_pad]              (zero in the row padding)
//   v        fp16 [n_groups * 80]      (zero in the column padding)
//   salient  int32 [n_salient]
//   spos     int32 [n_groups + 1]      first s with S_s >= 80 * g
//   rval     [n_pad/64][n_salient][16] fp16 (layout 2) or FP8 E4M3 bytes
//            (layout 3): residual of four-row group g in salient
//            column s at ((g / 16) * n_salient + s) * 16 + g % 16: the sixteen
//            groups of a tile are contiguous per column, and a tile's residual
//            over a run of salient columns is one contiguous run
//   ridx     u32  [n_pad/64][n_salient] 2-bit positions of 16 consecutive groups
//
// GEMV (one launch): workgroup = (row block, K slice).  For each chunk of
// 16-pack groups of its slice it computes a_j = v_j x_j, builds the 243-entry
// table of every pack of the chunk in LDS, then each lane (one output row)
// streams its row's packed bytes and adds one table entry per byte.  The
// salient residual of the slice's columns is added in the same pass.  The
// slice partials go to the workspace; the last workgroup of a row block to
// arrive sums them in slice order (deterministic) and writes y.
#include "qtea_internal.h"

namespace {

using namespace qtea_detail;


// ---------------------------------------------------------------------------
// Packing kernels (offline).
// ---------------------------------------------------------------------------
__global__ void validate_kernel(const int8_t* __restrict__ trits, int64_t nt,
                                const uint8_t* __restrict__ ridx, int64_t ni,
                                const int32_t* __restrict__ S, int64_t nS, int64_t K,
                                uint32_t* __restrict__ flags) {
  uint32_t f = 0;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < nt; i += stride) {
    const int8_t t = trits[i];
    if (t < -1 || t > 1) f |= kFlagBadTrit;
  }
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < ni; i += stride)
    if (ridx[i] > 3) f |= kFlagBadResid;
  for (int64_t s = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; s < nS; s += stride) {
    const int32_t c = S[s];
    if (c < 0 || c >= K || (s > 0 && c <= S[s - 1])) f |= kFlagBadResid;
  }
  if (f) atomicOr(flags, f);
}

// One thread per 16-byte unit (tile, group, row-in-tile).
__global__ void pack_trits_kernel(const int8_t* __restrict__ trits, int64_t N, int64_t K,
                                  int64_t n_groups, int64_t n_units, uint8_t* __restrict__ out) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; u < n_units; u += stride) {
    const int64_t l = u % kTileRows;
    const int64_t g = (u / kTileRows) % n_groups;
    const int64_t tile = u / (kTileRows * n_groups);
    const int64_t r = tile * kTileRows + l;
    uint32_t w[4] = {kZeroCode4, kZeroCode4, kZeroCode4, kZeroCode4};
    if (r < N) {
      const int8_t* row = trits + r * K;
      for (int i = 0; i < kGroupPacks; ++i) {
        const int64_t p = g * kGroupPacks + ((i + l) & (kGroupPacks - 1));
        uint32_t code = 0, pw = 1;
        for (int e = 0; e < 5; ++e) {
          const int64_t j = 5 * p + e;
          int t = j < K ? row[j] : 0;
          t = t < -1 ? -1 : (t > 1 ? 1 : t);  // invalid input is reported by validate_kernel
          code += uint32_t(t + 1) * pw;
          pw *= 3;
        }
        const int sh = 8 * (i & 3);
        w[i >> 2] = (w[i >> 2] & ~(0xffu << sh)) | (code << sh);
      }
    }
    const u32x4 v = {w[0], w[1], w[2], w[3]};
    *reinterpret_cast<u32x4*>(out + u * 16) = v;
  }
}

// Scales, salient list and residual blocks.  VT is the residual value type:
// uint16_t (fp16 bits, layout 2) or uint8_t (E4M3 bytes, layout 3; a NaN code
// is flagged).  With S == o_S the salient list is already in place (derived
// from a bitmap) and only read.
template <typename VT>
__global__ void pack_meta_kernel(const uint16_t* __restrict__ alpha, const uint16_t* __restrict__ v,
                                 const int32_t* S, const VT* __restrict__ rval,
                                 const uint8_t* __restrict__ ridx, int64_t N, int64_t K, int64_t nS,
                                 int64_t n_pad, int64_t n_groups, uint16_t* __restrict__ o_alpha,
                                 uint16_t* __restrict__ o_v, int32_t* o_S,
                                 int32_t* __restrict__ o_spos, VT* __restrict__ o_rval,
                                 uint32_t* __restrict__ o_ridx, uint32_t* __restrict__ flags, int g128) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  const int64_t t0 = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (o_alpha)  // layout 4: scales and v by pack_scales128_kernel
    for (int64_t i = t0; i < n_pad; i += stride) o_alpha[i] = i < N ? alpha[i] : 0;
  if (o_v)
    for (int64_t i = t0; i < n_groups * kGroupCols; i += stride) o_v[i] = i < K ? v[i] : 0;
  if (S != o_S)
    for (int64_t i = t0; i < nS; i += stride) o_S[i] = S[i];
  for (int64_t g = t0; g <= n_groups; g += stride) {
    // lower bound of the first column of 16-pack group g in the sorted
    // salient list (layout 4: group g holds columns from 128 (g / 2) + 80 (g % 2))
    int64_t lo = 0, hi = nS;
    const int64_t key = g128 ? kScaleCols * (g >> 1) + kGroupCols * (g & 1) : g * kGroupCols;
    while (lo < hi) {
      const int64_t mid = (lo + hi) / 2;
      if (S[mid] < key)
        lo = mid + 1;
      else
        hi = mid;
    }
    o_spos[g] = int32_t(lo);
  }
  const int64_t G = N / 4, Gp = n_pad / 4, Wp = n_pad / 64;
  uint32_t f = 0;
  for (int64_t i = t0; i < nS * Gp; i += stride) {
    const int64_t tile = i / (16 * nS), rem = i - tile * 16 * nS;
    const int64_t s = rem >> 4, g = 16 * tile + (rem & 15);
    const VT val = g < G ? rval[s * G + g] : VT(0);
    if (sizeof(VT) == 1 && e4m3_is_nan(val)) f |= kFlagBadResid;
    o_rval[i] = val;
  }
  if (f) atomicOr(flags, f);
  for (int64_t i = t0; i < nS * Wp; i += stride) {
    const int64_t w = i / nS, s = i % nS;
    uint32_t word = 0;
    for (int k = 0; k < 16; ++k) {
      const int64_t g = 16 * w + k;
      if (g < G) word |= uint32_t(ridx[s * G + g] & 3) << (2 * k);
    }
    o_ridx[i] = word;
  }
}

// Salient column list from a column bitmap (bit j % 32 of word j / 32 set
// when column j is salient), ascending, by one workgroup: each thread counts
// a contiguous run of words, a scan over the threads gives every run's first
// list position.  A bit at or past K, or a count other than nS, is flagged
// (and nothing is written).
__global__ __launch_bounds__(1024) void bitmap_salient_kernel(const uint32_t* __restrict__ bitmap,
                                                              int64_t K, int64_t nS,
                                                              int32_t* __restrict__ o_S,
                                                              uint32_t* __restrict__ flags) {
  __shared__ int64_t run[1024];
  const int t = threadIdx.x;
  const int64_t nw = (K + 31) / 32, per = (nw + 1023) / 1024;
  const int64_t w0 = min(nw, int64_t(t) * per), w1 = min(nw, w0 + per);
  const uint32_t tail = (K & 31) ? (1u << (K & 31)) - 1u : 0xffffffffu;
  uint32_t f = 0;
  int64_t cnt = 0;
  for (int64_t w = w0; w < w1; ++w) {
    uint32_t b = bitmap[w];
    if (w == nw - 1) {
      if (b & ~tail) f |= kFlagBadResid;
      b &= tail;
    }
    cnt += __popc(b);
  }
  run[t] = cnt;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {  // inclusive scan
    const int64_t add = t >= off ? run[t - off] : 0;
    __syncthreads();
    run[t] += add;
    __syncthreads();
  }
  if (run[1023] != nS) {
    f |= kFlagBadResid;
  } else {
    int64_t pos = run[t] - cnt;
    for (int64_t w = w0; w < w1; ++w) {
      uint32_t b = bitmap[w] & (w == nw - 1 ? tail : 0xffffffffu);
      while (b) {
        o_S[pos++] = int32_t(32 * w + (__ffs(b) - 1));
        b &= b - 1u;
      }
    }
  }
  if (f) atomicOr(flags, f);
}

__global__ void write_header_kernel(uint8_t* packed, int64_t N, int64_t K, int64_t nS, int layout) {
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    uint32_t* h = reinterpret_cast<uint32_t*>(packed);
    h[0] = QTEA_DESC_MAGIC;
    h[1] = uint32_t(layout);
    int64_t* h64 = reinterpret_cast<int64_t*>(packed + 8);
    h64[0] = N;
    h64[1] = K;
    h64[2] = nS;
    reinterpret_cast<uint32_t*>(packed + kFlagOffset)[0] = 0;
  }
}

// Layout 4 trits: one thread per 16-byte unit (tile, 16-pack group dg, row).
// Byte i of row l's unit holds pack slot 16 (dg % 2) + ((i + l) mod 16) of
// quantization group dg / 2: slot p < 26 codes the group's columns
// 5p..5p+4 (zero trits past its column 127 and past K), slots 26..31 the
// all-zero code.
__global__ void pack_trits128_kernel(const int8_t* __restrict__ trits, int64_t N, int64_t K,
                                     int64_t n_groups, int64_t n_units, uint8_t* __restrict__ out) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; u < n_units; u += stride) {
    const int64_t l = u % kTileRows;
    const int64_t dg = (u / kTileRows) % n_groups;
    const int64_t tile = u / (kTileRows * n_groups);
    const int64_t r = tile * kTileRows + l, g = dg >> 1;
    uint32_t w[4] = {kZeroCode4, kZeroCode4, kZeroCode4, kZeroCode4};
    if (r < N) {
      const int8_t* row = trits + r * K;
      for (int i = 0; i < kGroupPacks; ++i) {
        const int64_t p = kGroupPacks * (dg & 1) + ((i + l) & (kGroupPacks - 1));
        if (p >= kScalePacks) continue;  // the all-zero code stays
        uint32_t code = 0, pw = 1;
        for (int e = 0; e < 5; ++e) {
          const int64_t c = 5 * p + e, j = kScaleCols * g + c;
          int t = (c < kScaleCols && j < K) ? row[j] : 0;
          t = t < -1 ? -1 : (t > 1 ? 1 : t);  // invalid input is reported by validate_kernel
          code += uint32_t(t + 1) * pw;
          pw *= 3;
        }
        const int sh = 8 * (i & 3);
        w[i >> 2] = (w[i >> 2] & ~(0xffu << sh)) | (code << sh);
      }
    }
    const u32x4 v = {w[0], w[1], w[2], w[3]};
    *reinterpret_cast<u32x4*>(out + u * 16) = v;
  }
}

// Layout 4 scales and rescales: (alpha | beta << 16) per row and group as
// [n_pad/64][n_sg][64] (zero in padded rows), v in device column order
// (column c of 16-pack group dg is slot 16 (dg % 2) + c / 5, column c % 5 of
// that slot; zero in the padding).
__global__ void pack_scales128_kernel(const uint16_t* __restrict__ alpha, const uint16_t* __restrict__ beta,
                                      const uint16_t* __restrict__ v, int64_t N, int64_t K, int64_t n_pad,
                                      int64_t n_sg, uint32_t* __restrict__ o_ab, uint16_t* __restrict__ o_v) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  const int64_t t0 = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  for (int64_t i = t0; i < n_pad * n_sg; i += stride) {
    const int64_t tile = i / (n_sg * kTileRows), rem = i - tile * n_sg * kTileRows;
    const int64_t g = rem / kTileRows, r = tile * kTileRows + rem % kTileRows;
    o_ab[i] = r < N ? uint32_t(alpha[r * n_sg + g]) | (uint32_t(beta[r * n_sg + g]) << 16) : 0u;
  }
  for (int64_t i = t0; i < 2 * n_sg * kGroupCols; i += stride) {
    const int64_t dg = i / kGroupCols, col = i % kGroupCols;
    const int64_t p = kGroupPacks * (dg & 1) + col / 5, c = 5 * p + col % 5;
    const int64_t j = kScaleCols * (dg >> 1) + c;
    o_v[i] = (p < kScalePacks && c < kScaleCols && j < K) ? v[j] : uint16_t(0);
  }
}

// The vs region (u32 per device column): pass 1 copies the v bits, pass 2
// marks every salient column with 1 + its rank among the salient columns of
// its 320-column slice (device columns; layout 4 maps column j to device
// column 160 (j / 128) + j % 128).
__global__ void pack_vs_kernel(const uint16_t* __restrict__ o_v, int64_t n_cols, uint32_t* __restrict__ o_vs) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n_cols; i += stride) o_vs[i] = o_v[i];
}
// A salient list that failed validation (reported by the pack's flags) may
// hold any value: every index is checked before it is used.
__global__ void mark_salient_kernel(const int32_t* __restrict__ S, const int32_t* __restrict__ spos, int64_t nS,
                                    int64_t K, int64_t n_groups, int g128, uint32_t* __restrict__ o_vs) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t s = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; s < nS; s += stride) {
    const int64_t j = S[s];
    if (j < 0 || j >= K) continue;
    const int64_t dc = g128 ? 160 * (j / kScaleCols) + j % kScaleCols : j;
    const int64_t g0 = 4 * (dc / (4 * kGroupCols));
    if (dc >= n_groups * kGroupCols || g0 > n_groups) continue;
    const int64_t rank = s - spos[g0];
    if (rank < 0 || rank >= 4 * kGroupCols) continue;
    o_vs[dc] |= uint32_t(rank + 1) << 16;
  }
}

// Streaming-read ceiling: each workgroup of 256 streams one contiguous 64 KiB
// chunk with 16-byte non-temporal loads, eight in flight per thread (under
// sustained load this holds about 7 TB/s, grid-stride loads about 6.5), and
// stores the fold of its chunk to its own word of sink: one atomic per
// workgroup on a shared word instead would cost more than a third of the rate.
constexpr int kCeilUnroll = 8;
constexpr int kCeilThreads = 256;
constexpr int64_t kCeilChunk16 = int64_t(QTEA_READ_CEILING_CHUNK) / 16;
// (The chunk length is a kernel argument: the loop's code is then the one
// measured at the rate above.)
__global__ __launch_bounds__(kCeilThreads) void read_ceiling_kernel(const u32x4* __restrict__ buf, int64_t n16,
                                                                    int64_t chunk16, uint32_t* __restrict__ sink) {
  const int64_t b0 = int64_t(blockIdx.x) * chunk16;
  const int64_t b1 = b0 + chunk16 < n16 ? b0 + chunk16 : n16;
  uint32_t f = 0;
  int64_t i = b0 + threadIdx.x;
  for (; i + (kCeilUnroll - 1) * kCeilThreads < b1; i += kCeilUnroll * kCeilThreads) {
    u32x4 v[kCeilUnroll];
#pragma unroll
    for (int k = 0; k < kCeilUnroll; ++k) v[k] = __builtin_nontemporal_load(buf + i + k * kCeilThreads);
#pragma unroll
    for (int k = 0; k < kCeilUnroll; ++k) f ^= v[k].x + v[k].y + v[k].z + v[k].w;
  }
  for (; i < b1; i += kCeilThreads) {
    const u32x4 a = __builtin_nontemporal_load(buf + i);
    f ^= a.x + a.y + a.z + a.w;
  }
  for (int o = 32; o > 0; o >>= 1) f ^= __shfl_xor(f, o);
  __shared__ uint32_t red[kCeilThreads / 64];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = f;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
    for (int k = 0; k < kCeilThreads / 64; ++k) t ^= red[k];
    sink[blockIdx.x] = t;
  }
}

// ---------------------------------------------------------------------------
// Debug unpack (bit-exact read-back of the layout).
// ---------------------------------------------------------------------------
__global__ void unpack_codes_kernel(const uint8_t* __restrict__ tr, int64_t N, int64_t K,
                                    int64_t n_packs, int64_t n_groups, uint8_t* __restrict__ canon,
                                    int8_t* __restrict__ trits) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < N * n_packs; e += stride) {
    const int64_t r = e / n_packs, p = e % n_packs;
    const int64_t tile = r / kTileRows, l = r % kTileRows;
    const int64_t g = p / kGroupPacks, q = p % kGroupPacks;
    const int64_t i = (q - l) & (kGroupPacks - 1);
    const uint8_t c = tr[((tile * n_groups + g) * kTileRows + l) * 16 + i];
    if (canon) canon[e] = c;
    if (trits) {
      uint32_t rest = c;
      for (int d = 0; d < 5; ++d) {
        const int64_t j = 5 * p + d;
        if (j < K) trits[r * K + j] = int8_t(int(rest % 3) - 1);
        rest /= 3;
      }
    }
  }
}

// Layout 4: the paper's codes [N][26 n_sg] (26 per row and group) and trits.
__global__ void unpack_codes128_kernel(const uint8_t* __restrict__ tr, int64_t N, int64_t K,
                                       int64_t n_packs, int64_t n_groups, uint8_t* __restrict__ canon,
                                       int8_t* __restrict__ trits) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < N * n_packs; e += stride) {
    const int64_t r = e / n_packs, pp = e % n_packs;
    const int64_t g = pp / kScalePacks, p = pp % kScalePacks;
    const int64_t tile = r / kTileRows, l = r % kTileRows, dg = 2 * g + p / kGroupPacks;
    const int64_t i = ((p % kGroupPacks) - l) & (kGroupPacks - 1);
    const uint8_t c = tr[((tile * n_groups + dg) * kTileRows + l) * 16 + i];
    if (canon) canon[e] = c;
    if (trits) {
      uint32_t rest = c;
      for (int d = 0; d < 5; ++d) {
        const int64_t col = 5 * p + d, j = kScaleCols * g + col;
        if (col < kScaleCols && j < K) trits[r * K + j] = int8_t(int(rest % 3) - 1);
        rest /= 3;
      }
    }
  }
}

__global__ void unpack_resid_kernel(const uint32_t* __restrict__ ridx, int64_t N, int64_t nS,
                                    int64_t n_pad, int32_t* __restrict__ rows) {
  const int64_t G = N / 4;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < nS * G; e += stride) {
    const int64_t s = e / G, g = e % G;
    const uint32_t w = ridx[(g / 16) * nS + s];
    rows[e] = int32_t(4 * g + ((w >> (2 * (g % 16))) & 3));
  }
}

__global__ void fill_zero_kernel(uint32_t* __restrict__ p, int64_t n_words, uint8_t* __restrict__ tail,
                                 int64_t n_tail) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  const int64_t t0 = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  for (int64_t i = t0; i < n_words; i += stride) p[i] = 0;
  for (int64_t i = t0; i < n_tail; i += stride) tail[i] = 0;
}

// ---------------------------------------------------------------------------
// The lookup-table GEMV.
// ---------------------------------------------------------------------------
struct GemvArgs {
  const uint8_t* trits;
  const uint16_t* alpha;
  const uint16_t* v;
  const int32_t* S;
  const int32_t* spos;
  const uint16_t* rval;  // fp16, or E4M3 bytes when f8
  const uint32_t* ridx;
  const uint16_t* x;
  float* y;
  float* part;
  uint32_t* counters;
  int64_t N, K, n_pad;
  int n_groups, n_tiles, nS;
  int f8;  // residual values are E4M3 bytes (layout 3)
  int nrb, nslices, ks_groups;
};

// Batch vectors per table pass (BT) and 16-pack groups per table chunk (KC).
// Table word of (code, group k, slot, bt) = ((code * KC + k) * 16 + slot) * BT + bt:
// one code row is KC * 16 * BT floats = 256 bytes whenever KC * BT == 4, so
// an address is code * 256 + low byte, formed by one v_perm_b32.
template <int B>
struct Cfg {
  static constexpr int BT = B < 4 ? B : 4;
  static constexpr int NPASS = (B + BT - 1) / BT;
  static constexpr int KC = BT == 1 ? 4 : (BT == 2 ? 2 : 1);
  static constexpr int COLS = KC * kGroupCols;  // activation columns per chunk
  static constexpr bool PERM = KC * BT == 4;    // 256-byte code rows
  static constexpr int ROW = KC * kGroupPacks * BT;  // floats per code row
  static constexpr int LUT_FLOATS = kCodes * ROW;
  // Table-build task = (pack, DEPTH leading digits); it writes the 3^(5-DEPTH)
  // codes sharing those digits from a compile-time digit tree.
  static constexpr int DEPTH = BT <= 2 ? 1 : 2;
  static constexpr int NPRE = DEPTH == 1 ? 3 : 9;
  static constexpr int SUB = kCodes / NPRE;
  static constexpr int X_PER_THREAD = (B * COLS + kThreads - 1) / kThreads;
  static constexpr int V_PER_THREAD = (COLS + kThreads - 1) / kThreads;
};

constexpr int kResBatch = 8;  // salient columns whose loads are issued together


// Leaves of the digit tree below `t`: digit DIG (and the ones below it)
// enumerated at compile time; the value of code offset OFF + d * 3^DIG is
// t + (d - 1) * a[DIG].  Leaves are stored at compile-time offsets from dst.
template <int DIG, int OFF, int BT, int STRIDE>
__device__ __forceinline__ void tree(float* dst, const float (&t)[BT], const float (&a)[5][BT]) {
  constexpr int P3 = DIG == 0 ? 1 : DIG == 1 ? 3 : DIG == 2 ? 9 : DIG == 3 ? 27 : 81;
#pragma unroll
  for (int d = 0; d < 3; ++d) {
    float u[BT];
#pragma unroll
    for (int bt = 0; bt < BT; ++bt) u[bt] = d == 0 ? t[bt] - a[DIG][bt] : (d == 2 ? t[bt] + a[DIG][bt] : t[bt]);
    if constexpr (DIG == 0) {
#pragma unroll
      for (int bt = 0; bt < BT; ++bt) dst[(OFF + d) * STRIDE + bt] = u[bt];
    } else {
      if (d == 0) tree<DIG - 1, OFF, BT, STRIDE>(dst, u, a);
      if (d == 1) tree<DIG - 1, OFF + P3, BT, STRIDE>(dst, u, a);
      if (d == 2) tree<DIG - 1, OFF + 2 * P3, BT, STRIDE>(dst, u, a);
    }
  }
}

template <int B, int TPW>
__global__ __launch_bounds__(kThreads) void lut_gemv_kernel(const GemvArgs p) {
  using C = Cfg<B>;
  constexpr int BT = C::BT, KC = C::KC, COLS = C::COLS;
  __shared__ float lut[C::LUT_FLOATS];
  __shared__ float x_lds[B * COLS];  // this chunk's activations, fp32
  __shared__ float v_lds[COLS];      // this chunk's column rescales, fp32
  __shared__ int s_last;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int quarter = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rb = blockIdx.x / p.nslices;
  const int ks = blockIdx.x % p.nslices;
  const int g0 = ks * p.ks_groups;
  const int g1 = min(p.n_groups, g0 + p.ks_groups);

  int tile[TPW];
  bool valid[TPW];
#pragma unroll
  for (int j = 0; j < TPW; ++j) {
    tile[j] = rb * (kWaves * TPW) + j * kWaves + wave;
    valid[j] = tile[j] < p.n_tiles;
  }
  float acc[TPW][B], racc[TPW][B];
#pragma unroll
  for (int j = 0; j < TPW; ++j)
#pragma unroll
    for (int b = 0; b < B; ++b) acc[j][b] = racc[j][b] = 0.0f;

  // Byte i of a lane's unit holds slot (i + lane) mod 16: table offsets of
  // the 16 slots, one per byte, for the v_perm address formation.
  uint32_t rotw[4];
#pragma unroll
  for (int q4 = 0; q4 < 4; ++q4) {
    uint32_t v4 = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) v4 |= uint32_t(((q4 * 4 + e + lane) & 15) * BT * 4) << (8 * e);
    rotw[q4] = v4;
  }

  for (int c0 = g0; c0 < g1; c0 += KC) {
    const int nk = min(KC, g1 - c0);
    const int64_t col0 = int64_t(c0) * kGroupCols;
    // (1) activations and rescales of the chunk (issued first: needed first)
    float xr[C::X_PER_THREAD], vr[C::V_PER_THREAD];
#pragma unroll
    for (int u = 0; u < C::X_PER_THREAD; ++u) {
      const int e = tid + u * kThreads;
      const int b = e / COLS, col = e % COLS;
      xr[u] = (e < B * COLS && col < nk * kGroupCols && col0 + col < p.K) ? h2f(p.x[b * p.K + col0 + col]) : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < C::V_PER_THREAD; ++u) {
      const int col = tid + u * kThreads;
      vr[u] = (col < nk * kGroupCols) ? h2f(p.v[col0 + col]) : 0.0f;  // v is zero-padded to whole groups
    }
    // (2) packed bytes of this chunk for this lane's rows.  Quarter q of the
    // wave takes the chunk's groups in the order q, q+1, ... so that at any
    // step the four quarters address four different groups' table columns.
    u32x4 w[TPW][KC];
    int grp[KC];
#pragma unroll
    for (int k = 0; k < KC; ++k) {
      int gk = k + quarter;
      gk = gk >= nk ? gk - nk : gk;
      gk = gk >= nk ? gk - nk : gk;
      gk = gk >= nk ? gk - nk : gk;
      grp[k] = gk;
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
        if (valid[j] && k < nk) {
          const u32x4* src = reinterpret_cast<const u32x4*>(
              p.trits + ((int64_t(tile[j]) * p.n_groups + c0 + gk) * kTileRows + lane) * 16);
          w[j][k] = __builtin_nontemporal_load(src);
        } else {
          w[j][k] = u32x4(kZeroCode4);
        }
      }
    }
    // (3) salient columns of the chunk (uniform scalar loads)
    const int sb = p.spos[c0], se = p.spos[c0 + nk];

    __syncthreads();  // previous chunk's readers of lut / x_lds are done
#pragma unroll
    for (int u = 0; u < C::X_PER_THREAD; ++u) {
      const int e = tid + u * kThreads;
      if (e < B * COLS) x_lds[e] = xr[u];
    }
#pragma unroll
    for (int u = 0; u < C::V_PER_THREAD; ++u) {
      const int col = tid + u * kThreads;
      if (col < COLS) v_lds[col] = vr[u];
    }
    // residual metadata of the first salient batch: lands during the build
    int r_col[kResBatch];
    uint32_t r_word[TPW][kResBatch];
    uint16_t r_val[TPW][kResBatch];
    auto load_res = [&](int s0) {
#pragma unroll
      for (int u = 0; u < kResBatch; ++u) {
        const int s = s0 + u;
        const bool ok = s < se;
        r_col[u] = ok ? p.S[s] - int(col0) : 0;
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
          const int64_t r = int64_t(tile[j]) * kTileRows + lane;
          r_word[j][u] = ok && valid[j] ? p.ridx[int64_t(tile[j]) * p.nS + s] : 0u;
          const int64_t vi = rval_index(r >> 2, s, p.nS);
          r_val[j][u] = !(ok && valid[j]) ? uint16_t(0)
                        : p.f8 ? e4m3_to_half_bits(reinterpret_cast<const uint8_t*>(p.rval)[vi]) : p.rval[vi];
        }
      }
    };
    if (sb < se) load_res(sb);
    __syncthreads();

#pragma unroll
    for (int pass = 0; pass < C::NPASS; ++pass) {
      if (pass > 0) __syncthreads();  // lookups of the previous pass are done
      // (4) table build: entry (group k, slot, code) = sum_i (d_i(code) - 1) * v_j x_j,
      // j = 5 * pack + i.  Consecutive threads take consecutive slots.
      for (int task = tid; task < nk * kGroupPacks * C::NPRE; task += kThreads) {
        const int pk = task % (nk * kGroupPacks);
        const int pf = task / (nk * kGroupPacks);
        const int k = pk >> 4, slot = pk & 15;
        const int cb = pk * 5;
        float a[5][BT];
#pragma unroll
        for (int i = 0; i < 5; ++i)
#pragma unroll
          for (int bt = 0; bt < BT; ++bt) {
            const int b = pass * BT + bt;
            a[i][bt] = b < B ? v_lds[cb + i] * x_lds[b * COLS + cb + i] : 0.0f;
          }
        float t[BT];
        float* dst = lut + ((pf * C::SUB * KC + k) * kGroupPacks + slot) * BT;
        if constexpr (C::DEPTH == 1) {
#pragma unroll
          for (int bt = 0; bt < BT; ++bt) t[bt] = pf == 0 ? -a[4][bt] : (pf == 2 ? a[4][bt] : 0.0f);
          tree<3, 0, BT, C::ROW>(dst, t, a);
        } else {
          const int d4 = pf / 3, d3 = pf - 3 * d4;
#pragma unroll
          for (int bt = 0; bt < BT; ++bt) {
            const float t4 = d4 == 0 ? -a[4][bt] : (d4 == 2 ? a[4][bt] : 0.0f);
            t[bt] = d3 == 0 ? t4 - a[3][bt] : (d3 == 2 ? t4 + a[3][bt] : t4);
          }
          tree<2, 0, BT, C::ROW>(dst, t, a);
        }
      }
      __syncthreads();
      // (5) lookup-accumulate: one table entry (BT floats) per packed byte.
#pragma unroll
      for (int k = 0; k < KC; ++k) {
        if (k >= nk) break;
        const uint32_t gbyte = uint32_t(grp[k] * kGroupPacks * BT * 4) * 0x01010101u;
        const uint32_t lowb[4] = {rotw[0] | gbyte, rotw[1] | gbyte, rotw[2] | gbyte, rotw[3] | gbyte};
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
          if (!valid[j]) continue;
          const uint32_t ww[4] = {w[j][k].x, w[j][k].y, w[j][k].z, w[j][k].w};
#pragma unroll
          for (int i = 0; i < kGroupPacks; ++i) {
            uint32_t addr;
            if constexpr (C::PERM) {
              // [byte0 = low byte, byte1 = code, bytes 2-3 = 0] = code * 256 + low
              const uint32_t sel = 0x0c0c0000u | (uint32_t(4 + (i & 3)) << 8) | uint32_t(i & 3);
              addr = __builtin_amdgcn_perm(ww[i >> 2], lowb[i >> 2], sel);
            } else {
              const uint32_t code = (ww[i >> 2] >> (8 * (i & 3))) & 0xffu;
              addr = code * uint32_t(C::ROW * 4) +
                     uint32_t((grp[k] * kGroupPacks + ((i + lane) & 15)) * BT * 4);
            }
            const float* e = reinterpret_cast<const float*>(reinterpret_cast<const char*>(lut) + addr);
#pragma unroll
            for (int bt = 0; bt < BT; ++bt)
              if (pass * BT + bt < B) acc[j][pass * BT + bt] += e[bt];
          }
        }
      }
    }

    // (6) salient residual of the chunk's columns (scaled by neither alpha nor v)
    for (int s0 = sb; s0 < se; s0 += kResBatch) {
      if (s0 != sb) load_res(s0);
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
        const int64_t r = int64_t(tile[j]) * kTileRows + lane;
        const uint32_t shift = 2 * ((r >> 2) & 15);
#pragma unroll
        for (int u = 0; u < kResBatch; ++u) {
          const bool hit = s0 + u < se && ((r_word[j][u] >> shift) & 3u) == uint32_t(r & 3);
          if (hit) {
            const float rv = h2f(r_val[j][u]);
#pragma unroll
            for (int b = 0; b < B; ++b) racc[j][b] += rv * x_lds[b * COLS + r_col[u]];
          }
        }
      }
    }
  }

  // Slice partial: alpha_r * (table sum) + residual.
#pragma unroll
  for (int j = 0; j < TPW; ++j) {
    if (!valid[j]) continue;
    const int64_t r = int64_t(tile[j]) * kTileRows + lane;
    const float al = h2f(p.alpha[r]);
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const float v = al * acc[j][b] + racc[j][b];
      if (p.nslices == 1) {
        if (r < p.N) p.y[b * p.N + r] = v;
      } else {
        store_coherent(p.part + (int64_t(ks) * B + b) * p.n_pad + r, v);
      }
    }
  }
  if (p.nslices == 1) return;

  // The last workgroup of this row block to arrive sums the slices in
  // order.  Partials are written and read with agent-scope (L2-coherent)
  // accesses; the wait below makes this workgroup's partials complete
  // before its arrival is counted.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (tid == 0) {
    const uint32_t prev = __hip_atomic_fetch_add(p.counters + rb, 1u, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
    s_last = prev == uint32_t(p.nslices - 1);
  }
  __syncthreads();
  if (!s_last) return;
  if (tid == 0)
    __hip_atomic_store(p.counters + rb, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
  for (int j = 0; j < TPW; ++j) {
    if (!valid[j]) continue;
    const int64_t r = int64_t(tile[j]) * kTileRows + lane;
    if (r >= p.N) continue;
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const float* src = p.part + int64_t(b) * p.n_pad + r;
      const int64_t qstride = int64_t(B) * p.n_pad;
      float sum = 0.0f;
      for (int q0 = 0; q0 < p.nslices; q0 += 8) {
        float t[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) t[u] = q0 + u < p.nslices ? load_coherent(src + (q0 + u) * qstride) : 0.0f;
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (q0 + u < p.nslices) sum += t[u];
      }
      p.y[b * p.N + r] = sum;
    }
  }
}

// ---------------------------------------------------------------------------
// Factored-table kernel (whole K per workgroup).
//
// The 243-entry table of a pack factors into two small ones: with the code
// split c = lo + 9 hi (lo = d0 + 3 d1, hi = d2 + 3 d3 + 9 d4),
//   L[c] = T_lo[lo] + T_hi[hi],  T_lo[lo] = sum_{i<2} (d_i - 1) a_i,
//                                 T_hi[hi] = sum_{i=2..4} (d_i - 1) a_i.
// 36 instead of 243 entries per pack (144 bytes at batch 1) lets one CU hold
// the tables of K up to 5120 columns at once, so a workgroup owns whole rows:
// no K split, no cross-workgroup reduction, no workspace.  K beyond one
// table chunk is walked in chunks, the table rebuilt per chunk.
//
// Lane mapping: a wave covers 16 rows (one per lane of a quarter-wave) and
// four consecutive groups (one per quarter); the KS waves of a 16-row block
// take interleaved groups.  Byte i of a row's unit is pack slot (i + row) mod
// 16, so the 16 lanes of a quarter address 16 different packs and the four
// quarters four different groups: with tables laid out [index][pack] and a
// pack stride that is a multiple of 64 words, every lookup instruction hits
// 64 distinct banks.
// ---------------------------------------------------------------------------
struct FkArgs {
  const uint8_t* trits;
  const uint16_t* alpha;
  const uint16_t* v;
  const int32_t* S;
  const int32_t* spos;
  const uint16_t* rval;  // fp16, or E4M3 bytes when f8
  const uint32_t* ridx;
  const uint16_t* x;
  float* y;
  int64_t N, K, n_pad;
  int n_groups, nS;
  int f8;  // residual values are E4M3 bytes (layout 3)
  int R;   // rows per workgroup (multiple of 16)
  int KS;  // waves per 16-row block (K parts)
  int CG;  // 16-pack groups per table chunk (multiple of 4)
  int NP;  // table pack stride (multiple of 64, >= 16 CG)
};

constexpr int kFkU = 4;          // 16-byte units per lane per load batch
constexpr int kFkMaxThreads = 1024;

// Packs per table chunk (the table's pack stride) at batch B: 36 x NP x B
// floats stay within 150 KB, and NP * B is a multiple of 64 words.
template <int B>
constexpr int fk_np() {
  return B == 1 ? 1024 : B == 2 ? 512 : B == 3 ? 320 : 256;
}

template <int B>
__global__ __launch_bounds__(kFkMaxThreads) void fk_gemv_kernel(const FkArgs p) {
  extern __shared__ float smem[];
  constexpr int NP = fk_np<B>();
  float* tab = smem;                         // [36][NP][B]: T_lo rows 0..8, T_hi rows 9..35
  float* red = smem + 36 * NP * B;           // [R][KS][2B] per-wave partial sums
  const int nthreads = blockDim.x;
  const int tid = threadIdx.x, lane = tid & 63, q = lane >> 4, l16 = lane & 15;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rbk = wave / p.KS, kp = wave - rbk * p.KS;
  const int lpr = 4 * p.KS;                  // lanes per row
  const int li = q + 4 * kp;                 // this lane's index among its row's lanes
  const int64_t row = int64_t(blockIdx.x) * p.R + rbk * 16 + l16;
  const bool row_ok = rbk * 16 < p.R && row < p.n_pad;
  const int64_t tile = row >> 6;
  const uint32_t rowbit = uint32_t(row & 3), shift = 2 * uint32_t((row >> 2) & 15);

  // LDS byte address of this lane's first group, slot (i + row) mod 16, table row 0
  const lds_char* tab_l = (const lds_char*)smem;
  const uint32_t tab_base = uint32_t(size_t(tab_l));
  uint32_t soff[16];
#pragma unroll
  for (int i = 0; i < 16; ++i)
    soff[i] = tab_base + uint32_t((li * kGroupPacks + ((i + int(row)) & 15)) * B * 4);

  float acc[B], racc[B];
#pragma unroll
  for (int b = 0; b < B; ++b) acc[b] = racc[b] = 0.0f;

  constexpr uint32_t rstride = uint32_t(NP * B * 4);  // bytes per table index row
  constexpr uint32_t hi_off = 9u * rstride;            // T_hi follows the 9 rows of T_lo
  for (int cg0 = 0; cg0 < p.n_groups; cg0 += p.CG) {
    const int ncg = min(p.CG, p.n_groups - cg0);
    const int npk = ncg * kGroupPacks;
    const int64_t col0 = int64_t(cg0) * kGroupCols;
    // units (16-byte pieces of the row) of this lane: group li + lpr m of the chunk
    const int nu = row_ok && li < ncg ? (ncg - li + lpr - 1) / lpr : 0;
    auto unit_ptr = [&](int m) {
      return reinterpret_cast<const u32x4*>(
          p.trits + ((tile * p.n_groups + cg0 + li + lpr * m) * kTileRows + (row & 63)) * 16);
    };
    u32x4 wa[kFkU], wb[kFkU];
    auto load_units = [&](u32x4 (&w)[kFkU], int m0) {
#pragma unroll
      for (int u = 0; u < kFkU; ++u)
        w[u] = m0 + u < nu ? __builtin_nontemporal_load(unit_ptr(m0 + u)) : u32x4(kZeroCode4);
    };
    // salient columns of the chunk: this lane takes sb + li + lpr n
    const int sb = p.spos[cg0], se = p.spos[cg0 + ncg];
    // Activations of this thread's first table-build packs are requested
    // before any packed byte, so they do not queue behind the weight stream.
    constexpr int kFkT = 2;
    float xa[kFkT][5][B], va[kFkT][5];
    auto load_act = [&](int pl0) {
#pragma unroll
      for (int j = 0; j < kFkT; ++j) {
        const int pl = pl0 + j * nthreads;
        const int64_t c5 = col0 + 5 * pl;
#pragma unroll
        for (int i = 0; i < 5; ++i) {
          const bool use = pl < npk;
          va[j][i] = use ? h2f(p.v[c5 + i]) : 0.0f;  // v zero-padded to whole groups
#pragma unroll
          for (int b = 0; b < B; ++b) xa[j][i][b] = use && c5 + i < p.K ? h2f(p.x[b * p.K + c5 + i]) : 0.0f;
        }
      }
    };
    load_act(tid);
    load_units(wa, 0);  // first units stream in during the table build

    __syncthreads();  // previous chunk's readers of the tables are done
    // Table build: each thread takes whole packs (all 36 entries: T_lo from
    // digits 0-1, T_hi from digits 2-4), kFkT packs at a time with all their
    // activation loads issued first.
    for (int pl0 = tid; pl0 < npk; pl0 += kFkT * nthreads) {
      if (pl0 != tid) load_act(pl0);
#pragma unroll
      for (int j = 0; j < kFkT; ++j) {
        const int pl = pl0 + j * nthreads;
        if (pl >= npk) break;
        float a[5][B];
#pragma unroll
        for (int i = 0; i < 5; ++i)
#pragma unroll
          for (int b = 0; b < B; ++b) a[i][b] = va[j][i] * xa[j][i][b];
        float* dst = tab + int64_t(pl) * B;
        // T_lo[3 d1 + d0]
#pragma unroll
        for (int d1 = 0; d1 < 3; ++d1)
#pragma unroll
          for (int d0 = 0; d0 < 3; ++d0)
#pragma unroll
            for (int b = 0; b < B; ++b) {
              float e = d1 == 0 ? -a[1][b] : (d1 == 2 ? a[1][b] : 0.0f);
              e = d0 == 0 ? e - a[0][b] : (d0 == 2 ? e + a[0][b] : e);
              dst[int64_t(d1 * 3 + d0) * NP * B + b] = e;
            }
        // T_hi[9 d4 + 3 d3 + d2], rows 9..35
#pragma unroll
        for (int d4 = 0; d4 < 3; ++d4)
#pragma unroll
          for (int d3 = 0; d3 < 3; ++d3)
#pragma unroll
            for (int d2 = 0; d2 < 3; ++d2)
#pragma unroll
              for (int b = 0; b < B; ++b) {
                float e = d4 == 0 ? -a[4][b] : (d4 == 2 ? a[4][b] : 0.0f);
                e = d3 == 0 ? e - a[3][b] : (d3 == 2 ? e + a[3][b] : e);
                e = d2 == 0 ? e - a[2][b] : (d2 == 2 ? e + a[2][b] : e);
                dst[int64_t(9 + d4 * 9 + d3 * 3 + d2) * NP * B + b] = e;
              }
      }
    }
    // residual loads of this lane's salient columns (first batch), in flight during the build
    constexpr int RB = 8;
    int rs_col[RB];
    uint32_t rs_word[RB];
    uint16_t rs_val[RB];
    auto load_res = [&](int n0) {
#pragma unroll
      for (int u = 0; u < RB; ++u) {
        const int s = sb + li + lpr * (n0 + u);
        const bool ok = row_ok && s < se;
        rs_col[u] = ok ? p.S[s] : -1;
        rs_word[u] = ok ? p.ridx[tile * p.nS + s] : 0u;
        const int64_t vi = rval_index(row >> 2, s, p.nS);
        rs_val[u] = !ok ? uint16_t(0)
                    : p.f8 ? e4m3_to_half_bits(reinterpret_cast<const uint8_t*>(p.rval)[vi]) : p.rval[vi];
      }
    };
    load_res(0);
    __syncthreads();
    // activations at the first batch of salient columns: land during the lookups
    float xv[RB][B];
    auto load_xv = [&]() {
#pragma unroll
      for (int u = 0; u < RB; ++u)
#pragma unroll
        for (int b = 0; b < B; ++b) xv[u][b] = rs_col[u] >= 0 ? h2f(p.x[b * p.K + rs_col[u]]) : 0.0f;
    };
    load_xv();

    // Lookup-accumulate: two table entries per packed byte.
    auto consume = [&](const u32x4 (&w)[kFkU], int m0) {
#pragma unroll
      for (int u = 0; u < kFkU; ++u) {
        if (m0 + u >= nu) break;
        // groups of this lane are li + lpr m: the part beyond the first is wave-uniform
        const uint32_t um = uint32_t(lpr * (m0 + u) * kGroupPacks * B * 4);
        const uint32_t ww[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const uint32_t c = (ww[i >> 2] >> (8 * (i & 3))) & 0xffu;
          const uint32_t hi = __umul24(c, 57u) >> 9;  // c / 9 for c < 243
          const uint32_t lo = c - 9u * hi;
          const uint32_t so = soff[i] + um;
          const lds_float* elo = (const lds_float*)(size_t)(lo * rstride + so);
          const lds_float* ehi = (const lds_float*)(size_t)(hi * rstride + so + hi_off);
#pragma unroll
          for (int b = 0; b < B; ++b) acc[b] += elo[b] + ehi[b];
        }
      }
    };
    for (int m0 = 0; m0 < nu; m0 += 2 * kFkU) {
      load_units(wb, m0 + kFkU);
      consume(wa, m0);
      load_units(wa, m0 + 2 * kFkU);
      consume(wb, m0 + kFkU);
    }

    // Salient residual of the chunk: scaled by neither alpha nor v.
    const int nres = row_ok && sb + li < se ? (se - sb - li + lpr - 1) / lpr : 0;
    for (int n0 = 0; n0 < nres; n0 += RB) {
      if (n0 > 0) {
        load_res(n0);
        load_xv();
      }
#pragma unroll
      for (int u = 0; u < RB; ++u) {
        if (rs_col[u] >= 0 && ((rs_word[u] >> shift) & 3u) == rowbit) {
          const float rv = h2f(rs_val[u]);
#pragma unroll
          for (int b = 0; b < B; ++b) racc[b] += rv * xv[u][b];
        }
      }
    }
  }

  // Reduce the row's 4 KS partial sums in a fixed order: the four quarters
  // of the wave first, then the KS waves of the row block through LDS.
#pragma unroll
  for (int b = 0; b < B; ++b) {
    acc[b] += __shfl_xor(acc[b], 16);
    acc[b] += __shfl_xor(acc[b], 32);
    racc[b] += __shfl_xor(racc[b], 16);
    racc[b] += __shfl_xor(racc[b], 32);
  }
  if (q == 0 && rbk * 16 < p.R) {
    float* r = red + ((rbk * 16 + l16) * p.KS + kp) * 2 * B;
#pragma unroll
    for (int b = 0; b < B; ++b) {
      r[b] = acc[b];
      r[B + b] = racc[b];
    }
  }
  __syncthreads();
  for (int e = tid; e < p.R * B; e += nthreads) {
    const int rr = e / B, b = e - rr * B;
    const int64_t orow = int64_t(blockIdx.x) * p.R + rr;
    if (orow >= p.N) continue;
    float sa = 0.0f, sr = 0.0f;
    for (int k = 0; k < p.KS; ++k) {
      sa += red[(rr * p.KS + k) * 2 * B + b];
      sr += red[(rr * p.KS + k) * 2 * B + B + b];
    }
    p.y[b * p.N + orow] = h2f(p.alpha[orow]) * sa + sr;
  }
}

// ---------------------------------------------------------------------------
// Launch planning.
// ---------------------------------------------------------------------------
struct Plan {
  int tpw, nrb, nslices, ks_groups;
};

int kc_for_batch(int B) {
  const int bt = B < 4 ? B : 4;
  return bt == 1 ? 4 : (bt == 2 ? 2 : 1);
}

Plan make_plan(const qtea_desc& d, int B) {
  Plan pl;
  const int64_t n_tiles = d.n_pad / kTileRows;
  const int kc = kc_for_batch(B);
  pl.tpw = n_tiles >= 256 ? 2 : 1;
  pl.nrb = int(cdiv(n_tiles, int64_t(kWaves) * pl.tpw));
  const int64_t target_wgs = 640;
  int64_t nsl = cdiv(target_wgs, pl.nrb);
  // Partial sums cost 8 bytes per row and batch vector per slice (write and
  // read back); keep them to about a quarter of the row's packed bytes.
  const int64_t cap = d.n_packs / (32 * int64_t(B));
  if (nsl > cap) nsl = cap;
  if (nsl < 1) nsl = 1;
  int64_t ks = cdiv(d.n_groups, nsl);
  ks = cdiv(ks, kc) * kc;
  pl.ks_groups = int(ks);
  pl.nslices = int(cdiv(d.n_groups, ks));
  return pl;
}

// Batches up to 4 run the factored-table kernel (whole rows per workgroup,
// no partial sums); larger batches the K-split table kernel.
bool use_fk(int B) { return B <= 4; }

int64_t workspace_need(const qtea_desc& d, int B) {
  const Plan pl = make_plan(d, B);
  const int64_t counters = align_up(4 * cdiv(d.n_pad / kTileRows, kWaves), kAlign);
  const int64_t parts = !use_fk(B) && pl.nslices > 1 ? 4 * int64_t(pl.nslices) * B * d.n_pad : 0;
  return counters + parts;
}

template <int B, int TPW>
hipError_t launch_t(const GemvArgs& a, int grid, hipStream_t st) {
  hipLaunchKernelGGL((lut_gemv_kernel<B, TPW>), dim3(grid), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

template <int B>
hipError_t launch_b(const GemvArgs& a, int tpw, int grid, hipStream_t st) {
  return tpw == 2 ? launch_t<B, 2>(a, grid, st) : launch_t<B, 1>(a, grid, st);
}

hipError_t launch_gemv(const GemvArgs& a, int B, int tpw, int grid, hipStream_t st) {
  switch (B) {
    case 1: return launch_b<1>(a, tpw, grid, st);
    case 2: return launch_b<2>(a, tpw, grid, st);
    case 3: return launch_b<3>(a, tpw, grid, st);
    case 4: return launch_b<4>(a, tpw, grid, st);
    case 5: return launch_b<5>(a, tpw, grid, st);
    case 6: return launch_b<6>(a, tpw, grid, st);
    case 7: return launch_b<7>(a, tpw, grid, st);
    case 8: return launch_b<8>(a, tpw, grid, st);
    case 9: return launch_b<9>(a, tpw, grid, st);
    case 10: return launch_b<10>(a, tpw, grid, st);
    case 11: return launch_b<11>(a, tpw, grid, st);
    case 12: return launch_b<12>(a, tpw, grid, st);
    case 13: return launch_b<13>(a, tpw, grid, st);
    case 14: return launch_b<14>(a, tpw, grid, st);
    case 15: return launch_b<15>(a, tpw, grid, st);
    case 16: return launch_b<16>(a, tpw, grid, st);
    default: return hipErrorInvalidValue;
  }
}

int grid_for(int64_t n, int64_t per_thread_block = 256) {
  int64_t g = cdiv(n, per_thread_block);
  if (g < 1) g = 1;
  if (g > 65536) g = 65536;
  return int(g);
}

// Plan of the factored-table kernel.
struct FkPlan {
  int R, KS, CG, NP, threads, grid;
  size_t lds;
};

constexpr size_t kLdsBytes = 160 * 1024;

FkPlan fk_plan(const qtea_desc& d, int B) {
  FkPlan f;
  // Rows per workgroup: one workgroup per CU covers the matrix (multiples of 16 rows).
  f.R = int(cdiv(cdiv(d.N, 16), 256) * 16);
  if (f.R > 256) f.R = 256;
  f.grid = int(cdiv(d.N, f.R));
  const int blocks = f.R / 16;
  const int G = int(d.n_groups);
  // K parts per 16-row block: up to 16 waves per workgroup.
  int ks = 16 / blocks;
  if (ks < 1) ks = 1;
  // Table chunk: the kernel's fixed pack stride bounds the groups per chunk;
  // chunks are balanced.
  const int np = B == 1 ? fk_np<1>() : B == 2 ? fk_np<2>() : B == 3 ? fk_np<3>() : fk_np<4>();
  const int cgmax = np / kGroupPacks;
  const int nch = int(cdiv(G, cgmax));
  f.CG = int(cdiv(G, nch));
  f.NP = np;
  const int maxks = int(cdiv(f.CG, 4));  // at least one group per lane
  f.KS = ks < maxks ? ks : maxks;
  f.threads = blocks * f.KS * 64;
  f.lds = size_t(36) * f.NP * B * 4 + size_t(f.R) * f.KS * 2 * B * 4;
  return f;
}

template <int B>
hipError_t launch_fk(const FkArgs& a, const FkPlan& f, hipStream_t st) {
  static bool attr = false;
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&fk_gemv_kernel<B>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, int(kLdsBytes));
    if (e != hipSuccess) return e;
    attr = true;
  }
  hipLaunchKernelGGL(fk_gemv_kernel<B>, dim3(f.grid), dim3(f.threads), f.lds, st, a);
  return hipGetLastError();
}

hipError_t launch_fk_b(const FkArgs& a, const FkPlan& f, int B, hipStream_t st) {
  switch (B) {
    case 1: return launch_fk<1>(a, f, st);
    case 2: return launch_fk<2>(a, f, st);
    case 3: return launch_fk<3>(a, f, st);
    case 4: return launch_fk<4>(a, f, st);
    default: return hipErrorInvalidValue;
  }
}


}  // namespace

// ---------------------------------------------------------------------------
// C ABI.
// ---------------------------------------------------------------------------
extern "C" {

const char* qtea_status_string(int status) {
  switch (status) {
    case QTEA_OK: return "ok";
    case QTEA_ERR_INVALID_ARG: return "invalid argument";
    case QTEA_ERR_BAD_TRIT: return "trit outside {-1, 0, +1}";
    case QTEA_ERR_BAD_RESIDUAL: return "bad residual position or salient column list";
    case QTEA_ERR_BATCH: return "batch outside [1, 16]";
    case QTEA_ERR_WORKSPACE: return "workspace or packed buffer too small";
    case QTEA_ERR_HIP: return "HIP runtime error";
    case QTEA_ERR_NOT_POSITIVE: return "Hessian not positive definite";
    default: return "unknown status";
  }
}

int qtea_abi_version(void) { return QTEA_ABI_VERSION; }

int qtea_packed_bytes(int64_t N, int64_t K, int64_t n_salient, int64_t* out_bytes) {
  Layout L;
  if (!out_bytes || !make_layout(N, K, n_salient, &L)) return QTEA_ERR_INVALID_ARG;
  *out_bytes = L.total;
  return QTEA_OK;
}

int qtea_packed_bytes_e4m3(int64_t N, int64_t K, int64_t n_salient, int64_t* out_bytes) {
  Layout L;
  if (!out_bytes || !make_layout(N, K, n_salient, &L, kLayoutE4M3)) return QTEA_ERR_INVALID_ARG;
  *out_bytes = L.total;
  return QTEA_OK;
}

}  // extern "C"

namespace {

// The pack entry points: layout 2 takes a salient list and fp16 residual
// values, layout 3 a salient bitmap and E4M3 residual bytes, layout 4 that
// and per-row, per-128-column-group scales and biases (row_scale and
// row_bias [N][ceil(K/128)]).
int pack_any(int layout, const int8_t* trits, int64_t N, int64_t K, const uint16_t* row_scale,
             const uint16_t* row_bias, const uint16_t* col_rescale, const int32_t* salient,
             const uint32_t* bitmap, int64_t n_salient, const void* resid_val, const uint8_t* resid_idx,
             void* packed, int64_t packed_bytes, qtea_desc* out_desc, void* stream) {
  Layout L;
  if (!out_desc) return QTEA_ERR_INVALID_ARG;
  out_desc->magic = 0;
  if (!make_layout(N, K, n_salient, &L, layout)) return QTEA_ERR_INVALID_ARG;
  if (!trits || !row_scale || !col_rescale || !packed) return QTEA_ERR_INVALID_ARG;
  if (layout == kLayoutG128 && !row_bias) return QTEA_ERR_INVALID_ARG;
  if (n_salient > 0 && (!resid_val || !resid_idx)) return QTEA_ERR_INVALID_ARG;
  if (layout == kLayout ? (n_salient > 0 && !salient) : !bitmap) return QTEA_ERR_INVALID_ARG;
  if (packed_bytes < L.total) return QTEA_ERR_WORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* pk = static_cast<uint8_t*>(packed);
  uint32_t* flags = reinterpret_cast<uint32_t*>(pk + kFlagOffset);
  int32_t* o_S = reinterpret_cast<int32_t*>(pk + L.off_salient);

  hipLaunchKernelGGL(write_header_kernel, dim3(1), dim3(64), 0, st, pk, N, K, n_salient, layout);
  const int64_t ni = n_salient * (N / 4);
  // the salient list given is checked here; one derived from a bitmap is
  // checked as it is derived
  hipLaunchKernelGGL(validate_kernel, dim3(grid_for(N * K, 256 * 16)), dim3(256), 0, st, trits, N * K,
                     resid_idx, ni, layout == kLayout ? salient : nullptr,
                     layout == kLayout ? n_salient : int64_t(0), K, flags);
  if (layout != kLayout) {
    hipLaunchKernelGGL(bitmap_salient_kernel, dim3(1), dim3(1024), 0, st, bitmap, K, n_salient, o_S, flags);
    salient = o_S;
  }
  const int64_t n_units = L.n_tiles * L.n_groups * kTileRows;
  if (layout == kLayoutG128) {
    const int64_t n_sg = L.n_groups / 2;
    hipLaunchKernelGGL(pack_trits128_kernel, dim3(grid_for(n_units)), dim3(256), 0, st, trits, N, K,
                       L.n_groups, n_units, pk + L.off_trits);
    hipLaunchKernelGGL(pack_scales128_kernel, dim3(grid_for(L.n_pad * n_sg)), dim3(256), 0, st, row_scale,
                       row_bias, col_rescale, N, K, L.n_pad, n_sg, reinterpret_cast<uint32_t*>(pk + L.off_alpha),
                       reinterpret_cast<uint16_t*>(pk + L.off_v));
  } else {
    hipLaunchKernelGGL(pack_trits_kernel, dim3(grid_for(n_units)), dim3(256), 0, st, trits, N, K,
                       L.n_groups, n_units, pk + L.off_trits);
  }
  const int64_t meta_n = L.n_pad + L.n_groups * kGroupCols + n_salient * (L.n_pad / 4);
  uint16_t* o_alpha = layout == kLayoutG128 ? nullptr : reinterpret_cast<uint16_t*>(pk + L.off_alpha);
  uint16_t* o_v = layout == kLayoutG128 ? nullptr : reinterpret_cast<uint16_t*>(pk + L.off_v);
  int32_t* o_spos = reinterpret_cast<int32_t*>(pk + L.off_spos);
  uint32_t* o_ridx = reinterpret_cast<uint32_t*>(pk + L.off_ridx);
  if (layout == kLayout)
    hipLaunchKernelGGL(pack_meta_kernel<uint16_t>, dim3(grid_for(meta_n)), dim3(256), 0, st, row_scale,
                       col_rescale, salient, static_cast<const uint16_t*>(resid_val), resid_idx, N, K,
                       n_salient, L.n_pad, L.n_groups, o_alpha, o_v, o_S, o_spos,
                       reinterpret_cast<uint16_t*>(pk + L.off_rval), o_ridx, flags, 0);
  else
    hipLaunchKernelGGL(pack_meta_kernel<uint8_t>, dim3(grid_for(meta_n)), dim3(256), 0, st, row_scale,
                       col_rescale, salient, static_cast<const uint8_t*>(resid_val), resid_idx, N, K,
                       n_salient, L.n_pad, L.n_groups, o_alpha, o_v, o_S, o_spos, pk + L.off_rval, o_ridx,
                       flags, int(layout == kLayoutG128));
  {
    uint32_t* o_vs = reinterpret_cast<uint32_t*>(pk + L.off_vs);
    const uint16_t* v_dev = reinterpret_cast<const uint16_t*>(pk + L.off_v);
    const int64_t n_cols = L.n_groups * kGroupCols;
    hipLaunchKernelGGL(pack_vs_kernel, dim3(grid_for(n_cols)), dim3(256), 0, st, v_dev, n_cols, o_vs);
    if (n_salient > 0)
      hipLaunchKernelGGL(mark_salient_kernel, dim3(grid_for(n_salient)), dim3(256), 0, st, o_S, o_spos, n_salient,
                         K, L.n_groups, int(layout == kLayoutG128), o_vs);
  }
  if (hipGetLastError() != hipSuccess) return QTEA_ERR_HIP;
  uint32_t hflags = 0;
  if (hipMemcpyAsync(&hflags, flags, 4, hipMemcpyDeviceToHost, st) != hipSuccess) return QTEA_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return QTEA_ERR_HIP;
  if (hflags & kFlagBadTrit) return QTEA_ERR_BAD_TRIT;
  if (hflags & kFlagBadResid) return QTEA_ERR_BAD_RESIDUAL;

  qtea_desc d;
  d.magic = QTEA_DESC_MAGIC;
  d.layout = uint32_t(layout);
  d.N = N;
  d.K = K;
  d.n_salient = n_salient;
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
  *out_desc = d;
  return QTEA_OK;
}

}  // namespace

extern "C" {

int qtea_pack(const int8_t* trits, int64_t N, int64_t K, const uint16_t* row_scale,
              const uint16_t* col_rescale, const int32_t* salient, int64_t n_salient,
              const uint16_t* resid_val, const uint8_t* resid_idx, void* packed,
              int64_t packed_bytes, qtea_desc* out_desc, void* stream) {
  return pack_any(kLayout, trits, N, K, row_scale, nullptr, col_rescale, salient, nullptr, n_salient, resid_val,
                  resid_idx, packed, packed_bytes, out_desc, stream);
}

int qtea_pack_e4m3(const int8_t* trits, int64_t N, int64_t K, const uint16_t* row_scale,
                   const uint16_t* col_rescale, const uint32_t* salient_bitmap, int64_t n_salient,
                   const uint8_t* resid_val, const uint8_t* resid_idx, void* packed, int64_t packed_bytes,
                   qtea_desc* out_desc, void* stream) {
  return pack_any(kLayoutE4M3, trits, N, K, row_scale, nullptr, col_rescale, nullptr, salient_bitmap, n_salient,
                  resid_val, resid_idx, packed, packed_bytes, out_desc, stream);
}

int qtea_packed_bytes_g128(int64_t N, int64_t K, int64_t n_salient, int64_t* out_bytes) {
  Layout L;
  if (!out_bytes || !make_layout(N, K, n_salient, &L, kLayoutG128)) return QTEA_ERR_INVALID_ARG;
  *out_bytes = L.total;
  return QTEA_OK;
}

int qtea_pack_g128(const int8_t* trits, int64_t N, int64_t K, const uint16_t* group_scale,
                   const uint16_t* group_bias, const uint16_t* col_rescale, const uint32_t* salient_bitmap,
                   int64_t n_salient, const uint8_t* resid_val, const uint8_t* resid_idx, void* packed,
                   int64_t packed_bytes, qtea_desc* out_desc, void* stream) {
  return pack_any(kLayoutG128, trits, N, K, group_scale, group_bias, col_rescale, nullptr, salient_bitmap,
                  n_salient, resid_val, resid_idx, packed, packed_bytes, out_desc, stream);
}

int qtea_workspace_bytes(const qtea_desc* desc, int batch, int64_t* out_bytes) {
  if (!out_bytes || !desc_ok(desc) || desc->layout == kLayoutG128) return QTEA_ERR_INVALID_ARG;
  if (batch < 1 || batch > QTEA_MAX_BATCH) return QTEA_ERR_BATCH;
  *out_bytes = workspace_need(*desc, batch);
  return QTEA_OK;
}

int qtea_workspace_init(void* workspace, int64_t bytes, void* stream) {
  if (!workspace || bytes < 0 || (reinterpret_cast<uintptr_t>(workspace) & 3)) return QTEA_ERR_INVALID_ARG;
  if (bytes == 0) return QTEA_OK;
  const int64_t words = bytes / 4;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(grid_for(words)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<uint32_t*>(workspace), words,
                     static_cast<uint8_t*>(workspace) + 4 * words, bytes - 4 * words);
  return hipGetLastError() == hipSuccess ? QTEA_OK : QTEA_ERR_HIP;
}

int qtea_gemm_lowbatch(const qtea_desc* desc, const void* packed, const uint16_t* X, int batch,
                       float* Y, void* workspace, int64_t workspace_bytes, void* stream) {
  if (!desc_ok(desc) || !packed || !X || !Y) return QTEA_ERR_INVALID_ARG;
  if (desc->layout == kLayoutG128) return QTEA_ERR_INVALID_ARG;  // grouped entry points only
  if (batch < 1 || batch > QTEA_MAX_BATCH) return QTEA_ERR_BATCH;
  const qtea_desc& d = *desc;
  const Plan pl = make_plan(d, batch);
  const int64_t need = workspace_need(d, batch);
  if (!workspace || workspace_bytes < need) return QTEA_ERR_WORKSPACE;
  const uint8_t* pk = static_cast<const uint8_t*>(packed);
  GemvArgs a;
  a.trits = pk + d.off_trits;
  a.alpha = reinterpret_cast<const uint16_t*>(pk + d.off_alpha);
  a.v = reinterpret_cast<const uint16_t*>(pk + d.off_v);
  a.S = reinterpret_cast<const int32_t*>(pk + d.off_salient);
  a.spos = reinterpret_cast<const int32_t*>(pk + d.off_spos);
  a.rval = reinterpret_cast<const uint16_t*>(pk + d.off_rval);
  a.ridx = reinterpret_cast<const uint32_t*>(pk + d.off_ridx);
  a.x = X;
  a.y = Y;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  a.counters = reinterpret_cast<uint32_t*>(ws);
  a.part = reinterpret_cast<float*>(ws + align_up(4 * cdiv(d.n_pad / kTileRows, kWaves), kAlign));
  a.N = d.N;
  a.K = d.K;
  a.n_pad = d.n_pad;
  a.n_groups = int(d.n_groups);
  a.n_tiles = int(d.n_pad / kTileRows);
  a.nS = int(d.n_salient);
  a.f8 = d.layout == kLayoutE4M3;
  a.nrb = pl.nrb;
  a.nslices = pl.nslices;
  a.ks_groups = pl.ks_groups;
  if (use_fk(batch)) {
    const FkPlan f = fk_plan(d, batch);
    FkArgs k;
    k.trits = a.trits;
    k.alpha = a.alpha;
    k.v = a.v;
    k.S = a.S;
    k.spos = a.spos;
    k.rval = a.rval;
    k.ridx = a.ridx;
    k.x = a.x;
    k.y = a.y;
    k.N = a.N;
    k.K = a.K;
    k.n_pad = a.n_pad;
    k.n_groups = a.n_groups;
    k.nS = a.nS;
    k.f8 = a.f8;
    k.R = f.R;
    k.KS = f.KS;
    k.CG = f.CG;
    k.NP = f.NP;
    return launch_fk_b(k, f, batch, static_cast<hipStream_t>(stream)) == hipSuccess ? QTEA_OK : QTEA_ERR_HIP;
  }
  const int grid = pl.nrb * pl.nslices;
  if (launch_gemv(a, batch, pl.tpw, grid, static_cast<hipStream_t>(stream)) != hipSuccess)
    return QTEA_ERR_HIP;
  return QTEA_OK;
}

int qtea_gemv(const qtea_desc* desc, const void* packed, const uint16_t* x, float* y, void* workspace,
              int64_t workspace_bytes, void* stream) {
  return qtea_gemm_lowbatch(desc, packed, x, 1, y, workspace, workspace_bytes, stream);
}

int qtea_read_ceiling(const void* buf, int64_t bytes, uint32_t* sink, void* stream) {
  if (!buf || !sink || bytes <= 0 || bytes % 16 != 0 || (reinterpret_cast<uintptr_t>(buf) & 15))
    return QTEA_ERR_INVALID_ARG;
  const int64_t n16 = bytes / 16, grid = (n16 + kCeilChunk16 - 1) / kCeilChunk16;
  if (grid > int64_t(INT32_MAX)) return QTEA_ERR_INVALID_ARG;
  hipLaunchKernelGGL(read_ceiling_kernel, dim3(uint32_t(grid)), dim3(kCeilThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4*>(buf), n16, kCeilChunk16, sink);
  return hipGetLastError() == hipSuccess ? QTEA_OK : QTEA_ERR_HIP;
}

int qtea_debug_unpack(const qtea_desc* desc, const void* packed, uint8_t* canon_codes, int8_t* trits,
                      int32_t* resid_row, void* stream) {
  if (!desc_ok(desc) || !packed) return QTEA_ERR_INVALID_ARG;
  const qtea_desc& d = *desc;
  const uint8_t* pk = static_cast<const uint8_t*>(packed);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if ((canon_codes || trits) && d.layout == kLayoutG128)
    hipLaunchKernelGGL(unpack_codes128_kernel, dim3(grid_for(d.N * d.n_packs)), dim3(256), 0, st,
                       pk + d.off_trits, d.N, d.K, d.n_packs, d.n_groups, canon_codes, trits);
  else if (canon_codes || trits)
    hipLaunchKernelGGL(unpack_codes_kernel, dim3(grid_for(d.N * d.n_packs)), dim3(256), 0, st,
                       pk + d.off_trits, d.N, d.K, d.n_packs, d.n_groups, canon_codes, trits);
  if (resid_row && d.n_salient > 0)
    hipLaunchKernelGGL(unpack_resid_kernel, dim3(grid_for(d.n_salient * (d.N / 4))), dim3(256), 0, st,
                       reinterpret_cast<const uint32_t*>(pk + d.off_ridx), d.N, d.n_salient, d.n_pad,
                       resid_row);
  return hipGetLastError() == hipSuccess ? QTEA_OK : QTEA_ERR_HIP;
}

}  // extern "C"
