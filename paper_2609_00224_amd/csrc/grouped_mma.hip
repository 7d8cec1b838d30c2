// Grouped low-batch GEMM on the matrix cores: Y_m = X_m W_m^T for 2 <= B <=
// 16 activation rows per problem (Eq. 10 with one group and zero bias, plus
// the Eq. 11 residual), every problem of a plan in one persistent launch.
//
// At batch B the product is a dense contraction of the ternary weights with
// a B-column activation block, so it runs on v_mfma_f32_16x16x32_f16 with
// fp32 accumulation:
//
//   A (16 output rows x 32 columns): the ternary codes themselves as fp16
//     -1 / 0 / +1 (exact), decoded from the packed bytes by one table lookup
//     per byte in LDS;
//   B (32 columns x 16): a_j = v_j x[b][j] (exact in fp32: 11-bit by 11-bit
//     significands) split into two fp16 halves hi = fp16(a), lo = fp16(a -
//     hi), so hi + lo reproduces a (to 2^-25 absolute for |a| < 1/8, exactly
//     above); with B <= 8 the 16 columns hold hi of every batch row and lo of
//     every batch row, with B <= 16 hi and lo are two MFMAs (NB = 2);
//   y[b][r] = alpha_r (C[r][hi b] + C[r][lo b]) + residual.
//
// A slice whose |a| reaches the fp16 range is scaled by 2^-16 before the
// split (and its products by 2^16 after): rare, handled on a slow path.
//
// Work unit = (problem, panel of MRP rows, K slice of 4 sixteen-pack groups
// = 320 columns), the same units and plan as the batch-1 kernel; here one
// workgroup of MRP threads per CU (MShape below) takes one contiguous run of
// units.  Per unit:
//
//   - each wave owns one 64-row tile of the panel: four MFMA row tiles, tile
//     q holding rows 16m + 4q + s (m, s < 4), whose bytes are rotated by the
//     same 4q + s (byte i of row r is pack (i + r) mod 16 of its group): the
//     4q part is undone by register choice, the s part by one v_perm per
//     dword;
//   - lane (row i, k-block kb) decodes its row's 16-byte group unit (16 packs
//     of group kb of the slice): per byte one v_perm forms the LDS address of
//     that code's entry (32 copies of the 243-entry table, one per lane of a
//     half-wave, so a half-wave's reads hit distinct banks), one 8-byte read
//     gives digits 0-3 as two fp16 pairs (the A operand pairs as they are),
//     and a 2-byte read from a 32-copy digit-4 table at half that address
//     gives digit 4 (one v_perm pairs two bytes' digit 4 into one operand
//     register); with two column blocks (NB = 2, batch 9..16) one table of
//     16-byte entries (digits 0-4 and a pad, 16 copies) gives all five
//     digits in one 12-byte read per byte, and a v_perm pairs the digit-4
//     halves (half the LDS reads; at NB = 1 this form measured slower: its
//     entries' registers spill inside the loop);
//   - ten MFMAs per row tile and column block: eight take digits 0-3 of two
//     packs each, two take digit 4 of eight packs each; the B operands are
//     per slice images in LDS, one 16-byte slot per MFMA lane (slots swizzled
//     per MFMA), built one unit ahead from x and v;
//   - at the end of a panel part: scale by alpha, add the residual of the
//     part's salient columns with one more MFMA per 32 of them (A = the 1:4
//     residual expanded per row, B = x at the salient columns), add hi and
//     lo, and store y (or the part's partial rows, summed afterwards by
//     grouped_reduce_kernel in run order).
#include "grouped_plan.h"

namespace qtea_grouped {
namespace {

// Workgroup shape (one workgroup per CU; each wave owns one 64-row tile).
// Grouped launches: 1024 threads at NB = 1, 768 at NB = 2, whose larger
// register budget (168 instead of 128 per lane) takes its spills from about
// 40 registers to 5 (8B stack, batch 16: 827 -> 720 us per token; at NB = 1
// the 768-thread shape, with no spills to remove, lost 25 % to the fewer
// waves).  One matrix on its own: 512 threads at both (256 registers, no
// spills, and twice the panels of a short launch to spread over the CUs:
// the 8B stack chained at batch 4 / 8 / 16 takes 2104 / 2178 / 2685 us
// against 2406 / 2560 / 3314 with the grouped shapes; 256 threads were
// slower again).
template <int NB, bool ONE>
struct MShape {
  static constexpr int MT = ONE ? 512 : (NB == 1 ? 1024 : 768);  // threads per workgroup
  static constexpr int MRP = MT;                                  // rows per panel (64 per wave)
};
constexpr int kMu = 10;                   // MFMAs per group unit and column block
constexpr int kRowStride = 256;           // bytes per code in the digit 0-3 table (32 copies x 8)
// Rows of both decode tables: one per code; the debug build (QTEA_DEBUG)
// adds rows for the unused byte values 243..255 filled with fp16 NaN, so a
// packed byte that is no base-3 code makes its output rows NaN.
#ifdef QTEA_DEBUG
constexpr int kTabRows = 256;
#else
constexpr int kTabRows = kCodes;
#endif
constexpr int kTab = kTabRows * kRowStride; // 62,208 bytes (65,536 in the debug build)
// Digit-4 table: code c, copy k at kTab + c * 128 + 4 k, half the digit 0-3
// entry's address plus a constant (one shift per byte).  Its reads have a
// 4-byte stride across a half-wave; a table at the digit 0-3 entry's own
// address (8-byte stride) takes twice as long per 2-byte read.
constexpr int kT4Bytes = kTabRows * 128;
constexpr int kImg = kMu * 64 * 16;       // one B-operand image (10 MFMAs x 64 lanes x 16 bytes)
constexpr float kBigScale = 1.0f / 65536.0f;

template <int NB>
struct MLds {
  static constexpr bool E12 = NB == 2;  // one 16-byte entry per code and copy, no digit-4 table
  static constexpr int T4OFF = kTab;
  // (E12 leaves the digit-4 region unused: with the images at the same
  // offsets as at NB = 1 the kernel measured 5 % faster than with them moved
  // down into it)
  static constexpr int IMG = kTab + kT4Bytes;  // [2 buffers][NB] images
  static constexpr int FLAG = IMG + 2 * NB * kImg;    // int [3]: slice needs scaling
  // residual hit masks: u32x2 [position p][position byte t]
  static constexpr int RMASK = FLAG + 16;
  // the rest: the open panel part's activations at its salient columns,
  // fp16 [part rank][8 NB batch rows], gathered as the slices are staged
  static constexpr int XSAL = RMASK + 4 * 256 * 8;
  static constexpr int XCAP = (160 * 1024 - XSAL - 256) / (2 * 8 * NB);  // salient columns held
  static constexpr int XDUMMY = XSAL + XCAP * 2 * 8 * NB;  // a dword per lane: the stores of other columns
  static constexpr int BYTES = XDUMMY + 256;
};

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) const u32x2 lds_u32x2;
typedef __attribute__((address_space(1))) const u32x2 gu32x2;
typedef __attribute__((address_space(3))) const u32x4 lds_u32x4;
typedef unsigned int u32x3 __attribute__((ext_vector_type(3)));
typedef __attribute__((address_space(3))) const u32x3 lds_u32x3;
typedef __attribute__((address_space(3))) const _Float16 lds_h;
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

// Two table halves into one dword (the second into the high half).
__device__ __forceinline__ uint32_t lds_pair(uint32_t a0, uint32_t a1) {
  half2_t r;
  r.x = *(lds_h*)(size_t(a0));
  r.y = *(lds_h*)(size_t(a1));
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ half8 as_half8(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  const u32x4 v = {a, b, c, d};
  return __builtin_bit_cast(half8, v);
}

// Column (within the slice) of k slot h of MFMA mu for k-block kb: MFMAs 0-7
// take digits 0-3 of packs 2 mu and 2 mu + 1, MFMAs 8 and 9 digit 4 of packs
// 0-7 and 8-15 of the group.
__device__ __forceinline__ void slot_of_col(int c, int& kb, int& mu, int& h) {
  kb = c / kGroupCols;
  const int rem = c - kb * kGroupCols;
  const int pp = rem / 5, d = rem - 5 * pp;
  if (d < 4) {
    mu = pp >> 1;
    h = 4 * (pp & 1) + d;
  } else {
    mu = 8 + (pp >> 3);
    h = pp & 7;
  }
}

// Slot of MFMA lane L's 16-byte B operand in MFMA mu's 1 KiB image block:
// the low four bits of L are xored with mu.  The builders write 2-byte
// halves, consecutive threads taking consecutive columns, which fall in
// different MFMAs at one lane: unswizzled, those all sit 1 KiB apart, in
// the same four banks; with the xor their dwords spread over the banks.
// The MFMA lanes read the whole block either way.
__device__ __forceinline__ constexpr int img_lane(int L, int mu) { return L ^ (mu & 15); }

// The value of lane (l + 8) mod 16 of the lane's row of 16 (row_ror:8).
__device__ __forceinline__ float dpp_ror8(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x128, 0xf, 0xf, false));
}

// Four E4M3 bytes to four fp16 values (bytes 0, 1 in the first dword, 2, 3
// in the second).  A code's seven magnitude bits placed at bits 7..13 of a
// half are the fp16 bits of its value times 2^-8 (a subnormal code gives a
// subnormal half), so one exact multiply by 256 per pair restores the
// value; the sign bits move to bit 15 of their halves.
__device__ __forceinline__ u32x2 e4m3x4_to_half(uint32_t w) {
  const half2_t k256 = {(_Float16)256.0f, (_Float16)256.0f};
  const half2_t a = __builtin_bit_cast(half2_t, ((w & 0x7fu) << 7) | ((w & 0x7f00u) << 15)) * k256;
  const half2_t b = __builtin_bit_cast(half2_t, ((w & 0x7f0000u) >> 9) | ((w & 0x7f000000u) >> 1)) * k256;
  const uint32_t sa = ((w & 0x80u) << 8) | ((w & 0x8000u) << 16);
  const uint32_t sb = ((w & 0x800000u) >> 8) | (w & 0x80000000u);
  return u32x2{__builtin_bit_cast(uint32_t, a) | sa, __builtin_bit_cast(uint32_t, b) | sb};
}

// fp16 hi / lo split of a (RNE both); hi + lo == a whenever a - hi is
// representable (|a| >= 1/8), else within 2^-25.
__device__ __forceinline__ void split_hl(float a, _Float16& hi, _Float16& lo) {
  hi = (_Float16)a;
  lo = (_Float16)(a - (float)hi);
}

// F8: residual values are E4M3 bytes (layout 3), else fp16 (layout 2).
// ONE: a single problem launched on its own (GOne, no plan): workgroup g
// takes the units [g U / G, (g + 1) U / G); a panel split between runs has
// its parts stored and summed after the launch by one_reduce_kernel (a
// last-arriver sum inside this kernel cost more: the stores' completion,
// the arrival's round trip and one workgroup summing up to 45 parts alone
// stood between every split panel and its output).
template <int NB, bool F8, bool ONE = false>
__global__ __launch_bounds__((MShape<NB, ONE>::MT)) void grouped_mma_kernel(const uint8_t* __restrict__ plan,
                                                          float* __restrict__ part,
                                                          uint32_t* __restrict__ counters, const GOne one) {
  using L = MLds<NB>;
  constexpr int kMT = MShape<NB, ONE>::MT, kMRP = MShape<NB, ONE>::MRP;
  constexpr int BP = 8 * NB;  // batch rows per hi (or lo) column set
  extern __shared__ float smem[];
  char* lds = reinterpret_cast<char*>(smem);
  int* bigf = reinterpret_cast<int*>(lds + L::FLAG);

  const GPlanHeader* H = reinterpret_cast<const GPlanHeader*>(plan);
  const GProblem* P = reinterpret_cast<const GProblem*>(plan + kPlanProblemsOff);
  auto PR = [&](int m) -> const GProblem& {
    if constexpr (ONE) return one.pr;
    else return P[m];
  };
  const int g = blockIdx.x, G = int(gridDim.x);
  const int B = ONE ? one.batch : H->batch;
  int ub, ue;
  Cursor cur;
  if constexpr (ONE) {
    ub = int(one_first(g, one.n_units, G));
    ue = int(one_first(g + 1, one.n_units, G));
    cur = Cursor{0, ub / one.pr.n_slices, ub % one.pr.n_slices};
  } else {
    const GChunk* CR = reinterpret_cast<const GChunk*>(plan + H->off_chunks);
    if (g >= H->n_chunks) return;
    const GChunk rc = CR[g];
    ub = rc.ub;
    ue = rc.ue;
    cur = Cursor{rc.m, rc.panel, rc.slice};
  }

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int jr = lane & 15, kb = lane >> 4;  // MFMA A row / B column, and k-block
  const int rs = jr & 3;                     // byte rotation left after the tile's 4q

  // per-lane constants: table copy offset (byte 0 of lane_base), unrotation selector
  const uint32_t lane_base = L::E12 ? uint32_t(16 * (lane & 15)) : uint32_t(8 * (lane & 31));
  const uint32_t sel_rot = 0x07060504u - 0x01010101u * uint32_t(rs);


  // x and v of the image this thread builds: pairs p = tid + kMT i of (batch
  // row b = p / 320, slice column c = p % 320); their image byte offsets (hi
  // and lo halves) are fixed per thread
  constexpr int NPAIR = (kSliceCols * BP + kMT - 1) / kMT;
  uint32_t img_hi[NPAIR], img_lo[NPAIR];
  int pb[NPAIR], pc[NPAIR];
#pragma unroll
  for (int i = 0; i < NPAIR; ++i) {
    const int p = tid + kMT * i;
    pb[i] = p / kSliceCols;
    pc[i] = p - pb[i] * kSliceCols;
    int qb, mu, h;
    slot_of_col(pc[i], qb, mu, h);
    const int bb = pb[i] < BP ? pb[i] : 0;  // pairs past the image are not built
    img_hi[i] = uint32_t(((mu * 64 + img_lane(bb + 16 * qb, mu)) * 8 + h) * 2);
    img_lo[i] = NB == 1 ? uint32_t(((mu * 64 + img_lane(bb + 8 + 16 * qb, mu)) * 8 + h) * 2)
                        : img_hi[i] + uint32_t(kImg);
  }
  // loads through buffer resources over x [B][K] and vs [n_groups * 80] (v in
  // the low half, 1 + the column's rank among its slice's salient columns in
  // the high half, 0 if it is not salient): reads past either return zero,
  // which is the padding the images need
  uint16_t xr[NPAIR];
  uint32_t vr[NPAIR];
  auto load_xv = [&](const Cursor cc) {
    const GProblem& pr = PR(cc.m);
    const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(pr.x), 0, int(2 * uint32_t(B) * uint32_t(pr.K)), kBufferWord3);
    const __amdgpu_buffer_rsrc_t vres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint32_t*>(pr.vs), 0, int(4 * uint32_t(pr.n_groups) * kGroupCols), kBufferWord3);
    const int col0 = cc.slice * kSliceCols;
#pragma unroll
    for (int i = 0; i < NPAIR; ++i) {
      const int col = col0 + pc[i];
      // a column past K would read the next batch row: send it past the buffer instead
      const uint32_t xo = (pb[i] < B && col < pr.K) ? uint32_t(2 * (pb[i] * pr.K + col)) : 0x7ffffff0u;
      xr[i] = __builtin_amdgcn_raw_buffer_load_b16(xres, int(xo), 0, 0);
      vr[i] = __builtin_amdgcn_raw_buffer_load_b32(vres, 4 * col, 0, 0);
    }
  };
  // build the B-operand images of slice cc into buffer bb (scale: 1 or 2^-16),
  // and put x at the slice's salient columns into the part's gather array
  // from part rank xbase on; returns whether any |a| of the slice is beyond
  // the fp16 range at scale 1
  uint16_t* xsal = reinterpret_cast<uint16_t*>(lds + L::XSAL);
  auto build = [&](int bb, float scale, int xbase) -> bool {
    char* img = lds + L::IMG + bb * NB * kImg;
    bool big = false;
#pragma unroll
    for (int i = 0; i < NPAIR; ++i) {
      if (tid + kMT * i < kSliceCols * BP) {
        const float a = float(__builtin_bit_cast(_Float16, uint16_t(vr[i] & 0xffffu))) *
                        float(__builtin_bit_cast(_Float16, xr[i]));
        // every lane stores (no branch): a column that is not gathered goes
        // to the lane's own dummy slot (fewer spills in the grouped kernel;
        // the one-matrix kernel at NB = 2 measured faster with the branch)
        const int rank = xbase + int(vr[i] >> 16) - 1;
        const bool keep = (vr[i] >> 16) != 0u && rank < L::XCAP;
        if constexpr (ONE && NB == 2) {
          if (keep) xsal[rank * BP + pb[i]] = xr[i];
        } else {
          *reinterpret_cast<uint16_t*>(lds + (keep ? L::XSAL + 2 * (rank * BP + pb[i]) : L::XDUMMY + 4 * lane)) = xr[i];
        }
        big |= !(__builtin_fabsf(a) < 65504.0f);
        _Float16 hi, lo;
        split_hl(a * scale, hi, lo);
        *reinterpret_cast<_Float16*>(img + img_hi[i]) = hi;
        *reinterpret_cast<_Float16*>(img + img_lo[i]) = lo;
      }
    }
    return big;
  };

  // weight bytes of unit cc, MFMA row tile q: row 16 (jr >> 2) + 4q + (jr & 3)
  // of the wave's 64-row tile, group kb of the slice
  auto w_off = [&](const Cursor cc, int q) -> uint32_t {
    const GProblem& pr = PR(cc.m);
    const int ng = pr.n_groups, n_tiles = int(pr.n_pad >> 6);
    const int grp = min(cc.slice * kSliceGroups + kb, ng - 1);
    const int tl = min(cc.panel * (kMRP / 64) + w, n_tiles - 1);
    const int row = 16 * (jr >> 2) + 4 * q + (jr & 3);
    return (uint32_t(tl * ng + grp) * kTileRows + uint32_t(row)) * kGroupPacks;
  };

  u32x4 W[4];
#pragma unroll
  for (int q = 0; q < 4; ++q)
    W[q] = __builtin_nontemporal_load(reinterpret_cast<const gu32x4*>(gptr(PR(cur.m).trits) + w_off(cur, q)));
  load_xv(cur);
  // decode tables, copy = the lane's index in its half-wave: digits 0-3 of
  // code c as fp16 at c * 256 + 8 copy, digit 4 in the T4 table.  One copy
  // of each code is computed (in the first image buffer, free until the
  // first images are built), then every copy is written from it.
  {
    uint32_t* one_copy = reinterpret_cast<uint32_t*>(lds + L::IMG);  // [243][3] words
    if (tid < kCodes) {
      const int c = tid;
      const int d0 = c % 3, r1 = c / 3, d1 = r1 % 3, r2 = r1 / 3, d2 = r2 % 3, r3 = r2 / 3, d3 = r3 % 3, d4 = r3 / 3;
      _Float16 t[4] = {(_Float16)(d0 - 1), (_Float16)(d1 - 1), (_Float16)(d2 - 1), (_Float16)(d3 - 1)};
      u32x2 m;
      __builtin_memcpy(&m, t, 8);
      const _Float16 t4[2] = {(_Float16)(d4 - 1), (_Float16)0};
      uint32_t m4;
      __builtin_memcpy(&m4, t4, 4);
      one_copy[3 * c] = m.x;
      one_copy[3 * c + 1] = m.y;
      one_copy[3 * c + 2] = m4;
    }
    __syncthreads();
    if constexpr (L::E12) {
      for (int e = tid; e < kCodes * 16; e += kMT) {
        const int c = e >> 4, cp = e & 15;
        *reinterpret_cast<u32x4*>(lds + c * kRowStride + 16 * cp) =
            u32x4{one_copy[3 * c], one_copy[3 * c + 1], one_copy[3 * c + 2], 0u};
      }
    } else {
      for (int e = tid; e < kCodes * 32; e += kMT) {
        const int c = e >> 5, cp = e & 31;
        *reinterpret_cast<u32x2*>(lds + c * kRowStride + 8 * cp) = u32x2{one_copy[3 * c], one_copy[3 * c + 1]};
        *reinterpret_cast<uint32_t*>(lds + L::T4OFF + c * 128 + 4 * cp) = one_copy[3 * c + 2];
      }
    }
    __syncthreads();  // the first images overwrite the computed copy
  }
#ifdef QTEA_DEBUG
  for (int i = tid; i < (256 - kCodes) * 64; i += kMT)  // the rows of byte values 243..255 of both tables
    reinterpret_cast<uint32_t*>(lds + kCodes * kRowStride)[i] = 0x7e007e00u;
  if (!L::E12)
    for (int i = tid; i < (256 - kCodes) * 32; i += kMT)
      reinterpret_cast<uint32_t*>(lds + L::T4OFF + kCodes * 128)[i] = 0x7e007e00u;
#endif
  // Residual hit masks: entry p * 256 + t holds, for each of the four
  // four-row groups q whose positions (2 bits each) make up the byte t,
  // 0xffff in half q when that group's salient value sits in row p.
  for (int e = tid; e < 4 * 256; e += kMT) {
    const uint32_t p = uint32_t(e) >> 8, t = uint32_t(e) & 255u;
    uint32_t m[2] = {0u, 0u};
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (((t >> (2 * q)) & 3u) == p) m[q >> 1] |= 0xffffu << (16 * (q & 1));
    *reinterpret_cast<u32x2*>(lds + L::RMASK + 8 * e) = u32x2{m[0], m[1]};
  }
  if (tid < 3) bigf[tid] = 0;
  __syncthreads();  // flags cleared and masks written before the first images and residuals

  const bool big0 = build(0, 1.0f, 0);  // the run's first unit starts a part
  if (big0) bigf[0] = 1;
  __syncthreads();

  f32x4 C[4][NB];
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) C[q][nb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  int pstart_slice = cur.slice;
  bool part_first = true;  // the open panel part began at the run's first unit

  for (int it = 0, u = ub; u < ue; ++it, ++u) {
    const GProblem& pr = PR(cur.m);
    const bool has_next = u + 1 < ue;
    Cursor nxt = cur;
    if (has_next) {
      if constexpr (ONE) {
        if (++nxt.slice == one.pr.n_slices) {
          nxt.slice = 0;
          ++nxt.panel;
        }
      } else {
        nxt = advance(cur, P);
      }
    }
    const bool pstart = (cur.slice == 0) || (u == ub);
    const bool pend = (cur.slice == pr.n_slices - 1) || !has_next;
    if (pstart) {
      pstart_slice = cur.slice;
      part_first = u == ub;
    }
    // gather rank of the next unit's first salient column in its part (for
    // the image build at the unit's end)
    const int xb_n = (!has_next || nxt.slice == 0) ? 0
                                                   : cptr(pr.spos)[nxt.slice * kSliceGroups] -
                                                         cptr(pr.spos)[pstart_slice * kSliceGroups];
    const int sb = it & 1;
    const bool big = __builtin_amdgcn_readfirstlane(bigf[it % 3]) != 0;
    if (tid == 0) bigf[(it + 2) % 3] = 0;  // flag of the unit after next
    if (big) {
      // rare: this slice's |a| reaches the fp16 range; rebuild its images
      // at 2^-16 and scale the running sums around its products
      load_xv(cur);
      build(sb, kBigScale, cptr(pr.spos)[cur.slice * kSliceGroups] - cptr(pr.spos)[pstart_slice * kSliceGroups]);
      __syncthreads();
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) C[q][nb] *= kBigScale;
    }
    load_xv(nxt);

    // next unit's weight bytes through a buffer resource over its matrix
    const GProblem& pn = PR(nxt.m);
    const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(pn.trits), 0,
        int(uint32_t(pn.n_pad >> 6) * uint32_t(pn.n_groups) * (kTileRows * kGroupPacks)), kBufferWord3);

    const char* img = lds + L::IMG + sb * NB * kImg;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      half8 Bv[5][NB];
#pragma unroll
      for (int i = 0; i < 5; ++i) {
        const int mu = i < 4 ? 4 * half + i : 8 + half;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          Bv[i][nb] = __builtin_bit_cast(half8, *(lds_u32x4*)(size_t(img + nb * kImg + (mu * 64 + img_lane(lane, mu)) * 16)));
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        // packs 8 half .. 8 half + 7 of this lane's row, unrotated
        const uint32_t U0 = __builtin_amdgcn_perm(W[q][(2 * half - q) & 3], W[q][(2 * half - q - 1) & 3], sel_rot);
        const uint32_t U1 = __builtin_amdgcn_perm(W[q][(2 * half + 1 - q) & 3], W[q][(2 * half - q) & 3], sel_rot);
        uint32_t ad[8];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t sel = 0x0C0C0004u | (uint32_t(k) << 8);
          ad[k] = __builtin_amdgcn_perm(lane_base, U0, sel);
          ad[4 + k] = __builtin_amdgcn_perm(lane_base, U1, sel);
        }
        u32x2 d03[8];
        uint32_t d4[4];
        if constexpr (L::E12) {
          u32x3 ent[8];
#pragma unroll
          for (int k = 0; k < 8; ++k) ent[k] = *(lds_u32x3*)(size_t(ad[k]));
#pragma unroll
          for (int k = 0; k < 8; ++k) d03[k] = u32x2{ent[k].x, ent[k].y};
#pragma unroll
          for (int k = 0; k < 4; ++k) d4[k] = __builtin_amdgcn_perm(ent[2 * k + 1].z, ent[2 * k].z, 0x05040100u);
        } else {
#pragma unroll
          for (int k = 0; k < 8; ++k) d03[k] = *(lds_u32x2*)(size_t(ad[k]));
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            d4[k] = lds_pair((ad[2 * k] >> 1) + L::T4OFF, (ad[2 * k + 1] >> 1) + L::T4OFF);
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const half8 A = as_half8(d03[2 * i].x, d03[2 * i].y, d03[2 * i + 1].x, d03[2 * i + 1].y);
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) C[q][nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A, Bv[i][nb], C[q][nb], 0, 0, 0);
        }
        const half8 A4 = as_half8(d4[0], d4[1], d4[2], d4[3]);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) C[q][nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A4, Bv[4][nb], C[q][nb], 0, 0, 0);
        if (half == 1) {
          // refill after the last use of the old bytes (the last unit of the
          // run reloads its own first bytes: harmless)
          const uint32_t off = has_next ? w_off(nxt, q) : 0u;
          W[q] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(wres, int(off), 0, kAuxNT));
        }
      }
    }
    if (big) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) C[q][nb] *= 65536.0f;
    }

    // the next unit's images into the other buffer

    if (pend) {
      // 1. alpha of the lane's rows: slot v of tile q is row 16 kb + 4q + v
      // of the wave's tile, sixteen consecutive rows per lane
      const int tl = cur.panel * (kMRP / 64) + w;
      const int n_tiles = int(pr.n_pad >> 6);
      const int tlc = min(tl, n_tiles - 1);
      {
        gu32x4* ap = reinterpret_cast<gu32x4*>(gptr(pr.alpha) + tlc * 64 + 16 * kb);
        const u32x4 a01 = ap[0], a23 = ap[1];
        const uint32_t aw[8] = {a01.x, a01.y, a01.z, a01.w, a23.x, a23.y, a23.z, a23.w};
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const uint32_t wd = aw[2 * q + (v >> 1)];
            const float al = float(__builtin_bit_cast(_Float16, uint16_t((v & 1) ? wd >> 16 : wd & 0xffffu)));
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) C[q][nb][v] *= al;
          }
      }
      // 2. residual of the part's salient columns: one MFMA per 32 of them.
      // Row jr of tile q is row 16 (jr >> 2) + 4q + (jr & 3) of the 64-row
      // tile: four-row group 4 (jr >> 2) + q, position jr & 3; the lane's four
      // groups (q = 0..3) are consecutive, 8 bytes of the tile's residual
      // values of a column, and 8 bits of its position word.
      const int g0 = pstart_slice * kSliceGroups;
      const int g1 = min((cur.slice + 1) * kSliceGroups, pr.n_groups);
      const int s_lo = cptr(pr.spos)[g0], s_hi = cptr(pr.spos)[g1];
      // Every load of an iteration is issued before any of its values is
      // used (indices clamped into the part's range, unused slots masked
      // afterwards).  The activations at the salient columns come from the
      // gather array when the part's salient columns fit in it (one wait on
      // memory per iteration), else from x through the salient list (two).
      gi32* Sp = gptr(pr.S);
      gu16* xp = gptr(pr.x) + uint32_t(min(jr, B - 1)) * uint32_t(pr.K);
      // the lane's four values of a column: 8 bytes (fp16) or 4 (E4M3)
      gu8* rvp = reinterpret_cast<gu8*>(gptr(pr.rval)) +
                 (uint32_t(tlc) * uint32_t(pr.nS) * 16u + 4u * uint32_t(jr >> 2)) * (F8 ? 1u : 2u);
      gu32* rip = gptr(pr.ridx) + uint32_t(tlc) * uint32_t(pr.nS);
      const uint32_t psh = 8u * uint32_t(jr >> 2);
      const uint32_t rmask = uint32_t(L::RMASK) + 2048u * uint32_t(jr & 3);  // the lane's row's mask table
      const uint32_t bmask = (jr < B && jr < BP) ? 0xffffu : 0u;
      const bool gathered = s_hi - s_lo <= L::XCAP;  // uniform
      const uint16_t* xg = xsal + min(jr, BP - 1);
      for (int s0 = s_lo; s0 < s_hi; s0 += 32) {
        u32x2 rv[8];
        uint32_t pw[8];
        uint16_t xb[8];
        if (gathered) {
#pragma unroll
          for (int h = 0; h < 8; ++h) {
            const uint32_t sc = uint32_t(min(s0 + 8 * kb + h, s_hi - 1));
            if constexpr (F8)
              rv[h].x = *reinterpret_cast<gu32*>(rvp + 16u * sc);  // converted where used
            else
              rv[h] = *reinterpret_cast<gu32x2*>(rvp + 32u * sc);
            pw[h] = rip[sc];
            xb[h] = xg[(sc - uint32_t(s_lo)) * BP];
          }
        } else {
          int col[8];
#pragma unroll
          for (int h = 0; h < 8; ++h) {
            const uint32_t sc = uint32_t(min(s0 + 8 * kb + h, s_hi - 1));
            col[h] = Sp[sc];
            if constexpr (F8)
              rv[h].x = *reinterpret_cast<gu32*>(rvp + 16u * sc);
            else
              rv[h] = *reinterpret_cast<gu32x2*>(rvp + 32u * sc);
            pw[h] = rip[sc];
          }
#pragma unroll
          for (int h = 0; h < 8; ++h) xb[h] = xp[uint32_t(col[h])];
        }
        // B: x[j][S_s] in the hi columns (j < min(B, BP)), zero elsewhere
        // and past the part's last salient column (whose clamped duplicates
        // then add nothing); A: the value of four-row group 4 (jr >> 2) + q
        // in row jr & 3 only, masked by the hit-mask entry of the column's
        // position byte, then paired by column
        _Float16 bx[8];
        u32x2 mv[8];
#pragma unroll
        for (int h = 0; h < 8; ++h) {
          const uint32_t in = (s0 + 8 * kb + h < s_hi) ? 0xffffu : 0u;
          bx[h] = __builtin_bit_cast(_Float16, uint16_t(xb[h] & (in & bmask)));
          const u32x2 m = *(lds_u32x2*)(size_t(rmask + (__builtin_amdgcn_ubfe(pw[h], psh, 8) << 3)));
          const u32x2 hv = F8 ? e4m3x4_to_half(rv[h].x) : rv[h];
          mv[h] = u32x2{hv.x & m.x, hv.y & m.y};
        }
        const half8 Bx = {bx[0], bx[1], bx[2], bx[3], bx[4], bx[5], bx[6], bx[7]};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t sel = (q & 1) ? 0x07060302u : 0x05040100u;
          uint32_t dw[4];
#pragma unroll
          for (int d = 0; d < 4; ++d)
            dw[d] = __builtin_amdgcn_perm(q < 2 ? mv[2 * d + 1].x : mv[2 * d + 1].y, q < 2 ? mv[2 * d].x : mv[2 * d].y, sel);
          C[q][0] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_half8(dw[0], dw[1], dw[2], dw[3]), Bx, C[q][0], 0, 0, 0);
        }
      }
      // 3. hi + lo, and the store: lane jr < B holds rows 16 kb + 4q + v of batch row jr
      const int64_t row0 = int64_t(cur.panel) * kMRP + int64_t(w) * 64;
      const bool owned = pstart_slice == 0 && cur.slice == pr.n_slices - 1;
      float* dst = owned ? nullptr : part + (2 * int64_t(g) + (part_first ? 0 : 1)) * int64_t(kMRP) * B;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        f32x4 yv;
        if (NB == 1) {
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            // the element goes through a scalar first: a bit cast of a vector
            // element reads element 0 whatever the index (frontend bug)
            const float cv = C[q][0][v];
            yv[v] = cv + dpp_ror8(cv);
          }
        } else {
          yv = C[q][0] + C[q][NB - 1];
        }
        const int rl = 16 * kb + 4 * q;  // row within the wave's tile
        if (jr < B) {
          if (owned) {
            if (row0 + rl < pr.N) {  // N % 4 == 0: the four rows are all in or all out
              gf32* yp = (gf32*)(pr.y + int64_t(jr) * pr.N + row0 + rl);
#pragma unroll
              for (int v = 0; v < 4; ++v) yp[v] = yv[v];
            }
          } else {
            *reinterpret_cast<f32x4*>(dst + int64_t(jr) * kMRP + w * 64 + rl) = yv;
          }
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) C[q][nb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      }
    }
    // the next unit's images into the other buffer, after the part end's
    // reads of the gather array (a next unit after a part end starts a new
    // part and refills it from rank 0)
    if (pend && has_next) __syncthreads();
    if (has_next && build(sb ^ 1, 1.0f, xb_n)) bigf[(it + 1) % 3] = 1;
    __syncthreads();  // the next unit's images are complete; this unit's are free
    cur = nxt;
  }
}

// Sums the parts of the split panels of a one-problem launch in run order
// (deterministic): one workgroup per (panel, batch row), kRedGroups groups of
// RP / 4 threads; group h sums parts ga + h, ga + h + kRedGroups, ... (four
// consecutive rows per thread, eight parts' loads in flight), and the groups'
// sums are added in group order.  Part slot k holds [batch row][RP]
// floats (RP rows per panel): slot 2k the part of run k that starts at the
// run's first unit, 2k + 1 a part starting later in the run (only the first
// run of a panel can).
constexpr int kRedGroups = 4;
template <int RP>
__global__ __launch_bounds__(RP / 4 * kRedGroups) void one_reduce_kernel(const GOne one,
                                                                        const float* __restrict__ part, int grid) {
  constexpr int kMRP = RP;
  __shared__ f32x4 gsum[kRedGroups - 1][kMRP / 4];
  const int panel = blockIdx.x, b = blockIdx.y, B = one.batch;
  const int64_t U = one.n_units, G = grid, ns = one.pr.n_slices, p0 = int64_t(panel) * ns;
  const int ga = one_owner(p0, U, G), gb = one_owner(p0 + ns - 1, U, G);
  if (ga == gb) return;  // one run holds the panel: its rows of y were written by that run
  const int odd0 = one_first(ga, U, G) < p0 ? 1 : 0;
  const int v = threadIdx.x % (kMRP / 4), h = threadIdx.x / (kMRP / 4);
  const int row = 4 * v;
  f32x4 sum = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int k0 = ga + h; k0 <= gb; k0 += 8 * kRedGroups) {
    f32x4 t[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int k = min(k0 + j * kRedGroups, gb);
      const int64_t slot = 2 * int64_t(k) + (k == ga ? odd0 : 0);
      t[j] = *reinterpret_cast<const f32x4*>(part + (slot * B + b) * kMRP + row);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (k0 + j * kRedGroups <= gb) sum += t[j];
  }
  if (h > 0) gsum[h - 1][v] = sum;
  __syncthreads();
  if (h > 0) return;
#pragma unroll
  for (int i = 0; i < kRedGroups - 1; ++i) sum += gsum[i][v];
  const int64_t r = int64_t(panel) * kMRP + row;
  if (r < one.pr.N) {  // N % 4 == 0: the four rows are all in or all out
    float* y = one.pr.y + int64_t(b) * one.pr.N + r;
#pragma unroll
    for (int i = 0; i < 4; ++i) y[i] = sum[i];
  }
}

template <int NB, bool F8, bool ONE>
hipError_t launch(const uint8_t* plan, int grid, float* part, uint32_t* counters, const GOne& one, hipStream_t st) {
  static bool done = false;
  if (!done) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&grouped_mma_kernel<NB, F8, ONE>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, MLds<NB>::BYTES);
    if (e != hipSuccess) return e;
    done = true;
  }
  hipLaunchKernelGGL((grouped_mma_kernel<NB, F8, ONE>), dim3(grid), dim3(MShape<NB, ONE>::MT), MLds<NB>::BYTES, st, plan, part,
                     counters, one);
  return hipGetLastError();
}

}  // namespace

int grouped_mma_rows_per_panel(int batch) { return batch <= 8 ? MShape<1, false>::MRP : MShape<2, false>::MRP; }
int one_mma_rows_per_panel(int batch) { return batch <= 8 ? MShape<1, true>::MRP : MShape<2, true>::MRP; }

hipError_t launch_grouped_mma(const uint8_t* plan, int grid, int batch, bool f8, float* part, hipStream_t st) {
  const GOne none{};
  if (f8) return batch <= 8 ? launch<1, true, false>(plan, grid, part, nullptr, none, st)
                            : launch<2, true, false>(plan, grid, part, nullptr, none, st);
  return batch <= 8 ? launch<1, false, false>(plan, grid, part, nullptr, none, st)
                    : launch<2, false, false>(plan, grid, part, nullptr, none, st);
}

hipError_t launch_one_mma(const GOne& one, int grid, bool f8, float* part, uint32_t* counters, hipStream_t st) {
  hipError_t e;
  if (f8) e = one.batch <= 8 ? launch<1, true, true>(nullptr, grid, part, counters, one, st)
                             : launch<2, true, true>(nullptr, grid, part, counters, one, st);
  else e = one.batch <= 8 ? launch<1, false, true>(nullptr, grid, part, counters, one, st)
                          : launch<2, false, true>(nullptr, grid, part, counters, one, st);
  if (e != hipSuccess) return e;
  bool split = false;
  const int64_t ns = one.pr.n_slices;
  for (int p = 0; p < one.pr.n_panels && !split; ++p)
    split = one_owner(p * ns, one.n_units, grid) != one_owner(p * ns + ns - 1, one.n_units, grid);
  if (!split) return hipSuccess;
  constexpr int RP = MShape<1, true>::MRP;
  static_assert(MShape<2, true>::MRP == RP, "one panel height for one-matrix launches");
  hipLaunchKernelGGL(one_reduce_kernel<RP>, dim3(one.pr.n_panels, one.batch), dim3(RP / 4 * kRedGroups), 0, st, one,
                     part, grid);
  return hipGetLastError();
}

}  // namespace qtea_grouped
