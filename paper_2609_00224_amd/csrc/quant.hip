// QTEA offline quantizer for gfx950 (include/qtea_quant.h), fp64 throughout.
//
// Steps of one qtea_quantize call, all on the caller's stream:
//   0. (qtea_quant_hessian) H = (2/n) X^T X in 128 x 128 tiles.
//   1. salient columns (Eq. 3): per-column max of W^2 (atomic max on the
//      bit patterns of non-negative doubles), times diag(H)^2; each column's
//      rank counted against every other column (exact, deterministic ties);
//      one workgroup compacts the selected columns in ascending order.
//   2. damped Hessian H_d (dead columns fixed), then U with H_d^-1 = U^T U:
//      H_d = V V^T with V upper (Cholesky from the last column backwards,
//      64-column blocks: diagonal block in LDS, panel by per-row triangular
//      solves, symmetric rank-64 update of the leading block), and U = V^-1
//      (diagonal blocks inverted in LDS, then block rows from the bottom up,
//      each a product with the rows already inverted).  U is the upper
//      Cholesky factor of H_d^-1 (unique with a positive diagonal).
//   3. W transposed into the workspace (column j contiguous over rows, dead
//      columns zeroed); per 128-column block: the rows' group scale and bias,
//      then the columns one by one (one thread per row): codes, rescale
//      refinement (Eq. 4-5, its column mean summed over workgroups in a fixed
//      order by the next launch), the 1:4 residual, the decayed GPTQ error
//      (Eq. 6-9) and its update of the block's later columns; after the
//      block, the trailing columns' rank-128 update.
// Floating-point contraction is off in this file: every product and sum is
// rounded as written, in the order the method states it.  The dense products
// (Hessian, factorization, inverse, trailing update) accumulate with explicit
// fused multiply-adds: in the Hessian the products of fp32 inputs are exact
// in fp64, so fusing changes nothing; elsewhere their summation order is the
// kernel's own anyway.
#include <math.h>

#include "qtea_internal.h"
#include "qtea_quant.h"

#pragma clang fp contract(off)

namespace {

constexpr int kQG = QTEA_QUANT_GROUP;  // columns per group and per GPTQ block
constexpr int kNB = 64;                // factorization block
constexpr int kNBH = 32;               // panel columns staged per LDS pass of the trailing update
static_assert(kNB <= 64, "the diagonal block's elimination maps one column per lane of a wave");
constexpr int kCT = 64;                // threads of the row-parallel kernels (one wave)
constexpr int kColChunk = 16;          // later columns of a block updated per workgroup
constexpr int64_t kQAlign = 256;
constexpr int64_t kQMaxRows = 65536;
constexpr int64_t kQMaxCols = 65536;

inline int64_t q_up(int64_t x) { return (x + kQAlign - 1) / kQAlign * kQAlign; }
inline int64_t q_cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct QLayout {
  int64_t wt, a, u, et, score, flag, rank, dmean, scal, part, vst, total;
};

// Workspace regions (bytes from the start, 256-byte aligned).
QLayout q_layout(int64_t N, int64_t K) {
  QLayout L;
  int64_t o = 0;
  L.wt = o;    o = q_up(o + K * N * 8);                 // fp64 [K][N] current weights
  L.a = o;     o = q_up(o + K * K * 8);                 // fp64 [K][K] H_d, then V (upper)
  L.u = o;     o = q_up(o + K * K * 8);                 // fp64 [K][K] U (upper; scratch below)
  L.et = o;    o = q_up(o + int64_t(kQG) * N * 8);      // fp64 [128][N] decayed errors of a block
  L.score = o; o = q_up(o + K * 8);                     // u64/fp64 [K] max W^2, then scores
  L.flag = o;  o = q_up(o + K * 4);                     // int32 [K] selected
  L.rank = o;  o = q_up(o + K * 4);                     // int32 [K] salient rank or -1
  L.dmean = o; o = q_up(o + q_cdiv(K, kQG) * 8);        // fp64 per block: mean of diag U
  L.scal = o;  o = q_up(o + 64);                        // fp64 mean diag H; int32 status at +8
  L.part = o;  o = q_up(o + 2 * q_cdiv(N, kCT) * 2 * 8);  // fp64 [2][workgroups][2] column partials
  L.vst = o;   o = q_up(o + 2 * 8);                     // fp64 [2] previous v
  L.total = o;
  return L;
}

// fp64 -> fp16 bits, nearest with ties to even (subnormals included,
// magnitudes from 65520 up become infinity); the sign follows x.
__device__ uint16_t f64_to_f16(double x) {
  const uint16_t s = signbit(x) ? 0x8000 : 0;
  const double m = fabs(x);
  if (isnan(x)) return 0x7E00;
  if (m >= 65520.0) return s | 0x7C00;
  if (m < 0x1p-14) return s | uint16_t(rint(m * 0x1p24));  // units of 2^-24; 1024 is 2^-14
  int e;
  frexp(m, &e);
  e -= 1;  // 2^e <= m < 2^(e+1)
  const int k = int(rint(ldexp(m, 10 - e)));  // 1024..2048 (2048 carries into the exponent)
  return s | uint16_t(((e + 15) << 10) + (k - 1024));
}

__device__ double f16_to_f64(uint16_t h) {
  const int e = (h >> 10) & 31, m = h & 1023;
  double v = e == 0 ? ldexp(double(m), -24) : e == 31 ? INFINITY : ldexp(double(m + 1024), e - 25);
  return (h & 0x8000) ? -v : v;
}

// fp64 -> OCP E4M3 (FN) code: nearest finite value with ties to the even
// code, magnitudes above 448 saturate to 448; the sign bit follows x < 0.
__device__ uint8_t f64_to_e4m3(double x) {
  const uint8_t s = x < 0.0 ? 0x80 : 0;
  const double m = fabs(x);
  uint8_t c;
  if (m > 448.0) {
    c = 0x7E;
  } else if (m < 0x1p-6) {
    c = uint8_t(rint(m * 0x1p9));  // subnormal steps of 2^-9; 8 is 2^-6
  } else {
    int e;
    frexp(m, &e);
    e -= 1;                                    // -6..8
    const int k = int(rint(ldexp(m, 3 - e)));  // 8..16 (16 carries into the exponent)
    c = uint8_t(((e + 7) << 3) + (k - 8));
  }
  return s | c;
}

__device__ double e4m3_to_f64(uint8_t c) {
  const int e = (c >> 3) & 15, m = c & 7;
  const double v = e == 0 ? ldexp(double(m), -9) : ldexp(double(8 + m), e - 10);
  return (c & 0x80) ? -v : v;
}

__device__ inline int tern(double x, double thr) { return x > thr ? 1 : (x < -thr ? -1 : 0); }

// ---------------------------------------------------------------------------
// Hessian and salient columns.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void hess_kernel(const float* __restrict__ X, int64_t n, int64_t K, double scale,
                                                   double* __restrict__ H) {
  // 128 x 128 output tile, 8 x 8 per thread, calibration rows staged 16 at a time
  __shared__ double xa[16][129], xb[16][129];
  const int64_t a0 = int64_t(blockIdx.y) * 128, b0 = int64_t(blockIdx.x) * 128;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  double acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.0;
  for (int64_t t0 = 0; t0 < n; t0 += 16) {
    for (int e = threadIdx.x; e < 16 * 128; e += 256) {
      const int tt = e >> 7, c = e & 127;
      const int64_t t = t0 + tt;
      xa[tt][c] = (t < n && a0 + c < K) ? double(X[t * K + a0 + c]) : 0.0;
      xb[tt][c] = (t < n && b0 + c < K) ? double(X[t * K + b0 + c]) : 0.0;
    }
    __syncthreads();
    for (int tt = 0; tt < 16; ++tt) {
      double va[8], vb[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        va[i] = xa[tt][ty + 16 * i];
        vb[i] = xb[tt][tx + 16 * i];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = fma(va[i], vb[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t a = a0 + ty + 16 * i, b = b0 + tx + 16 * j;
      if (a < K && b < K) H[a * K + b] = scale * acc[i][j];
    }
}

__global__ void fill_f64_kernel(double* __restrict__ p, int64_t n, double v) {
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
    p[i] = v;
}

__global__ void fill_i32_kernel(int32_t* __restrict__ p, int64_t n, int32_t v) {
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
    p[i] = v;
}

// max over a run of rows of W[r][j]^2, merged by an atomic max on the bits
// (non-negative doubles order like their bit patterns)
__global__ __launch_bounds__(256) void maxsq_kernel(const double* __restrict__ W, int64_t N, int64_t K,
                                                    int64_t rows, unsigned long long* __restrict__ out) {
  const int64_t j = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (j >= K) return;
  const int64_t r0 = int64_t(blockIdx.y) * rows, r1 = r0 + rows < N ? r0 + rows : N;
  double m = 0.0;
  for (int64_t r = r0; r < r1; ++r) {
    const double w = W[r * K + j];
    const double s = w * w;
    m = s > m ? s : m;
  }
  atomicMax(out + j, static_cast<unsigned long long>(__double_as_longlong(m)));
}

// s_j = (max_i W_ij^2 * d_j) * d_j, d_j = H_jj, in place
__global__ void score_kernel(double* __restrict__ s, const double* __restrict__ H, int64_t K) {
  const int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (j >= K) return;
  const double d = H[j * K + j];
  s[j] = (s[j] * d) * d;
}

// column j is selected when fewer than n_sel columns rank before it
// (a larger score, or an equal score at a lower column)
__global__ __launch_bounds__(256) void select_kernel(const double* __restrict__ s, int64_t K, int64_t n_sel,
                                                     int32_t* __restrict__ flag) {
  __shared__ double ts[1024];
  const int64_t j = int64_t(blockIdx.x) * 256 + threadIdx.x;
  const double sj = j < K ? s[j] : 0.0;
  int64_t rank = 0;
  for (int64_t k0 = 0; k0 < K; k0 += 1024) {
    for (int e = threadIdx.x; e < 1024; e += 256) ts[e] = k0 + e < K ? s[k0 + e] : 0.0;
    __syncthreads();
    const int lim = K - k0 < 1024 ? int(K - k0) : 1024;
    for (int e = 0; e < lim; ++e) {
      const double sk = ts[e];
      rank += (sk > sj || (sk == sj && k0 + e < j)) ? 1 : 0;
    }
    __syncthreads();
  }
  if (j < K) flag[j] = rank < n_sel ? 1 : 0;
}

// one workgroup: selected columns in ascending order, each column's rank
// among them (or -1), and the bitmap
__global__ __launch_bounds__(1024) void compact_kernel(const int32_t* __restrict__ flag, int64_t K, int64_t n_sel,
                                                       int32_t* __restrict__ S, int32_t* __restrict__ rank,
                                                       uint32_t* __restrict__ bitmap) {
  __shared__ int32_t wsum[16];
  __shared__ int32_t base_s;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (threadIdx.x == 0) base_s = 0;
  __syncthreads();
  for (int64_t c0 = 0; c0 < K; c0 += 1024) {
    const int64_t j = c0 + threadIdx.x;
    const int f = j < K ? flag[j] : 0;
    const uint64_t bal = __ballot(f);
    const int pre = __popcll(bal & ((1ull << lane) - 1));
    if (lane == 0) wsum[wv] = __popcll(bal);
    if (bitmap && j < K && (lane & 31) == 0) bitmap[j >> 5] = uint32_t(bal >> lane);
    __syncthreads();
    int off = 0, tot = 0;
    for (int w = 0; w < 16; ++w) {
      off += w < wv ? wsum[w] : 0;
      tot += wsum[w];
    }
    const int pos = base_s + off + pre;
    if (j < K) {  // (pos < n_sel always holds unless a score is NaN)
      rank[j] = f && pos < n_sel ? pos : -1;
      if (f && pos < n_sel) S[pos] = int32_t(j);
    }
    __syncthreads();
    if (threadIdx.x == 0) base_s += tot;
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Damped Hessian, its reverse Cholesky factor V and U = V^-1.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void diag_mean_kernel(const double* __restrict__ H, int64_t K,
                                                        double* __restrict__ dm) {
  __shared__ double red[256];
  double s = 0.0;
  for (int64_t j = threadIdx.x; j < K; j += 256) {
    const double d = H[j * K + j];
    s += d == 0.0 ? 1.0 : d;
  }
  red[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int i = 0; i < 256; ++i) t += red[i];
    dm[0] = t / double(K);
  }
}

// upper triangle and diagonal of H_d = H (dead diagonal -> 1) + damp mean I
__global__ void damp_copy_kernel(const double* __restrict__ H, int64_t K, const double* __restrict__ dm,
                                 double damp, double* __restrict__ A) {
  const double add = damp * dm[0];
  for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < K * K; e += int64_t(gridDim.x) * blockDim.x) {
    const int64_t p = e / K, q = e % K;
    if (q < p) continue;
    double h = H[e];
    if (p == q) h = (h == 0.0 ? 1.0 : h) + add;
    A[e] = h;
  }
}

// diagonal block [c0, c0 + n) of the reverse factorization, in LDS: eliminate
// columns from the last one down, then V = column / sqrt(pivot)
__global__ __launch_bounds__(256) void chol_diag_kernel(double* __restrict__ A, int64_t K, int64_t c0, int n,
                                                        int32_t* __restrict__ status) {
  __shared__ double D[kNB][kNB + 1];
  for (int e = threadIdx.x; e < kNB * kNB; e += 256) {
    const int p = e / kNB, q = e % kNB;
    D[p][q] = (p <= q && q < n) ? A[(c0 + p) * K + c0 + q] : 0.0;
  }
  __syncthreads();
  for (int c = n - 1; c >= 0; --c) {
    double piv = D[c][c];
    if (!(piv > 0.0)) {
      if (threadIdx.x == 0) status[0] = 1;
      piv = 1.0;
    }
    // lane q = tid % 64 of the four row phases p = tid / 64, +4, ... (no
    // per-element division); D[q][c] / piv is the same factor for a column
    const int q = threadIdx.x & 63;
    if (q < c) {
      const double f = D[q][c] / piv;
      for (int p = threadIdx.x >> 6; p <= q; p += 4) D[p][q] -= D[p][c] * f;
    }
    __syncthreads();
  }
  for (int e = threadIdx.x; e < n * n; e += 256) {
    const int p = e / n, c = e % n;
    if (p <= c) {
      const double piv = D[c][c];
      A[(c0 + p) * K + c0 + c] = D[p][c] / (piv > 0.0 ? sqrt(piv) : 1.0);
    }
  }
}

// rows p < c0 of the 64 columns [c0, c0 + 64): solve x V_D^T = panel row
__global__ __launch_bounds__(256) void chol_panel_kernel(double* __restrict__ A, int64_t K, int64_t c0) {
  __shared__ double D[kNB][kNB + 1];
  for (int e = threadIdx.x; e < kNB * kNB; e += 256) {
    const int p = e / kNB, q = e % kNB;
    D[p][q] = p <= q ? A[(c0 + p) * K + c0 + q] : 0.0;
  }
  __syncthreads();
  const int64_t p = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (p >= c0) return;
  double* row = A + p * K + c0;
  double x[kNB];
#pragma unroll
  for (int c = 0; c < kNB; ++c) x[c] = row[c];
#pragma unroll
  for (int c = kNB - 1; c >= 0; --c) {
    double s = x[c];
#pragma unroll
    for (int k = c + 1; k < kNB; ++k) s -= x[k] * D[c][k];
    x[c] = s / D[c][c];
  }
#pragma unroll
  for (int c = 0; c < kNB; ++c) row[c] = x[c];
}

// upper triangle of the leading c0 x c0 block -= panel panel^T (the block's
// 64 columns): 128 x 128 tiles, 8 x 8 outputs per thread (16 LDS reads per
// 64 products), the panel staged 32 columns at a time
__global__ __launch_bounds__(256) void chol_trail_kernel(double* __restrict__ A, int64_t K, int64_t c0) {
  const int64_t tp = blockIdx.y, tq = blockIdx.x;
  if (tp > tq) return;
  __shared__ double Pp[kNBH][129], Pq[kNBH][129];  // [k][row of the tile]
  const int64_t p0 = tp * 128, q0 = tq * 128;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  double acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.0;
  for (int h = 0; h < kNB; h += kNBH) {
    for (int e = threadIdx.x; e < 128 * kNBH; e += 256) {
      const int i = e / kNBH, k = e % kNBH;
      Pp[k][i] = p0 + i < c0 ? A[(p0 + i) * K + c0 + h + k] : 0.0;
      Pq[k][i] = q0 + i < c0 ? A[(q0 + i) * K + c0 + h + k] : 0.0;
    }
    __syncthreads();
    for (int k = 0; k < kNBH; ++k) {
      double va[8], vb[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        va[i] = Pp[k][ty + 16 * i];
        vb[i] = Pq[k][tx + 16 * i];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = fma(va[i], vb[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t p = p0 + ty + 16 * i, q = q0 + tx + 16 * j;
      if (p < c0 && q < c0 && p <= q) A[p * K + q] -= acc[i][j];
    }
}

// U = V^-1 by recursive doubling: the 64 x 64 diagonal blocks (from the
// top left, the last one ragged) are inverted in LDS; then at block size
// s = 64, 128, ... each pair of neighbouring inverted blocks A = [2ps, 2ps+s)
// and C = [2ps+s, 2ps+2s) is joined by U_AC = -U_A (V_AC U_C), two batched
// products per level.  The intermediate V_AC U_C is kept transposed in U's
// lower triangle (the mirror of U_AC), which nothing else reads.
__global__ __launch_bounds__(64) void trinv_diag_kernel(const double* __restrict__ A, int64_t K,
                                                        double* __restrict__ U) {
  __shared__ double Vd[kNB][kNB + 1], Ud[kNB][kNB + 1];
  const int64_t lo = int64_t(blockIdx.x) * kNB;
  const int n = int(K - lo < kNB ? K - lo : kNB);
  for (int e = threadIdx.x; e < kNB * kNB; e += 64) {
    const int p = e / kNB, q = e % kNB;
    Vd[p][q] = (p <= q && q < n) ? A[(lo + p) * K + lo + q] : 0.0;
    Ud[p][q] = 0.0;
  }
  __syncthreads();
  const int c = threadIdx.x;  // one column of the inverse per thread
  if (c < n) {
    Ud[c][c] = 1.0 / Vd[c][c];
    for (int i = c - 1; i >= 0; --i) {
      double s = 0.0;
      for (int k = i + 1; k <= c; ++k) s += Vd[i][k] * Ud[k][c];
      Ud[i][c] = -s / Vd[i][i];
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < n * n; e += 64) {
    const int p = e / n, q = e % n;
    if (p <= q) U[(lo + p) * K + lo + q] = Ud[p][q];
  }
}

// MODE 0: T = V_AC U_C, stored as U[C][A] = T^T.  MODE 1: U_AC = -U_A T.
// Pair p = blockIdx.z; tile of 64 rows of A (blockIdx.y) x 64 columns of C
// (blockIdx.x); the triangular factor's zero half is skipped by index.
template <int MODE>
__global__ __launch_bounds__(256) void trinv_join_kernel(const double* __restrict__ A, int64_t K, int64_t s,
                                                         double* __restrict__ U) {
  __shared__ double La[16][65], Lb[16][65];
  const int64_t a0 = int64_t(blockIdx.z) * 2 * s, c0 = a0 + s;
  if (c0 >= K) return;
  const int64_t cn = K - c0 < s ? K - c0 : s;  // columns of C
  const int64_t i0 = int64_t(blockIdx.y) * 64, j0 = int64_t(blockIdx.x) * 64;
  if (i0 >= s || j0 >= cn) return;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  double acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
  // MODE 0: k over C columns [0, j0 + 64); MODE 1: k over A rows [i0, s)
  const int64_t kb = MODE == 0 ? 0 : i0;
  const int64_t ke = MODE == 0 ? (j0 + 64 < cn ? j0 + 64 : cn) : s;
  for (int64_t k0 = kb; k0 < ke; k0 += 16) {
    for (int e = threadIdx.x; e < 16 * 64; e += 256) {
      const int kk = e >> 6, m = e & 63;
      const int64_t k = k0 + kk, i = i0 + m, j = j0 + m;
      double va = 0.0, vb = 0.0;
      if (k < ke) {
        if (MODE == 0) {
          va = i < s ? A[(a0 + i) * K + c0 + k] : 0.0;                 // V_AC[i][k]
          vb = (j < cn && k <= j) ? U[(c0 + k) * K + c0 + j] : 0.0;    // U_C[k][j]
        } else {
          va = (i < s && k >= i) ? U[(a0 + i) * K + a0 + k] : 0.0;     // U_A[i][k]
          vb = j < cn ? U[(c0 + j) * K + a0 + k] : 0.0;                // T[k][j] = U[C j][A k]
        }
      }
      La[kk][m] = va;
      Lb[kk][m] = vb;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      double va[4], vb[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        va[m] = La[kk][ty + 16 * m];
        vb[m] = Lb[kk][tx + 16 * m];
      }
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int n = 0; n < 4; ++n) acc[m][n] = fma(va[m], vb[n], acc[m][n]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int64_t i = i0 + ty + 16 * m, j = j0 + tx + 16 * n;
      if (i < s && j < cn) {
        if (MODE == 0)
          U[(c0 + j) * K + a0 + i] = acc[m][n];
        else
          U[(a0 + i) * K + c0 + j] = -acc[m][n];
      }
    }
}

// mean of diag U over each 128-column block
__global__ void dmean_kernel(const double* __restrict__ U, int64_t K, double* __restrict__ dmean) {
  const int64_t g = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (g * kQG >= K) return;
  const int64_t b0 = g * kQG, b1 = b0 + kQG < K ? b0 + kQG : K;
  double s = 0.0;
  for (int64_t k = b0; k < b1; ++k) s += U[k * K + k];
  dmean[g] = s / double(b1 - b0);
}

// Wt[k][r] = W[r][k], zero for a dead column (H_kk = 0)
__global__ __launch_bounds__(256) void transpose_kernel(const double* __restrict__ W, int64_t N, int64_t K,
                                                        const double* __restrict__ H, double* __restrict__ Wt) {
  __shared__ double tile[32][33];
  const int64_t k0 = int64_t(blockIdx.x) * 32, r0 = int64_t(blockIdx.y) * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int i = ty; i < 32; i += 8) {
    const int64_t r = r0 + i, k = k0 + tx;
    tile[i][tx] = (r < N && k < K) ? W[r * K + k] : 0.0;
  }
  __syncthreads();
  for (int i = ty; i < 32; i += 8) {
    const int64_t k = k0 + i, r = r0 + tx;
    if (k < K && r < N) Wt[k * N + r] = H[k * K + k] == 0.0 ? 0.0 : tile[tx][i];
  }
}

// ---------------------------------------------------------------------------
// Column-by-column quantization.
// ---------------------------------------------------------------------------
// one row's scale and bias of block g from the current weights
__global__ __launch_bounds__(kCT) void group_params_kernel(const double* __restrict__ Wt, int64_t N, int64_t K,
                                                           int64_t G, int64_t g, uint16_t* __restrict__ alpha,
                                                           uint16_t* __restrict__ beta) {
  // the row's block values are read from memory once, eight loads in flight,
  // into this thread's LDS column; the passes below read them there
  __shared__ double wl[kQG][kCT];
  const int64_t r = int64_t(blockIdx.x) * kCT + threadIdx.x;
  if (r >= N) return;
  const int64_t b0 = g * kQG, b1 = b0 + kQG < K ? b0 + kQG : K;
  const int nb = int(b1 - b0);
  const double n = double(nb);
  {
    const double* src = Wt + b0 * N + r;
    int k = 0;
    for (; k + 8 <= nb; k += 8) {
      double v[8];
#pragma unroll
      for (int m = 0; m < 8; ++m) v[m] = src[int64_t(k + m) * N];
#pragma unroll
      for (int m = 0; m < 8; ++m) wl[k + m][threadIdx.x] = v[m];
    }
    for (; k < nb; ++k) wl[k][threadIdx.x] = src[int64_t(k) * N];
  }
  auto w = [&](int k) { return wl[k][threadIdx.x]; };
  double sw = 0.0;
  for (int k = 0; k < nb; ++k) sw += w(k);
  double be = sw / n, sa = 0.0;
  for (int k = 0; k < nb; ++k) sa += fabs(w(k) - be);
  double al = sa / n;
  for (int round = 0; round < 2; ++round) {
    if (!(al > 0.0)) break;
    const double thr = al / 2.0;
    double s1 = 0.0, s2 = 0.0, stw = 0.0;
    for (int k = 0; k < nb; ++k) {
      const double x = w(k);
      const int t = tern(x - be, thr);
      s1 += double(t);
      s2 += double(t * t);
      stw += double(t) * x;
    }
    const double det = s2 * n - s1 * s1;
    if (det > 0.0) {
      const double a = (n * stw - s1 * sw) / det;
      if (a > 0.0) {
        al = a;
        be = (s2 * sw - s1 * stw) / det;
      }
    }
  }
  uint16_t a16 = f64_to_f16(al);
  if ((a16 & 0x7FFF) == 0) a16 = 0x3C00;  // 1.0
  alpha[r * G + g] = a16;
  beta[r * G + g] = f64_to_f16(be);
}

struct ColArgs {
  double* Wt;
  const double* U;
  const double* dmean;
  const uint16_t* alpha;
  const uint16_t* beta;
  const int32_t* rank;
  double* part_in;   // [workgroups][2] partials of the previous stage
  double* part_out;  // [workgroups][2] this stage's partials
  double* vst_in;    // previous v
  double* vst_out;
  double* Et;
  int8_t* T;
  double* Q;
  uint16_t* vout;
  uint8_t* rval;
  uint8_t* ridx;
  int64_t N, K, G, g, b0, b1, j;
  int32_t nwg, iters;
  double lambda;
};

enum ColMode { kStart = 0, kRefine = 1, kFinal = 2 };

// v from the previous stage's partials: mean of |x| / alpha over non-zero
// codes (summed over workgroups in order), rounded to fp16; the previous v
// when every code is zero
__device__ double stage_v(const ColArgs& a, double* red) {
  __shared__ double vv;
  double su = 0.0, cn = 0.0;  // each thread: workgroups t, t + kCT, ... in order
  for (int w = threadIdx.x; w < a.nwg; w += kCT) {
    su += a.part_in[2 * w];
    cn += a.part_in[2 * w + 1];
  }
  red[threadIdx.x] = su;
  red[kCT + threadIdx.x] = cn;
  __syncthreads();
  for (int s = kCT / 2; s > 0; s >>= 1) {  // fixed tree order
    if (threadIdx.x < s) {
      red[threadIdx.x] += red[threadIdx.x + s];
      red[kCT + threadIdx.x] += red[kCT + threadIdx.x + s];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) vv = red[kCT] > 0.0 ? f16_to_f64(f64_to_f16(red[0] / red[kCT])) : a.vst_in[0];
  __syncthreads();
  return vv;
}

// this workgroup's sum of |x| / alpha and count over non-zero codes
__device__ void stage_partial(const ColArgs& a, double u, double c, double* red) {
  __syncthreads();
  red[threadIdx.x] = u;
  red[kCT + threadIdx.x] = c;
  __syncthreads();
  for (int s = kCT / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) {
      red[threadIdx.x] += red[threadIdx.x + s];
      red[kCT + threadIdx.x] += red[kCT + threadIdx.x + s];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    a.part_out[2 * blockIdx.x] = red[0];
    a.part_out[2 * blockIdx.x + 1] = red[kCT];
  }
}

template <int MODE>
__global__ __launch_bounds__(kCT) void col_kernel(ColArgs a) {
  __shared__ double red[2 * kCT];
  const int64_t r = int64_t(blockIdx.x) * kCT + threadIdx.x;
  const bool live = r < a.N;
  const double al = live ? f16_to_f64(a.alpha[r * a.G + a.g]) : 1.0;
  const double be = live ? f16_to_f64(a.beta[r * a.G + a.g]) : 0.0;
  const int64_t j = a.j;
  const double w = live ? a.Wt[j * a.N + r] : 0.0;
  const double x = w - be;
  if (MODE == kStart) {
    const int t = tern(x, al / 2.0);
    stage_partial(a, t != 0 ? fabs(x) / al : 0.0, t != 0 ? 1.0 : 0.0, red);
    if (blockIdx.x == 0 && threadIdx.x == 0) a.vst_out[0] = 1.0;
    return;
  }
  const double v = a.iters > 0 ? stage_v(a, red) : 1.0;
  if (MODE == kRefine) {
    const int t = tern(x, v * al / 2.0);
    stage_partial(a, t != 0 ? fabs(x) / al : 0.0, t != 0 ? 1.0 : 0.0, red);
    if (blockIdx.x == 0 && threadIdx.x == 0) a.vst_out[0] = v;
    return;
  }
  // final: codes, quantized value, residual, decayed error, in-block update;
  // workgroup (x, y) updates chunk y of the block's later columns, and only
  // the y = 0 workgroups write the column's results
  const bool primary = blockIdx.y == 0;
  const int t = tern(x, v * al / 2.0);
  double q = be + (v * al) * double(t);
  const int32_t srank = a.rank[j];
  if (srank >= 0) {
    const double res = w - q;
    const int lane = threadIdx.x & 63, g0 = lane & ~3;
    double best = fabs(__shfl(res, g0));
    int bk = 0;
#pragma unroll
    for (int k = 1; k < 4; ++k) {
      const double m = fabs(__shfl(res, g0 + k));
      if (m > best) {
        best = m;
        bk = k;
      }
    }
    const double rk = __shfl(res, g0 + bk);
    const uint8_t code = f64_to_e4m3(rk);
    if (lane - g0 == bk) q += e4m3_to_f64(code);
    if (primary && live && lane == g0) {
      a.rval[int64_t(srank) * (a.N / 4) + r / 4] = code;
      a.ridx[int64_t(srank) * (a.N / 4) + r / 4] = uint8_t(bk);
    }
  }
  const int64_t i = j - a.b0, B = a.b1 - a.b0;
  const double d = a.U[j * a.K + j];
  const double gamma = exp((-a.lambda * (d / a.dmean[a.g])) * (double(i) / double(B)));
  const double e = (gamma * (w - q)) / d;
  if (live && primary) {
    a.T[r * a.K + j] = int8_t(t);
    if (a.Q) a.Q[r * a.K + j] = q;
    a.Et[i * a.N + r] = e;
  }
  if (live) {
    // this workgroup's chunk of the block's later columns, eight at a time:
    // their loads are issued before any store
    const double* urow = a.U + j * a.K;
    double* wt = a.Wt + r;
    const int64_t kb = j + 1 + int64_t(blockIdx.y) * kColChunk;
    const int64_t ke = kb + kColChunk < a.b1 ? kb + kColChunk : a.b1;
    int64_t k = kb;
    for (; k + 8 <= ke; k += 8) {
      double wv[8], uv[8];
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        uv[m] = urow[k + m];
        wv[m] = wt[(k + m) * a.N];
      }
#pragma unroll
      for (int m = 0; m < 8; ++m) wt[(k + m) * a.N] = wv[m] - e * uv[m];
    }
    for (; k < ke; ++k) wt[k * a.N] -= e * urow[k];
  }
  if (!primary) return;
  if (blockIdx.x == 0 && threadIdx.x == 0) a.vout[j] = f64_to_f16(v);
  if (a.iters > 0 && j + 1 < a.b1) {  // the next column's first assignment (in chunk 0)
    const double x2 = live ? a.Wt[(j + 1) * a.N + r] - be : 0.0;
    const int t2 = tern(x2, al / 2.0);
    stage_partial(a, t2 != 0 ? fabs(x2) / al : 0.0, t2 != 0 ? 1.0 : 0.0, red);
    if (blockIdx.x == 0 && threadIdx.x == 0) a.vst_out[0] = 1.0;
  }
}

// Wt[k][r] -= sum_{i < B} U[b0 + i][k] Et[i][r] for k in [b1, K)
__global__ __launch_bounds__(256) void trail_gemm_kernel(double* __restrict__ Wt, const double* __restrict__ U,
                                                         const double* __restrict__ Et, int64_t N, int64_t K,
                                                         int64_t b0, int64_t B, int64_t b1) {
  __shared__ double Us[32][65], Es[32][65];
  const int64_t r0 = int64_t(blockIdx.x) * 64, k0 = b1 + int64_t(blockIdx.y) * 64;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  double acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
  for (int64_t i0 = 0; i0 < B; i0 += 32) {
    for (int e = threadIdx.x; e < 32 * 64; e += 256) {
      const int ii = e >> 6, c = e & 63;
      const bool in = i0 + ii < B;
      Us[ii][c] = (in && k0 + c < K) ? U[(b0 + i0 + ii) * K + k0 + c] : 0.0;
      Es[ii][c] = (in && r0 + c < N) ? Et[(i0 + ii) * N + r0 + c] : 0.0;
    }
    __syncthreads();
    for (int ii = 0; ii < 32; ++ii) {
      double uk[4], er[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        uk[m] = Us[ii][ty + 16 * m];
        er[m] = Es[ii][tx + 16 * m];
      }
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int n = 0; n < 4; ++n) acc[m][n] = fma(uk[m], er[n], acc[m][n]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int64_t k = k0 + ty + 16 * m, r = r0 + tx + 16 * n;
      if (k < K && r < N) Wt[k * N + r] -= acc[m][n];
    }
}

int grid1(int64_t n, int per) { return int(q_cdiv(n, per) < 65535 * 16 ? q_cdiv(n, per) : 65535 * 16); }

}  // namespace

extern "C" {

int qtea_quant_hessian(const float* X, int64_t n, int64_t K, double* H, void* stream) {
  if (!X || !H || n < 1 || K < 1 || K > kQMaxCols) return QTEA_ERR_INVALID_ARG;
  const int64_t T = q_cdiv(K, 128);
  if (T > 65535) return QTEA_ERR_INVALID_ARG;
  hipLaunchKernelGGL(hess_kernel, dim3(uint32_t(T), uint32_t(T)), dim3(256), 0, static_cast<hipStream_t>(stream), X,
                     n, K, 2.0 / double(n), H);
  return hipGetLastError() == hipSuccess ? QTEA_OK : QTEA_ERR_HIP;
}

int qtea_quant_workspace_bytes(int64_t N, int64_t K, int64_t* out_bytes) {
  if (!out_bytes || N < 4 || N % 4 != 0 || K < 1 || N > kQMaxRows || K > kQMaxCols) return QTEA_ERR_INVALID_ARG;
  *out_bytes = q_layout(N, K).total;
  return QTEA_OK;
}

int qtea_quantize(const double* W, const double* H, int64_t N, int64_t K, const qtea_quant_params* p, int8_t* T,
                  uint16_t* group_scale, uint16_t* group_bias, uint16_t* col_rescale, int32_t* salient,
                  uint32_t* salient_bitmap, uint8_t* resid_val, uint8_t* resid_idx, double* Q, void* workspace,
                  int64_t workspace_bytes, void* stream) {
  int64_t need = 0;
  if (qtea_quant_workspace_bytes(N, K, &need) != QTEA_OK) return QTEA_ERR_INVALID_ARG;
  if (!W || !H || !p || !T || !group_scale || !group_bias || !col_rescale) return QTEA_ERR_INVALID_ARG;
  if (p->n_salient < 0 || p->n_salient > K || (p->n_salient > 0 && (!salient || !resid_val || !resid_idx)))
    return QTEA_ERR_INVALID_ARG;
  if (p->iters < 0 || p->iters > QTEA_QUANT_MAX_ITERS || p->reserved != 0) return QTEA_ERR_INVALID_ARG;
  if (!(p->lambda_decay >= 0.0) || !isfinite(p->lambda_decay) || !(p->damp >= 0.0) || !isfinite(p->damp))
    return QTEA_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < need) return QTEA_ERR_WORKSPACE;
  const QLayout L = q_layout(N, K);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  double* Wt = reinterpret_cast<double*>(ws + L.wt);
  double* A = reinterpret_cast<double*>(ws + L.a);
  double* U = reinterpret_cast<double*>(ws + L.u);
  double* Et = reinterpret_cast<double*>(ws + L.et);
  double* score = reinterpret_cast<double*>(ws + L.score);
  int32_t* flag = reinterpret_cast<int32_t*>(ws + L.flag);
  int32_t* rank = reinterpret_cast<int32_t*>(ws + L.rank);
  double* dmean = reinterpret_cast<double*>(ws + L.dmean);
  double* dm = reinterpret_cast<double*>(ws + L.scal);
  int32_t* status = reinterpret_cast<int32_t*>(ws + L.scal + 8);
  double* part = reinterpret_cast<double*>(ws + L.part);
  double* vst = reinterpret_cast<double*>(ws + L.vst);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t G = q_cdiv(K, kQG);
  const int nwg = int(q_cdiv(N, kCT));
  // (salient may be NULL only when n_salient == 0: then nothing is written to it)
  int32_t* S = salient ? salient : flag;

  hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(64), 0, st, status, int64_t(1), 0);
  hipLaunchKernelGGL(fill_f64_kernel, dim3(grid1(K * K, 256)), dim3(256), 0, st, U, K * K, 0.0);
  hipLaunchKernelGGL(fill_f64_kernel, dim3(grid1(K, 256)), dim3(256), 0, st, score, K, 0.0);
  // 1. salient columns
  const int64_t rows = 256, ry = q_cdiv(N, rows);
  if (ry > 65535) return QTEA_ERR_INVALID_ARG;
  hipLaunchKernelGGL(maxsq_kernel, dim3(uint32_t(q_cdiv(K, 256)), uint32_t(ry)), dim3(256), 0, st, W, N, K, rows,
                     reinterpret_cast<unsigned long long*>(score));
  hipLaunchKernelGGL(score_kernel, dim3(uint32_t(q_cdiv(K, 256))), dim3(256), 0, st, score, H, K);
  hipLaunchKernelGGL(select_kernel, dim3(uint32_t(q_cdiv(K, 256))), dim3(256), 0, st, score, K, p->n_salient, flag);
  hipLaunchKernelGGL(compact_kernel, dim3(1), dim3(1024), 0, st, flag, K, p->n_salient, S, rank, salient_bitmap);
  // 2. H_d = V V^T, U = V^-1
  hipLaunchKernelGGL(diag_mean_kernel, dim3(1), dim3(256), 0, st, H, K, dm);
  hipLaunchKernelGGL(damp_copy_kernel, dim3(grid1(K * K, 256)), dim3(256), 0, st, H, K, dm, p->damp, A);
  for (int64_t hi = K; hi > 0; hi -= kNB) {
    const int64_t lo = hi - kNB > 0 ? hi - kNB : 0;
    hipLaunchKernelGGL(chol_diag_kernel, dim3(1), dim3(256), 0, st, A, K, lo, int(hi - lo), status);
    if (lo > 0) {
      hipLaunchKernelGGL(chol_panel_kernel, dim3(uint32_t(q_cdiv(lo, 256))), dim3(256), 0, st, A, K, lo);
      const int64_t tl = q_cdiv(lo, 128);
      hipLaunchKernelGGL(chol_trail_kernel, dim3(uint32_t(tl), uint32_t(tl)), dim3(256), 0, st, A, K, lo);
    }
  }
  const int64_t nblk = q_cdiv(K, kNB);
  hipLaunchKernelGGL(trinv_diag_kernel, dim3(uint32_t(nblk)), dim3(64), 0, st, A, K, U);
  for (int64_t sz = kNB; sz < K; sz *= 2) {
    const int64_t pairs = q_cdiv(K, 2 * sz), t = q_cdiv(sz, 64);
    if (pairs > 65535) return QTEA_ERR_INVALID_ARG;
    hipLaunchKernelGGL(trinv_join_kernel<0>, dim3(uint32_t(t), uint32_t(t), uint32_t(pairs)), dim3(256), 0, st, A, K,
                       sz, U);
    hipLaunchKernelGGL(trinv_join_kernel<1>, dim3(uint32_t(t), uint32_t(t), uint32_t(pairs)), dim3(256), 0, st, A, K,
                       sz, U);
  }
  hipLaunchKernelGGL(dmean_kernel, dim3(uint32_t(q_cdiv(G, 256))), dim3(256), 0, st, U, K, dmean);
  // 3. columns
  hipLaunchKernelGGL(transpose_kernel, dim3(uint32_t(q_cdiv(K, 32)), uint32_t(q_cdiv(N, 32))), dim3(256), 0, st, W,
                     N, K, H, Wt);
  ColArgs a{};
  a.Wt = Wt;
  a.U = U;
  a.dmean = dmean;
  a.alpha = group_scale;
  a.beta = group_bias;
  a.rank = rank;
  a.Et = Et;
  a.T = T;
  a.Q = Q;
  a.vout = col_rescale;
  a.rval = resid_val;
  a.ridx = resid_idx;
  a.N = N;
  a.K = K;
  a.G = G;
  a.nwg = nwg;
  a.iters = p->iters;
  a.lambda = p->lambda_decay;
  int s = 0;  // partials / previous-v buffer the next stage reads
  auto stage = [&](int mode) {
    a.part_in = part + s * nwg * 2;
    a.part_out = part + (s ^ 1) * nwg * 2;
    a.vst_in = vst + s;
    a.vst_out = vst + (s ^ 1);
    if (mode == kStart)
      hipLaunchKernelGGL(col_kernel<kStart>, dim3(uint32_t(nwg)), dim3(kCT), 0, st, a);
    else if (mode == kRefine)
      hipLaunchKernelGGL(col_kernel<kRefine>, dim3(uint32_t(nwg)), dim3(kCT), 0, st, a);
    else {
      const int64_t later = a.b1 - a.j - 1, ny = later > 0 ? q_cdiv(later, kColChunk) : 1;
      hipLaunchKernelGGL(col_kernel<kFinal>, dim3(uint32_t(nwg), uint32_t(ny)), dim3(kCT), 0, st, a);
    }
    s ^= 1;
  };
  for (int64_t g = 0; g < G; ++g) {
    const int64_t b0 = g * kQG, b1 = b0 + kQG < K ? b0 + kQG : K;
    hipLaunchKernelGGL(group_params_kernel, dim3(uint32_t(nwg)), dim3(kCT), 0, st, Wt, N, K, G, g, group_scale,
                       group_bias);
    a.g = g;
    a.b0 = b0;
    a.b1 = b1;
    a.j = b0;
    if (p->iters > 0) stage(kStart);
    for (int64_t j = b0; j < b1; ++j) {
      a.j = j;
      for (int it = 1; it < p->iters; ++it) stage(kRefine);
      stage(kFinal);
    }
    if (b1 < K)
      hipLaunchKernelGGL(trail_gemm_kernel, dim3(uint32_t(q_cdiv(N, 64)), uint32_t(q_cdiv(K - b1, 64))), dim3(256), 0,
                         st, Wt, U, Et, N, K, b0, b1 - b0, b1);
  }
  if (hipGetLastError() != hipSuccess) return QTEA_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return QTEA_ERR_HIP;
  int32_t host_status = 0;
  if (hipMemcpy(&host_status, status, sizeof(host_status), hipMemcpyDeviceToHost) != hipSuccess) return QTEA_ERR_HIP;
  return host_status ? QTEA_ERR_NOT_POSITIVE : QTEA_OK;
}

}  // extern "C"
