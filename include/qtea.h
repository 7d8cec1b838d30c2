/*
 * qtea.h - C ABI of the MI355X (gfx950) compressed ternary GEMV library.
 *
 * The operation (paper: "Efficient Ternary Computation", Eq. 10 with one
 * quantization group spanning all K input columns and zero bias, plus the
 * salient residual of Eq. 11):
 *
 *   y[b][r] = alpha_r * sum_{j<K} T[r][j] * v_j * x[b][j]
 *           + sum_{s<nS} [r == 4g + idx[s][g], g = r/4] * R[s][g] * x[b][S_s]
 *
 * T[r][j] in {-1, 0, +1} are ternary codes (stored five per byte in base 3,
 * "3^5 < 2^8"), alpha_r a per-output-row fp16 scale, v_j a per-input-column
 * fp16 rescale (folded into the activations, as the paper fuses v_j x_j into
 * the table precompute), S the sorted salient input columns and, in each
 * salient column, one fp16 residual R[s][g] per group g of four consecutive
 * output rows at in-group position idx[s][g] in 0..3 (the paper's 1:4
 * semi-structured residual with a 2-bit local index).  The residual is
 * scaled by neither alpha nor v.  Weight orientation is nn.Linear's:
 * W is N (out) x K (in), y = W x.
 *
 * Conventions for every entry point:
 *   - All pointers named "device" are HIP device pointers owned by the
 *     caller.  The library never allocates or frees memory and keeps no
 *     global state; every entry point is reentrant.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Device work is
 *     enqueued on it and is stream-ordered with the caller's other work.
 *     Only qtea_pack synchronizes the stream (to return its validation
 *     result); the GEMV entry points never synchronize.
 *   - Return value: QTEA_OK (0) or a negative QTEA_ERR_* code; no exception
 *     crosses the ABI.  On an argument error nothing is enqueued.
 *   - fp16 values are passed as their IEEE binary16 bit patterns (uint16_t).
 *   - y / Y are fully overwritten (not accumulated into).  Outputs must not
 *     alias any input.
 */
#ifndef QTEA_H_
#define QTEA_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define QTEA_ABI_VERSION 9
#define QTEA_MAX_BATCH 16

enum qtea_status {
  QTEA_OK = 0,
  QTEA_ERR_INVALID_ARG = -1, /* null pointer, bad size, bad descriptor      */
  QTEA_ERR_BAD_TRIT = -2,    /* a trit outside {-1, 0, +1}                   */
  QTEA_ERR_BAD_RESIDUAL = -3,/* idx > 3, S not strictly increasing in [0,K),
                                a salient bitmap that disagrees with n_salient
                                or marks a column >= K, an E4M3 NaN value,
                                an fp16 residual value that is not finite */
  QTEA_ERR_BATCH = -4,       /* batch outside [1, QTEA_MAX_BATCH]            */
  QTEA_ERR_WORKSPACE = -5,   /* workspace or packed buffer too small         */
  QTEA_ERR_HIP = -6,         /* a HIP runtime call or kernel launch failed   */
  QTEA_ERR_NOT_POSITIVE = -7,/* a Hessian that is not positive definite
                                (qtea_quantize, include/qtea_quant.h)      */
};

/*
 * Host-side description of one packed matrix.  Filled by qtea_pack, owned
 * by the caller, read by the other entry points.  The packed device buffer
 * it describes is opaque: its tiling is private to the library and may
 * change between library versions (`layout` records which one).
 */
typedef struct qtea_desc {
  uint32_t magic;       /* QTEA_DESC_MAGIC when valid                        */
  uint32_t layout;      /* device layout version: 2 = fp16 residual values,
                           3 = FP8 E4M3 residual values (qtea_pack_e4m3),
                           4 = 128-column groups (qtea_pack_g128)          */
  int64_t N, K;         /* output rows, input columns                        */
  int64_t n_salient;    /* |S|                                               */
  int64_t n_packs;      /* one-byte packs per row: ceil(K / 5), or 26 per
                           128-column group in layout 4                      */
  int64_t n_groups;     /* ceil(n_packs / 16) sixteen-pack groups; layout 4:
                           two per 128-column group, 13 packs each          */
  int64_t n_pad;        /* N rounded up to a multiple of 64                  */
  int64_t bytes_total;  /* size of the packed buffer in bytes                */
  int64_t off_trits, off_alpha, off_v, off_salient, off_spos, off_rval, off_ridx;
} qtea_desc;

#define QTEA_DESC_MAGIC 0x51544541u /* "QTEA" */

/* Text for a status code (static storage; never NULL). */
const char* qtea_status_string(int status);

/* Library ABI version (QTEA_ABI_VERSION of the built library). */
int qtea_abi_version(void);

/*
 * Size of the packed device buffer for an N x K matrix with n_salient
 * salient columns.  Requires N >= 4, N % 4 == 0 (four-row residual groups),
 * K >= 1, 0 <= n_salient <= K.  Writes *out_bytes.
 */
int qtea_packed_bytes(int64_t N, int64_t K, int64_t n_salient, int64_t* out_bytes);

/*
 * Pack dense inputs into the device layout (paper: five trits per byte in
 * base 3; per-row scale; per-column rescale; salient residual with one value
 * and a 2-bit position per four entries).  Offline: synchronizes `stream`.
 *
 *   trits       device int8  [N][K], row-major, values in {-1, 0, +1}
 *   row_scale   device fp16  [N]       alpha
 *   col_rescale device fp16  [K]       v
 *   salient     device int32 [n_salient], strictly increasing, in [0, K)
 *   resid_val   device fp16  [n_salient][N/4]   R[s][g], finite
 *   resid_idx   device uint8 [n_salient][N/4]   position of R[s][g] in rows 4g..4g+3
 *   packed      device buffer of packed_bytes >= qtea_packed_bytes(...)
 *   out_desc    host; filled on success
 *
 * Byte code of columns 5p..5p+4 of a row: sum_i (T[r][5p+i] + 1) * 3^i, with
 * the zero trit in place of columns >= K.  The salient/residual pointers may
 * be NULL when n_salient == 0.
 * Errors: QTEA_ERR_INVALID_ARG, QTEA_ERR_WORKSPACE (packed buffer too small),
 * QTEA_ERR_BAD_TRIT, QTEA_ERR_BAD_RESIDUAL (checked on the device; *out_desc
 * is left invalid), QTEA_ERR_HIP.
 */
int qtea_pack(const int8_t* trits, int64_t N, int64_t K, const uint16_t* row_scale,
              const uint16_t* col_rescale, const int32_t* salient, int64_t n_salient,
              const uint16_t* resid_val, const uint8_t* resid_idx, void* packed,
              int64_t packed_bytes, qtea_desc* out_desc, void* stream);

/*
 * The paper's storage of the salient residual (the "compact
 * semi-structured format" of its GEMV section, at its evaluation setting of
 * FP8 E4M3 values in 5% of the columns): a bitmap over the input columns
 * marks the salient ones, and every four-entry group of a salient column
 * holds one one-byte E4M3 value with its 2-bit position.  Same operation as
 * qtea_pack with R[s][g] = the E4M3 value (exact in fp16 and fp32; every
 * GEMV entry point accepts either layout).
 *
 *   salient_bitmap device uint32 [ceil(K/32)]: bit (j % 32) of word j / 32
 *                  set when column j is salient; bits at or past K clear;
 *                  exactly n_salient bits set.  S is the set bits ascending.
 *   resid_val      device uint8 [n_salient][N/4]: E4M3 codes (sign, four
 *                  exponent bits of bias 7, three mantissa bits; the two
 *                  NaN codes 0x7f, 0xff are rejected)
 *   packed         device buffer of packed_bytes >= qtea_packed_bytes_e4m3(...)
 * Other arguments, errors and synchronization as qtea_pack.
 */
int qtea_packed_bytes_e4m3(int64_t N, int64_t K, int64_t n_salient, int64_t* out_bytes);
int qtea_pack_e4m3(const int8_t* trits, int64_t N, int64_t K, const uint16_t* row_scale,
                   const uint16_t* col_rescale, const uint32_t* salient_bitmap, int64_t n_salient,
                   const uint8_t* resid_val, const uint8_t* resid_idx, void* packed, int64_t packed_bytes,
                   qtea_desc* out_desc, void* stream);

/*
 * The paper's full format (Eq. 10 with its group size of 128, and its
 * storage): for row r and the g-th group of 128 input columns a scale
 * alpha[r][g] and a bias beta[r][g],
 *
 *   y[b][r] = sum_g ( alpha[r][g] * sum_{j in g} T[r][j] * v_j * x[b][j]
 *                   + beta[r][g]  * sum_{j in g} x[b][j] )  + the residual;
 *
 * each group's 128 trits packed into 26 bytes (25 of five columns, the last
 * of three columns and two zero trits; 1.625 bits per weight), the residual
 * stored as in qtea_pack_e4m3.
 *
 *   group_scale, group_bias  device fp16 [N][ceil(K/128)]
 *   other arguments          as qtea_pack_e4m3
 *   packed                   >= qtea_packed_bytes_g128(...)
 *
 * A matrix in this layout runs through the batch-1 table kernel (the per-
 * group scale and bias are applied as each group's table sums are added):
 * at batch B, qtea_gemm_lowbatch and the grouped entry points run the B
 * activation rows one after another (B batch-1 launches, or B batch-1
 * problems in one grouped launch), so its weights are streamed once per
 * row.  qtea_debug_unpack returns its codes as [N][26 ceil(K/128)], group
 * after group.
 */
int qtea_packed_bytes_g128(int64_t N, int64_t K, int64_t n_salient, int64_t* out_bytes);
int qtea_pack_g128(const int8_t* trits, int64_t N, int64_t K, const uint16_t* group_scale,
                   const uint16_t* group_bias, const uint16_t* col_rescale, const uint32_t* salient_bitmap,
                   int64_t n_salient, const uint8_t* resid_val, const uint8_t* resid_idx, void* packed,
                   int64_t packed_bytes, qtea_desc* out_desc, void* stream);

/*
 * Workspace bytes that qtea_gemv (batch = 1) / qtea_gemm_lowbatch need for
 * this matrix at this batch size on the current device.  A call splits the
 * matrix's output panels (512 rows) and its K range
 * into work units over one launch; a panel whose units fall to more than
 * one workgroup is summed from their partial rows in a fixed order, at
 * batch 1 by the last of them to arrive, at batch 2..16 by a second small
 * kernel on the same stream.  The workspace holds one arrival counter per
 * panel and two slots of partial rows per workgroup.  It must be zero-filled before its first use
 * (qtea_workspace_init or any zero fill); every call that runs to
 * completion leaves the counters at zero again, so one workspace serves any
 * sequence of stream-ordered calls.  Calls that may overlap in time must
 * not share a workspace.  Errors: QTEA_ERR_INVALID_ARG, QTEA_ERR_BATCH
 * (batch outside 1..16), QTEA_ERR_HIP.
 */
int qtea_workspace_bytes(const qtea_desc* desc, int batch, int64_t* out_bytes);

/* Enqueue a zero fill of `bytes` bytes of `workspace` (a kernel, not a
 * memset node, so it is safe inside captured graphs). */
int qtea_workspace_init(void* workspace, int64_t bytes, void* stream);

/*
 * y = W x for one activation vector (batch 1).
 *   packed      device buffer filled by qtea_pack, qtea_pack_e4m3 or
 *               qtea_pack_g128 for *desc
 *   x           device fp16 [K]
 *   y           device fp32 [N]
 *   workspace   device, >= qtea_workspace_bytes(desc, 1), see above
 * One launch, no host work beyond argument checks (graph-capturable).  fp32
 * accumulation; results are run-to-run deterministic (partial sums are
 * added in a fixed order).  Identical to qtea_gemm_lowbatch with batch 1.
 * Errors: QTEA_ERR_INVALID_ARG (null pointer, invalid descriptor, a matrix
 * whose packed codes or residual values take 2 GiB or more: the kernels
 * use 32-bit offsets), QTEA_ERR_WORKSPACE (workspace smaller than
 * qtea_workspace_bytes), QTEA_ERR_HIP (launch failure).
 */
int qtea_gemv(const qtea_desc* desc, const void* packed, const uint16_t* x, float* y,
              void* workspace, int64_t workspace_bytes, void* stream);

/*
 * Y = X W^T for 1 <= batch <= QTEA_MAX_BATCH activation rows (low-batch
 * decode: one token per row).
 *   X  device fp16 [batch][K] row-major;  Y  device fp32 [batch][N] row-major.
 * Batch 1 runs the table-lookup kernel, batch 2..16 the matrix-core kernel
 * (fp16 products of the exact ternary codes with the activations split
 * into two fp16 halves, fp32 accumulation).  Errors as qtea_gemv plus
 * QTEA_ERR_BATCH.
 */
int qtea_gemm_lowbatch(const qtea_desc* desc, const void* packed, const uint16_t* X, int batch,
                       float* Y, void* workspace, int64_t workspace_bytes, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * operation as qtea_gemm_lowbatch, through the same kernels, without a
 * workspace argument.  The library keeps its own fixed workspace of
 * QTEA_NOALLOC_SCRATCH_BYTES per GPU, a device array held until the process
 * ends; this call allocates nothing (no hipMalloc, no hipFree).  Its first
 * call on a device enqueues a zero fill of the array's counter words on
 * `stream`; every call that completes leaves them at zero.  Every call on
 * one GPU uses that GPU's array: calls that may overlap in time on one GPU
 * (other streams, other host threads) race and must not be made.
 * Errors as qtea_gemm_lowbatch, with QTEA_ERR_WORKSPACE for a call whose
 * workspace (qtea_workspace_bytes) would not fit the array: on a device of
 * up to 256 CUs every batch fits a matrix of up to 16384 x 512 rows (one
 * arrival counter per 512-row panel).
 */
#define QTEA_NOALLOC_SCRATCH_BYTES (16 * 1048576 + 65536)
int qtea_gemm_lowbatch_noalloc(const qtea_desc* desc, const void* packed, const uint16_t* X, int batch,
                               float* Y, void* stream);

/*
 * Measurement support: stream `bytes` (a multiple of 16) of a device buffer
 * from HBM with the same 16-byte non-temporal loads the GEMV kernels use,
 * and nothing else: each workgroup reads one contiguous chunk of
 * QTEA_READ_CEILING_CHUNK bytes (the last one may be shorter) and stores its
 * fold to sink[chunk] (device uint32 [ceil(bytes / QTEA_READ_CEILING_CHUNK)],
 * caller-owned; the fold is the XOR over the chunk's 16-byte words of the
 * 32-bit sum of their four little-endian u32 lanes, so the reads are not
 * removed and can be checked).  The rate of this kernel on a buffer far
 * beyond the last-level cache, held under load, is the streaming-read
 * ceiling the GEMV rates are compared with.  Does not synchronize.
 * Errors: QTEA_ERR_INVALID_ARG (null pointer, size not a positive multiple
 * of 16, buffer not 16-byte aligned), QTEA_ERR_HIP.
 */
#define QTEA_READ_CEILING_CHUNK 65536
int qtea_read_ceiling(const void* buf, int64_t bytes, uint32_t* sink, void* stream);

/*
 * Test support: read the packed buffer back into plain form, bit for bit.
 *   canon_codes device uint8 [N][n_packs]  canonical byte codes (or NULL)
 *   trits       device int8  [N][K]        decoded trits          (or NULL)
 *   resid_row   device int32 [n_salient][N/4] output row 4g + idx (or NULL)
 * Does not synchronize.
 */
int qtea_debug_unpack(const qtea_desc* desc, const void* packed, uint8_t* canon_codes,
                      int8_t* trits, int32_t* resid_row, void* stream);

/*
 * Grouped GEMV: Y_m = X_m W_m^T for a list of n_problems independent problems
 * at one batch size (each W_m packed by qtea_pack or, all of them,
 * qtea_pack_e4m3; the same operation as qtea_gemm_lowbatch applied to every
 * problem) in one persistent launch.  Matrices packed by qtea_pack_g128 run
 * here as one batch-1 problem per activation row (the plan and its info
 * count those problems, at batch 1).  The problems' packed bytes are
 * streamed back to back: a workgroup already loads the next problem's
 * weights while it finishes the current one.  No problem may read another
 * problem's output (all activations must be ready when the launch starts);
 * for a chain of dependent products call qtea_gemv per product instead.
 *
 * Usage: qtea_grouped_plan once (offline, synchronizes `stream`), then
 * qtea_grouped_gemv any number of times (graph-capturable, no host work).
 * The plan binds the device pointers given to qtea_grouped_plan; change
 * any of them and plan again.
 */
typedef struct qtea_grouped_info {
  uint32_t magic;          /* set by qtea_grouped_plan                    */
  int32_t n_problems;
  int32_t batch;           /* activation rows per problem (1..16)         */
  int32_t grid;            /* workgroups of the launch (batch 1: two per
                              CU, table lookups; batch 2..16: one per CU,
                              matrix cores)                               */
  int32_t rows_per_panel;  /* output rows of one work unit               */
  int32_t max_parts;       /* chunks sharing one panel, at most          */
  int32_t n_chunks;        /* chunks of work units (scheduling grain)    */
  int32_t n_split_panels;  /* panels whose parts are summed by a second launch */
  int32_t layout;          /* layout of every problem (2, 3 or 4)       */
  int32_t reserved;
  int64_t n_units;
  int64_t plan_bytes;      /* device plan buffer size                    */
  int64_t workspace_bytes; /* workspace needed by qtea_grouped_gemv      */
} qtea_grouped_info;

/* Size of the device plan buffer for n_problems problems at any batch size
 * on the current device (room for QTEA_MAX_BATCH rows per problem of the
 * grouped format).  QTEA_ERR_INVALID_ARG for n_problems outside 1..2^24. */
int qtea_grouped_plan_bytes(int n_problems, int64_t* out_bytes);

/*
 * Build the plan of a grouped GEMV.
 *   descs[m], packed[m]  host array of descriptors / host array of device
 *                        pointers to the packed buffers (qtea_pack)
 *   x[m]                 host array of device pointers, fp16 [batch][K_m]
 *   y[m]                 host array of device pointers, fp32 [batch][N_m]
 *   batch                activation rows per problem, 1..QTEA_MAX_BATCH
 *                        (QTEA_ERR_BATCH otherwise)
 *   plan                 device buffer, >= qtea_grouped_plan_bytes(n_problems)
 *   info                 host, filled on success
 * Errors: QTEA_ERR_INVALID_ARG (also for a matrix whose packed codes or
 * residual values take 2 GiB or more: the kernel uses 32-bit offsets; and
 * for a list that mixes the two residual layouts),
 * QTEA_ERR_BATCH, QTEA_ERR_WORKSPACE (plan buffer too small), QTEA_ERR_HIP.
 */
int qtea_grouped_plan(const qtea_desc* descs, const void* const* packed, const uint16_t* const* x,
                      float* const* y, int n_problems, int batch, void* plan, int64_t plan_bytes,
                      qtea_grouped_info* info, void* stream);

/*
 * Run a planned grouped GEMV: one persistent launch, followed by a small
 * second launch that sums the parts of split panels (when the plan has
 * any, info->n_split_panels).  `workspace` (>= info->workspace_bytes) holds
 * the chunk queue's counters and error flags (its first 256 bytes) and the
 * partial rows of split panels.  Zero-fill it once before the first call;
 * every call leaves the counters at zero (see qtea_grouped_status for the
 * error flags).  Calls that may overlap in time must not share a workspace.  fp32 accumulation, run-to-run
 * deterministic (parts are summed in a fixed order).  `info` must be the
 * record qtea_grouped_plan filled for this `plan` buffer: the launch shape
 * and the position of the plan's split records are taken from it.  Errors:
 * QTEA_ERR_INVALID_ARG (an info that no plan could have filled),
 * QTEA_ERR_WORKSPACE (workspace smaller than info->workspace_bytes).
 */
int qtea_grouped_gemv(const qtea_grouped_info* info, const void* plan, void* workspace,
                      int64_t workspace_bytes, void* stream);

/*
 * Error flags a grouped workspace has collected, read into *flags (host);
 * synchronizes `stream` (after the calls whose outcome is wanted).  The
 * batch-1 launch hands out chunks from a counter in the workspace and
 * checks its own accounting:
 *   QTEA_QUEUE_STALE  a take found the counter past the plan's count: the
 *                     counter did not start at zero (a workspace that was
 *                     not zero-filled, or one left by a call that did not
 *                     complete); that take yields no chunk, so some outputs
 *                     of the call were not written
 *   QTEA_QUEUE_COUNT  the chunks the launch ran (a hashed tag per chunk,
 *                     summed at each workgroup's exit) or its takes did not
 *                     add up to the plan's: queue words left over from an
 *                     earlier call made it skip or repeat chunks
 * Either flag means the outputs of the flagged call are not to be used.
 * The last workgroup of every launch leaves the counters at zero, so the
 * next call starts clean; the flags stay set until the workspace is
 * zero-filled again (qtea_workspace_init).  Errors: QTEA_ERR_INVALID_ARG
 * (null pointer), QTEA_ERR_HIP.
 */
#define QTEA_QUEUE_STALE 1u
#define QTEA_QUEUE_COUNT 2u
int qtea_grouped_status(const void* workspace, uint32_t* flags, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* QTEA_H_ */
