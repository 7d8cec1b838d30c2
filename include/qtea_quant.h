/*
 * QTEA offline quantizer on the GPU: turns a full-precision weight matrix and
 * its calibration Hessian into the inputs of qtea_pack_g128 (ternary codes,
 * per-group scale and bias, per-column rescale, the salient columns and
 * their 1:4 FP8 E4M3 residual).  Section 3 of the paper: ternary base with
 * per-group scale and bias (Eq. 1-2), salient-column score (Eq. 3),
 * column-wise rescale refinement inside GPTQ-style column-by-column
 * quantization (Eq. 4-5), error decay (Eq. 6-9).
 *
 * Conventions as in qtea.h: plain C, device pointers, the caller owns every
 * buffer, every call returns a qtea_status code.  fp64 arithmetic throughout
 * (the integer decisions, codes and residual positions, are taken in fp64).
 *
 * Where the paper leaves a choice open, this implementation takes:
 *   - group = GPTQ block = 128 consecutive columns of a row; a group's
 *     alpha, beta are fitted to the current (error-updated) weights when its
 *     block starts: beta = mean, alpha = mean |w - beta|, then two rounds of
 *     (codes at threshold alpha/2, least-squares alpha and beta for those
 *     codes, kept when the system is non-singular and alpha > 0), rounded to
 *     fp16 (a zero alpha becomes 1);
 *   - rescale refinement of column j: codes at v = 1, then `iters` rounds of
 *     (v = mean over non-zero codes of |w - beta| / alpha, rounded to fp16,
 *     unchanged when every code is zero; codes at threshold v alpha / 2);
 *     the quantized value is beta + (v alpha) t;
 *   - on a salient column each four-row group keeps the row with the
 *     largest |w - q| (the first on ties); its residual is w - q rounded to
 *     E4M3 (nearest, ties to even, saturating at 448) and is part of the
 *     quantized value before the GPTQ error is formed;
 *   - [H^-1]_jj is the diagonal of U, the upper Cholesky factor of the
 *     damped inverse Hessian (H^-1 = U^T U); the decay's mean runs over the
 *     block's columns, i is the position in the block, B the block length;
 *   - damping H + damp mean(diag H) I; a column with H_jj = 0 is dead (its
 *     weights become 0, H_jj becomes 1 before damping);
 *   - salient columns: the n_salient largest s_j = max_i W_ij^2 diag(H)_j^2
 *     (original weights, undamped Hessian), ties to the lower column.
 */
#ifndef QTEA_QUANT_H_
#define QTEA_QUANT_H_

#include <stdint.h>

#include "qtea.h"

#ifdef __cplusplus
extern "C" {
#endif

#define QTEA_QUANT_GROUP 128
#define QTEA_QUANT_MAX_ITERS 16

typedef struct qtea_quant_params {
  int64_t n_salient;   /* salient columns, 0..K (the paper: 5% of K)        */
  double lambda_decay; /* error decay strength, >= 0 (the paper: 1; 0 = GPTQ) */
  double damp;         /* relative Hessian damping, >= 0 (0.01)             */
  int32_t iters;       /* rescale refinement rounds, 0..QTEA_QUANT_MAX_ITERS
                          (the paper: 2)                                    */
  int32_t reserved;    /* must be 0                                         */
} qtea_quant_params;

/*
 * H = (2/n) X^T X for n calibration rows (Section 3.2's approximate Hessian).
 *   X  device fp32 [n][K] row-major;  H  device fp64 [K][K], overwritten.
 * fp64 accumulation of exact fp32 products, ascending rows: H is exactly
 * symmetric.  Does not synchronize.  Errors: QTEA_ERR_INVALID_ARG (null
 * pointer, n < 1, K outside [1, 65536]), QTEA_ERR_HIP.
 */
int qtea_quant_hessian(const float* X, int64_t n, int64_t K, double* H, void* stream);

/* Workspace bytes qtea_quantize needs for an N x K matrix. */
int qtea_quant_workspace_bytes(int64_t N, int64_t K, int64_t* out_bytes);

/*
 * Quantize one weight matrix.
 *   W             device fp64 [N][K] row-major (not modified);
 *                 4 <= N <= 65536, N % 4 == 0, 1 <= K <= 65536
 *   H             device fp64 [K][K] symmetric (not modified)
 *   T             device int8 [N][K]: ternary codes
 *   group_scale   device fp16 [N][ceil(K/128)]: alpha
 *   group_bias    device fp16 [N][ceil(K/128)]: beta
 *   col_rescale   device fp16 [K]: v
 *   salient       device int32 [n_salient]: salient columns, ascending
 *   salient_bitmap device uint32 [ceil(K/32)] (or NULL): bit j%32 of word
 *                 j/32 set for a salient column
 *   resid_val     device uint8 [n_salient][N/4]: E4M3 residual codes
 *   resid_idx     device uint8 [n_salient][N/4]: row within the four-row group
 *                 (salient, resid_val and resid_idx may be NULL when
 *                 n_salient is 0)
 *   Q             device fp64 [N][K] (or NULL): the dequantized weights
 *                 beta + (v alpha) t plus the residual
 *   workspace     device, >= qtea_quant_workspace_bytes(N, K)
 * T, group_scale, group_bias, col_rescale, salient_bitmap, resid_val and
 * resid_idx are exactly the inputs of qtea_pack_g128.  Synchronizes
 * `stream` (the factorization's status is read back).  Errors:
 * QTEA_ERR_INVALID_ARG (null pointer, bad size or parameter),
 * QTEA_ERR_WORKSPACE, QTEA_ERR_NOT_POSITIVE (the damped Hessian is not
 * positive definite; outputs undefined), QTEA_ERR_HIP.
 */
int qtea_quantize(const double* W, const double* H, int64_t N, int64_t K, const qtea_quant_params* params,
                  int8_t* T, uint16_t* group_scale, uint16_t* group_bias, uint16_t* col_rescale,
                  int32_t* salient, uint32_t* salient_bitmap, uint8_t* resid_val, uint8_t* resid_idx,
                  double* Q, void* workspace, int64_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* QTEA_QUANT_H_ */
