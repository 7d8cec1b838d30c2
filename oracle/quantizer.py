"""Plain fp64 CPU oracle of the QTEA offline quantizer (Section 3 of the
paper): salient-column scoring (Eq. 3), the ternary base with per-group
scale and bias (Eq. 1-2), GPTQ-style column-by-column quantization with
column-wise rescale refinement (Eq. 4-5) and error decay (Eq. 6-9), and the
1:4 semi-sparse FP8 E4M3 residual on the salient columns.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The GPU library never imports or
runs anything here, and nothing here imports the GPU library.  numpy in
fp64 throughout; numpy's Cholesky and inverse are the only library steps.

Readings of points the paper leaves open (each a choice made here):
  * A quantization group is 128 consecutive columns of one row (the format
    stores alpha and beta per row and group); the GPTQ block is the group,
    so a group's alpha, beta are estimated from the current (already
    error-updated) weights when its block starts.
  * alpha, beta of a group: start from beta = mean(w), alpha = mean|w - beta|,
    then two rounds of (assign T with threshold alpha/2, least-squares fit of
    alpha, beta to w given T), a fit kept only when it is non-degenerate and
    alpha > 0; then rounded to fp16 (stored precision).  A zero alpha (a
    constant group) becomes 1.
  * Rescale refinement of column j: T from v = 1, then `iters` rounds of
    (v = mean over T != 0 of |w - beta| / alpha, rounded to fp16; reassign T
    with threshold v alpha / 2); v stays at its previous value when T has no
    non-zero.  The quantized value is q = beta + (v alpha) T.
  * Residual: on a salient column, after its ternary assignment, each 4-row
    group keeps the row with the largest |w - q| (first on ties); its value
    is w - q rounded to E4M3 (nearest, ties to even, saturating at 448), and
    that decoded value is added to q before the GPTQ error is formed, so the
    error that propagates is the one left after the residual.
  * [H^-1]_ii in the error and the decay is the diagonal of the upper
    Cholesky factor U of the damped inverse Hessian (H^-1 = U^T U), as in
    GPTQ; the decay's mean runs over the current block's columns, i is the
    column's position in its block (0-based) and B the block's length; the
    decayed error gamma_i e_i feeds both the in-block and the trailing
    updates.
  * Damping: H + damp * mean(diag H) * I, damp = 0.01; a column with
    H_jj = 0 is dead: its weights are set to 0 and H_jj to 1 (GPTQ's rule).
  * Salient columns: the n_salient largest scores s_j (ties to the lower
    column), returned in ascending order; scores use the original weights
    and the undamped Hessian diagonal.

Pins (tests/test_quant_oracle.py): an independent sequential form of the
GPTQ update (inverse Hessian of the remaining columns by a fresh inverse at
every column, no Cholesky, no blocking), the identity-Hessian case against
a brute-force nearest-point search, an exactly representable matrix
reproduced exactly, the group fit against a library least-squares solve,
the E4M3 rounding against torch's float8_e4m3fn conversion and the format's
tie and saturation rules, the salient set against brute force over subsets
and its invariances, the paper's statement that lambda = 0 gives the GPTQ
update, the Hessian against explicit sums, and the Hessian-weighted error
below round-to-nearest.
"""
from __future__ import annotations

import numpy as np

from . import e4m3_to_double

GROUP = 128
DAMP = 0.01

_E4M3_CODES = np.arange(0x7F, dtype=np.int64)  # 0x00..0x7e: the finite non-negative codes
_E4M3_VALUES = np.array([e4m3_to_double(int(c)) for c in _E4M3_CODES])


def hessian(X) -> np.ndarray:
    """H = (2/n) X^T X for n calibration rows X [n][K] (Section 3.2)."""
    X = np.asarray(X, dtype=np.float64)
    return (2.0 / X.shape[0]) * (X.T @ X)


def fp16(x):
    """Round to the nearest fp16 value (ties to even), as fp64."""
    return np.asarray(x, dtype=np.float64).astype(np.float16).astype(np.float64)


def e4m3_round(x: float) -> int:
    """E4M3 code of the representable value nearest x (ties to the even
    code, magnitudes beyond 448 saturate to 448); the sign bit follows x."""
    m = abs(float(x))
    d = np.abs(_E4M3_VALUES - m)
    best = d.min()
    cand = _E4M3_CODES[d == best]
    code = int(cand[0]) if cand.size == 1 else int(cand[cand % 2 == 0][0])
    return code | (0x80 if x < 0 else 0)


def tern(x, thr):
    """Eq. 2: +1 above thr, -1 below -thr, else 0."""
    x = np.asarray(x, dtype=np.float64)
    return np.where(x > thr, 1, np.where(x < -thr, -1, 0)).astype(np.int8)


def salient_scores(W, H) -> np.ndarray:
    """Eq. 3: s_j = max_i W_ij^2 diag(H)_j^2."""
    W = np.asarray(W, dtype=np.float64)
    d = np.diag(np.asarray(H, dtype=np.float64))
    return (W * W).max(axis=0) * d * d


def select_salient(scores, n_salient: int) -> np.ndarray:
    """The n_salient largest scores, ties to the lower column, ascending."""
    order = sorted(range(len(scores)), key=lambda j: (-scores[j], j))
    return np.array(sorted(order[:n_salient]), dtype=np.int32)


def group_fit(w):
    """alpha, beta in fp64 before rounding, and the codes of the last
    least-squares fit (None when no fit was kept)."""
    w = np.asarray(w, dtype=np.float64)
    n = w.size
    beta = w.mean()
    alpha = np.abs(w - beta).mean()
    t_fit = None
    for _ in range(2):
        if alpha <= 0:
            break
        t = tern(w - beta, alpha / 2).astype(np.float64)
        s1, s2, sw, stw = t.sum(), (t * t).sum(), w.sum(), (t * w).sum()
        det = s2 * n - s1 * s1
        if det > 0:
            a = (n * stw - s1 * sw) / det
            if a > 0:
                alpha, beta, t_fit = a, (s2 * sw - s1 * stw) / det, t
    return alpha, beta, t_fit


def group_params(w):
    """alpha, beta (fp16-rounded, as fp64) of one row's group of weights w."""
    alpha, beta, _ = group_fit(w)
    a16, b16 = float(fp16(alpha)), float(fp16(beta))
    return (a16 if a16 > 0 else 1.0), b16


def decay(lam, d, dmean, i, B):
    """Eq. 8: gamma_i = exp(-lam * (d / dmean) * i / B)."""
    return float(np.exp(-lam * (d / dmean) * (i / B)))


def inv_hessian_factor(H, damp=DAMP):
    """Damped H (dead columns fixed), and U upper with (H_damped)^-1 = U^T U."""
    H = np.array(H, dtype=np.float64, copy=True)
    dead = np.diag(H) == 0
    H[dead, dead] = 1.0
    H += damp * np.mean(np.diag(H)) * np.eye(H.shape[0])
    U = np.linalg.cholesky(np.linalg.inv(H)).T
    return H, U, dead


def quantize_column(w, alpha, beta, iters, salient):
    """One column: ternary codes, v (fp16), q, and the residual if salient.
    Returns T, v, q, codes, idx (codes/idx None when not salient)."""
    x = w - beta
    T = tern(x, alpha / 2)
    v = 1.0
    for _ in range(iters):
        nz = T != 0
        if nz.any():
            v = float(fp16(np.mean(np.abs(x[nz]) / alpha[nz])))
        T = tern(x, v * alpha / 2)
    q = beta + (v * alpha) * T
    codes = idx = None
    if salient:
        r = w - q
        ng = w.size // 4
        codes = np.zeros(ng, np.uint8)
        idx = np.zeros(ng, np.uint8)
        for g in range(ng):
            k = int(np.argmax(np.abs(r[4 * g:4 * g + 4])))
            c = e4m3_round(r[4 * g + k])
            codes[g], idx[g] = c, k
            q[4 * g + k] += e4m3_to_double(c)
    return T, v, q, codes, idx


def quantize(W, H, n_salient, lam=1.0, iters=2, group=GROUP, damp=DAMP):
    """The whole QTEA quantization of one weight matrix W [N][K] (N % 4 == 0)
    with Hessian H [K][K].  Returns a dict: T int8 [N][K], alpha, beta fp16
    [N][n_groups] (as fp64), v fp16 [K], S int32 [n_salient], rval uint8 E4M3
    codes [n_salient][N/4], ridx uint8 [n_salient][N/4], Q (the dequantized
    weights beta + v alpha T + residual) and U."""
    W = np.array(W, dtype=np.float64, copy=True)
    N, K = W.shape
    S = select_salient(salient_scores(W, H), n_salient)
    is_sal = np.zeros(K, bool)
    is_sal[S] = True
    sal_rank = {int(j): r for r, j in enumerate(S)}
    _, U, dead = inv_hessian_factor(H, damp)
    W[:, dead] = 0.0
    G = -(-K // group)
    T = np.zeros((N, K), np.int8)
    alpha = np.zeros((N, G))
    beta = np.zeros((N, G))
    v = np.ones(K)
    Q = np.zeros((N, K))
    rval = np.zeros((len(S), N // 4), np.uint8)
    ridx = np.zeros((len(S), N // 4), np.uint8)
    for g in range(G):
        b0, b1 = g * group, min(K, (g + 1) * group)
        B = b1 - b0
        for r in range(N):
            alpha[r, g], beta[r, g] = group_params(W[r, b0:b1])
        dmean = np.mean(np.diag(U)[b0:b1])
        Err = np.zeros((N, B))
        for i in range(B):
            j = b0 + i
            w = W[:, j].copy()
            t, vj, q, codes, idx = quantize_column(w, alpha[:, g], beta[:, g], iters, is_sal[j])
            T[:, j], v[j], Q[:, j] = t, vj, q
            if codes is not None:
                rval[sal_rank[j]], ridx[sal_rank[j]] = codes, idx
            d = U[j, j]
            e = decay(lam, d, dmean, i, B) * (w - q) / d
            W[:, j + 1:b1] -= np.outer(e, U[j, j + 1:b1])
            Err[:, i] = e
        W[:, b1:] -= Err @ U[b0:b1, b1:]
    return {"T": T, "alpha": alpha, "beta": beta, "v": v, "S": S, "rval": rval, "ridx": ridx, "Q": Q, "U": U}
