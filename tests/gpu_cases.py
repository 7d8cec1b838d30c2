"""Shared helpers of the GPU parity tests: seeded cases, the HIP path run
through the C ABI, and the tolerance check against the fp64 oracle.

Tolerance (floating point outputs): per batch vector the relative L2 error
is at most 1e-3, and per output row r the absolute error is at most
2e-3 * ||x_b||_1 * max_j |W_eff[r][j]| (W_eff includes the residual).
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

import oracle
import synth

REL_L2 = 1e-3
ROW_ABS = 2e-3


def dyadic_case(seed, N, K, B, nS):
    """Inputs whose every partial sum is exact in fp32: then the GPU result
    equals the fp64 oracle bit for bit, whatever the summation order."""
    rng = np.random.default_rng(seed)
    S = np.sort(rng.choice(K, size=nS, replace=False)).astype(np.int32) if nS else np.zeros(0, np.int32)
    return {
        "N": N, "K": K,
        "trits": rng.integers(-1, 2, size=(N, K)).astype(np.int8),
        "alpha": (2.0 ** -rng.integers(0, 6, size=N)).astype(np.float16),
        "v": rng.choice([0.5, 1.0, 1.5, 2.0], size=K).astype(np.float16),
        "S": S,
        "R": (rng.integers(-64, 65, size=(nS, N // 4)) / 64.0).astype(np.float16),
        "idx": rng.integers(0, 4, size=(nS, N // 4)).astype(np.uint8),
        "x": (rng.integers(-8, 9, size=(B, K)) / 4.0).astype(np.float16),
    }


def fine_case(seed, N, K, B):
    """Exact inputs whose a_j = v_j x_j need both fp16 halves of the
    low-batch kernel's activation split: x = k / 1024 (|k| < 2048, 11 bits),
    v in {1, 1.25, 1.5, 1.75}, alpha = 1, no salient columns.  Every product
    is a multiple of 2^-12 below 4 in magnitude, so for K <= 1000 every
    partial sum is exact in fp32 and the GPU result equals the oracle's."""
    assert K <= 1000
    rng = np.random.default_rng(seed)
    return {
        "N": N, "K": K,
        "trits": rng.integers(-1, 2, size=(N, K)).astype(np.int8),
        "alpha": np.ones(N, np.float16),
        "v": rng.choice([1.0, 1.25, 1.5, 1.75], size=K).astype(np.float16),
        "S": np.zeros(0, np.int32),
        "R": np.zeros((0, N // 4), np.float16),
        "idx": np.zeros((0, N // 4), np.uint8),
        "x": (rng.integers(-2047, 2048, size=(B, K)) / 1024.0).astype(np.float16),
    }


def synth_case(seed, N, K, B, p0=Fraction(2, 5), frac=Fraction(2, 100), layer=0, mat=0, nS=None):
    L = synth.layer_inputs(seed, layer, mat, N, K, p0=p0, frac=frac)
    if nS is not None:  # override the salient count (edge cases)
        rng = np.random.default_rng(seed + 1)
        L["S"] = np.sort(rng.choice(K, size=nS, replace=False)).astype(np.int32)
        L["R"] = (rng.standard_normal((nS, N // 4)) * 0.01).astype(np.float16)
        L["idx"] = rng.integers(0, 4, size=(nS, N // 4)).astype(np.uint8)
    L["x"] = synth.activations(seed, layer, mat, B, K)
    return L


def to_dev(a, dev="cuda"):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def gpu_pack(case, dev="cuda"):
    import paper_2609_00224_amd as q

    return q.pack_matrix(to_dev(case["trits"], dev), to_dev(case["alpha"], dev), to_dev(case["v"], dev),
                         to_dev(case["S"], dev), to_dev(case["R"], dev), to_dev(case["idx"], dev))


def gpu_unpack(pm, dev="cuda"):
    import torch

    import paper_2609_00224_amd as q

    d = pm.desc
    codes = torch.empty((d.N, d.n_packs), dtype=torch.uint8, device=dev)
    trits = torch.empty((d.N, d.K), dtype=torch.int8, device=dev)
    rows = torch.empty((max(d.n_salient, 1), d.N // 4), dtype=torch.int32, device=dev)
    q.qtea_debug_unpack(d, pm.packed, canon_codes=codes, trits=trits,
                        resid_row=rows if d.n_salient else None)
    torch.cuda.synchronize()
    return codes.cpu().numpy(), trits.cpu().numpy(), rows.cpu().numpy()[: d.n_salient]


def gpu_gemm(pm, x, dev="cuda", ws=None, use_gemv=False):
    import torch

    import paper_2609_00224_amd as q

    B = x.shape[0]
    X = to_dev(x, dev)
    Y = torch.full((B, pm.desc.N), float("nan"), dtype=torch.float32, device=dev)
    if ws is None:
        ws = q.new_workspace(pm.desc, B, dev)
    if use_gemv:
        assert B == 1
        q.qtea_gemv(pm.desc, pm.packed, X, Y, ws)
    else:
        q.qtea_gemm_lowbatch(pm.desc, pm.packed, X, B, Y, ws)
    torch.cuda.synchronize()
    return Y.cpu().numpy()


def oracle_rows(case, rows=None, codes=None, need_wmax=True, block=512):
    """fp64 oracle outputs and max |W_eff| of the given rows (default all).
    The dense rows for max |W_eff| are formed a block of rows at a time."""
    N, K = case["N"], case["K"]
    if rows is None:
        rows = np.arange(N, dtype=np.int64)
    if codes is None:
        codes = oracle.pack(case["trits"][rows])
    args = (N, K, codes, case["alpha"], case["v"], case["S"], case["R"], case["idx"])
    y = oracle.gemv(*args, case["x"], rows=rows)
    if not need_wmax:
        return y, None
    wmax = np.empty(rows.size)
    for i in range(0, rows.size, block):
        sl = slice(i, i + block)
        W = oracle.dense_rows(N, K, codes[sl], *args[3:], rows=rows[sl])
        wmax[sl] = np.abs(W).max(axis=1)
    return y, wmax


# The kernels' own precision on synthetic inputs (fp32 sums of ~1e4 terms,
# and the fp16 activation halves of the low-batch kernel) is about 1e-7
# relative; this bar, far tighter than the acceptance bound, catches a lost
# term or half that the acceptance bound would let through.
REL_L2_PRECISE = 1e-5


def assert_precise(y_gpu, y_ref, what=""):
    y_gpu = np.asarray(y_gpu, dtype=np.float64)
    for b in range(y_ref.shape[0]):
        nrm = np.linalg.norm(y_ref[b])
        if nrm > 0:
            rel = np.linalg.norm(y_gpu[b] - y_ref[b]) / nrm
            assert rel <= REL_L2_PRECISE, f"{what}: batch {b} relative L2 error {rel:.3e} above {REL_L2_PRECISE}"


def assert_close(y_gpu, y_ref, x, wmax, what=""):
    """The tolerance stated in the module docstring."""
    y_gpu = np.asarray(y_gpu, dtype=np.float64)
    assert np.all(np.isfinite(y_gpu)), f"{what}: non-finite outputs"
    xl1 = np.abs(x.astype(np.float64)).sum(axis=1)
    for b in range(y_ref.shape[0]):
        d = np.abs(y_gpu[b] - y_ref[b])
        nrm = np.linalg.norm(y_ref[b])
        if nrm > 0:
            rel = np.linalg.norm(d) / nrm
            assert rel <= REL_L2, f"{what}: batch {b} relative L2 error {rel:.3e}"
        bound = ROW_ABS * xl1[b] * wmax
        bad = np.nonzero(d > bound)[0]
        assert bad.size == 0, (f"{what}: batch {b} row bound exceeded at {bad[:5]} "
                               f"err {d[bad[:5]]} bound {bound[bad[:5]]}")


# ---------------------------------------------------------------------------
# The paper's residual storage: FP8 E4M3 values, salient column bitmap.
# ---------------------------------------------------------------------------
def e4m3_dyadic_case(seed, N, K, B, nS):
    """dyadic_case with E4M3 residual codes of exponent field 4..9: values
    (1 + m/8) 2^(e-7) are multiples of 2^-6 below 8, so every product with x
    and every partial sum stays exact in fp32 and the GPU result equals the
    oracle's bit for bit."""
    c = dyadic_case(seed, N, K, B, nS)
    rng = np.random.default_rng(seed + 7)
    shape = (nS, N // 4)
    sgn, e, m = rng.integers(0, 2, shape), rng.integers(4, 10, shape), rng.integers(0, 8, shape)
    c["R8"] = ((sgn << 7) | (e << 3) | m).astype(np.uint8)
    c["R"] = oracle.e4m3_as_half(c["R8"])
    return c


def e4m3_synth_case(seed, N, K, B, frac=Fraction(5, 100), layer=0, mat=0):
    """Synthetic inputs with E4M3 residual codes (the N(0, 0.01) draw rounded:
    mostly subnormal codes) on a fraction frac of the columns."""
    L = synth.layer_inputs(seed, layer, mat, N, K, frac=frac, resid="e4m3")
    L["R"] = oracle.e4m3_as_half(L["R8"])
    L["x"] = synth.activations(seed, layer, mat, B, K)
    return L


def gpu_pack_e4m3(case, dev="cuda"):
    import paper_2609_00224_amd as q

    return q.pack_matrix_e4m3(to_dev(case["trits"], dev), to_dev(case["alpha"], dev), to_dev(case["v"], dev),
                              to_dev(synth.column_bitmap(case["S"], case["K"]), dev), int(case["S"].size),
                              to_dev(case["R8"], dev), to_dev(case["idx"], dev))


# ---------------------------------------------------------------------------
# The paper's grouped format: 128-column groups with a scale and a bias.
# ---------------------------------------------------------------------------
def g128_dyadic_case(seed, N, K, B, nS):
    """e4m3_dyadic_case plus dyadic group scales 2^-e and biases k/64: every
    product and partial sum, the groups' sums of x included, stays exact in
    fp32."""
    c = e4m3_dyadic_case(seed, N, K, B, nS)
    rng = np.random.default_rng(seed + 11)
    ng = (K + 127) // 128
    c["alpha_g"] = (2.0 ** -rng.integers(0, 6, size=(N, ng))).astype(np.float16)
    c["beta_g"] = (rng.integers(-8, 9, size=(N, ng)) / 64.0).astype(np.float16)
    return c


def g128_synth_case(seed, N, K, B, frac=Fraction(5, 100), layer=0, mat=0):
    L = synth.layer_inputs(seed, layer, mat, N, K, frac=frac, resid="e4m3", groups=128)
    L["R"] = oracle.e4m3_as_half(L["R8"])
    L["x"] = synth.activations(seed, layer, mat, B, K)
    return L


def gpu_pack_g128(case, dev="cuda"):
    import paper_2609_00224_amd as q

    return q.pack_matrix_g128(to_dev(case["trits"], dev), to_dev(case["alpha_g"], dev), to_dev(case["beta_g"], dev),
                              to_dev(case["v"], dev), to_dev(synth.column_bitmap(case["S"], case["K"]), dev),
                              int(case["S"].size), to_dev(case["R8"], dev), to_dev(case["idx"], dev))


def oracle_rows_g128(case, rows=None, need_wmax=True, block=512):
    """fp64 oracle outputs of the grouped format and, per row, max |W_eff|
    (alpha[r][g] v_j T[r][j] plus the residual) for the tolerance."""
    N, K = case["N"], case["K"]
    if rows is None:
        rows = np.arange(N, dtype=np.int64)
    codes = oracle.pack128(case["trits"][rows])
    y = oracle.gemv128(N, K, codes, case["alpha_g"], case["beta_g"], case["v"], case["S"], case["R"],
                       case["idx"], case["x"], rows=rows)
    if not need_wmax:
        return y, None
    wmax = np.empty(rows.size)
    ng = (K + 127) // 128
    v = case["v"].astype(np.float64)
    for i in range(0, rows.size, block):
        sl = rows[i:i + block]
        a = np.repeat(case["alpha_g"][sl].astype(np.float64), 128, axis=1)[:, :K]
        W = a * v[None, :] * case["trits"][sl].astype(np.float64)
        G = N // 4
        for s, col in enumerate(case["S"]):
            hit = case["idx"][s, sl // 4] == (sl % 4)
            W[hit, col] += case["R"][s, sl[hit] // 4].astype(np.float64)
        # the bias acts like a weight beta[r][g] on every column of the group
        W = np.maximum(np.abs(W), np.repeat(np.abs(case["beta_g"][sl].astype(np.float64)), 128, axis=1)[:, :K])
        wmax[i:i + block] = W.max(axis=1)
    return y, wmax
