"""GPU parity of the offline quantizer (include/qtea_quant.h) with the fp64
oracle (oracle/quantizer.py), through the C ABI.

Bar: the integer results are bit-exact (ternary codes, salient columns and
bitmap, E4M3 residual codes and positions) and so are the fp16 results
(group scale and bias, column rescale): both sides take every decision and
rounding in fp64, from the same formulas in the same order; only summation
orders differ (about 1e-16 relative), which moves a decision only at an
exact tie.  The dequantized weights agree to 1e-12 of the weights' scale.
The Hessian agrees to 1e-13 relative and is exactly symmetric.

Sizes: several 128-column blocks with a ragged last one, rows that do not
fill the last 256-row workgroup, the paper's settings (5% salient columns,
lambda = 1, two refinement rounds) and the GPTQ special case (lambda = 0,
no refinement, no residual), a dead input channel, a Hessian that is not
positive definite, and the quantizer's output packed and multiplied by the
grouped GEMV.
"""
from __future__ import annotations

import numpy as np
import pytest

import synth
from oracle import quantizer as qz

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch

    import paper_2609_00224_amd as q

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    q.load()


def _report(what):
    print(f"[case] {what}", flush=True)


def _dev(a):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def _gpu_hessian(X):
    import torch

    import paper_2609_00224_amd as q

    H = torch.empty((X.shape[1], X.shape[1]), dtype=torch.float64, device="cuda")
    q.qtea_quant_hessian(_dev(X), H)
    torch.cuda.synchronize()
    return H


def test_hessian_matches_oracle():
    _report("quant hessian n=300 K=200")
    _, X = synth.quant_inputs(3, 4, 200, 300)
    H = _gpu_hessian(X).cpu().numpy()
    ref = qz.hessian(X)
    assert np.abs(H - ref).max() <= 1e-13 * np.abs(ref).max()
    np.testing.assert_array_equal(H, H.T)


def _check(N, K, nS, lam, iters, seed, dead=None):
    import paper_2609_00224_amd as q

    _report(f"quantize N={N} K={K} nS={nS} lambda={lam} iters={iters} dead={dead}")
    W, X = synth.quant_inputs(seed, N, K, 4 * K)
    if dead is not None:
        X[:, dead] = 0.0
    Hd = _gpu_hessian(X)
    H = qz.hessian(X)  # the oracle's own Hessian
    out = q.quantize_matrix(_dev(W), Hd, nS, lambda_decay=lam, iters=iters, want_q=True)
    ref = qz.quantize(W, H, nS, lam=lam, iters=iters)
    np.testing.assert_array_equal(out["T"].cpu().numpy(), ref["T"])
    np.testing.assert_array_equal(out["alpha"].cpu().numpy().view(np.uint16),
                                  ref["alpha"].astype(np.float16).view(np.uint16))
    np.testing.assert_array_equal(out["beta"].cpu().numpy().view(np.uint16),
                                  ref["beta"].astype(np.float16).view(np.uint16))
    np.testing.assert_array_equal(out["v"].cpu().numpy().view(np.uint16), ref["v"].astype(np.float16).view(np.uint16))
    np.testing.assert_array_equal(out["S"].cpu().numpy(), ref["S"])
    bits = out["bitmap"].cpu().numpy().view(np.uint32)
    got_cols = [j for j in range(K) if (bits[j >> 5] >> (j & 31)) & 1]
    assert got_cols == ref["S"].tolist()
    np.testing.assert_array_equal(out["R8"].cpu().numpy(), ref["rval"])
    np.testing.assert_array_equal(out["idx"].cpu().numpy(), ref["ridx"])
    Qg = out["Q"].cpu().numpy()
    assert np.abs(Qg - ref["Q"]).max() <= 1e-12 * np.abs(W).max()
    return out, W


@pytest.mark.parametrize("N,K,nS,lam,iters,seed", [
    (64, 300, 15, 1.0, 2, 1),     # paper settings, three blocks (last of 44 columns)
    (100, 129, 0, 0.0, 0, 2),     # GPTQ special case, a one-column last block, 100 rows
    (32, 40, 2, 3.0, 1, 3),       # one ragged block
    (256, 1024, 51, 1.0, 2, 4),   # eight blocks, 5% salient
])
def test_quantize_matches_oracle(N, K, nS, lam, iters, seed):
    _check(N, K, nS, lam, iters, seed)


@pytest.mark.parametrize("case", ["A", "B", "C"])
def test_salient_choice_hand_derived_eq3(case):
    """The GPU's salient column on the hand-derived Eq. 3 cases of the
    oracle's pins (each case flips under a mean over rows, diag(H) to the
    first power, or |W| in place of W^2): expected column written by hand."""
    import paper_2609_00224_amd as q

    _report(f"quantize salient hand case {case}")
    W, H, chosen = {
        "A": ([[-3.0, 2.0], [0.0, 2.0], [0.0, 2.0], [0.0, 2.0]], [[1.0, 0.0], [0.0, 1.0]], 0),
        "B": ([[2.0, 1.0], [0.0, 0.0], [0.0, 0.0], [0.0, 0.0]], [[1.0, 0.9], [0.9, 3.0]], 1),
        "C": ([[0.0, 0.0], [2.0, 0.0], [0.0, -1.0], [0.0, 0.0]], [[1.0, 1.2], [1.2, 1.5]], 0),
    }[case]
    out = q.quantize_matrix(_dev(np.array(W)), _dev(np.array(H)), 1)
    assert out["S"].cpu().tolist() == [chosen]
    assert int(out["bitmap"][0].item()) == 1 << chosen


def test_quantize_dead_channel():
    _check(48, 200, 10, 1.0, 2, 5, dead=7)


def test_quantize_not_positive_definite():
    import torch

    import paper_2609_00224_amd as q

    _report("quantize with a negative definite Hessian")
    K = 40
    W = _dev(np.zeros((8, K)))
    H = -torch.eye(K, dtype=torch.float64, device="cuda")
    with pytest.raises(q.QteaError) as e:
        q.quantize_matrix(W, H, 2)
    assert e.value.status == q.QTEA_ERR_NOT_POSITIVE


def test_quantized_matrix_through_grouped_gemv():
    """The quantizer's outputs are qtea_pack_g128's inputs: the packed matrix
    times x matches the dequantized weights times x."""
    import torch

    import paper_2609_00224_amd as q

    out, W = _check(128, 640, 32, 1.0, 2, 6)
    N, K = W.shape
    _report("quantized matrix through the grouped GEMV")
    pm = q.pack_matrix_g128(out["T"], out["alpha"], out["beta"], out["v"], out["bitmap"], 32, out["R8"], out["idx"])
    x = np.random.default_rng(7).normal(size=(1, K)).astype(np.float16)
    xd = _dev(x)
    y = torch.full((1, N), float("nan"), dtype=torch.float32, device="cuda")
    gp = q.plan_grouped([pm], [xd], [y], batch=1)
    gp.run()
    torch.cuda.synchronize()
    ref = out["Q"].cpu().numpy() @ x[0].astype(np.float64)
    got = y.cpu().numpy()[0].astype(np.float64)
    assert np.linalg.norm(got - ref) <= 1e-3 * np.linalg.norm(ref)


def test_quantize_full_size_matrix():
    """A whole Llama-3-8B-shaped O projection (4096 x 4096, 205 salient
    columns, the paper's settings), bit-exact against the oracle."""
    _check(4096, 4096, 205, 1.0, 2, 8)


def test_quantize_concurrent_streams_match_sequential():
    """Two matrices quantized at the same time on two streams from two host
    threads (the library keeps no state between calls) give exactly the
    results of one after the other."""
    from concurrent.futures import ThreadPoolExecutor

    import torch

    import paper_2609_00224_amd as q

    _report("quantize two matrices concurrently on two streams")
    cases = [synth.quant_inputs(11, 128, 520, 600), synth.quant_inputs(12, 256, 300, 600)]
    Hs = [_gpu_hessian(X) for _, X in cases]
    Ws = [_dev(W) for W, _ in cases]
    seq = [q.quantize_matrix(W, H, 20) for W, H in zip(Ws, Hs)]
    streams = [torch.cuda.Stream() for _ in cases]

    def run(i):
        with torch.cuda.stream(streams[i]):
            return q.quantize_matrix(Ws[i], Hs[i], 20, stream=streams[i])

    with ThreadPoolExecutor(max_workers=2) as pool:
        con = list(pool.map(run, range(2)))
    torch.cuda.synchronize()
    for a, b in zip(seq, con):
        for key in ("T", "alpha", "beta", "v", "S", "bitmap", "R8", "idx"):
            assert torch.equal(a[key], b[key]), key


@pytest.mark.parametrize("N,K,nS,lam,iters,seed", [
    (8, 1, 1, 1.0, 2, 21),     # one column: one block, one factor element, salient
    (4, 5, 0, 1.0, 2, 22),     # the smallest row count (one four-row group)
    (16, 70, 70, 1.0, 2, 23),  # every column salient, two factorization blocks
])
def test_quantize_degenerate_shapes(N, K, nS, lam, iters, seed):
    _check(N, K, nS, lam, iters, seed)
