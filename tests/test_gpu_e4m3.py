"""GPU parity of the paper's residual storage (one FP8 E4M3 value and a
2-bit position per four entries of a salient column, the salient columns
marked by a column bitmap): packing, the per-matrix GEMV at batch 1..16 and
the grouped GEMV at batch 1..16 against the fp64 oracle (which decodes the
E4M3 codes from the format's definition), bit for bit on dyadic inputs and
within the tolerance of gpu_cases on synthetic ones (mostly subnormal
codes); the same values stored as fp16 give bit-identical outputs; invalid
inputs are rejected."""
from __future__ import annotations

from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_cases import (assert_close, assert_precise, e4m3_dyadic_case, e4m3_synth_case, gpu_gemm,
                             gpu_pack, gpu_pack_e4m3, gpu_unpack, oracle_rows, to_dev)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch

    import paper_2609_00224_amd as q

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    q.load()


def _report(what):
    print(f"[case] {what}", flush=True)


def _grouped(mats, cases, B):
    import torch

    import paper_2609_00224_amd as q

    xs = [to_dev(c["x"]) for c in cases]
    ys = [torch.full((B, c["N"]), float("nan"), dtype=torch.float32, device="cuda") for c in cases]
    gp = q.plan_grouped(mats, xs, ys, batch=B)
    gp.run()
    torch.cuda.synchronize()
    return [y.cpu().numpy() for y in ys], gp


SHAPES = [(256, 1000, 37), (4160, 640, 100), (64, 5, 1), (1024, 14336, 300), (192, 81, 0)]


def test_e4m3_layout_decode_bit_exact():
    import paper_2609_00224_amd as q

    for N, K, nS in SHAPES:
        _report(f"decode N={N} K={K} nS={nS}")
        c = e4m3_dyadic_case(3, N, K, 1, nS)
        pm = gpu_pack_e4m3(c)
        assert pm.desc.layout == q.QTEA_LAYOUT_E4M3
        assert pm.desc.bytes_total == q.qtea_packed_bytes_e4m3(N, K, nS)
        # one byte less per residual value (regions are 256-byte aligned)
        assert q.qtea_packed_bytes_e4m3(N, K, nS) <= q.qtea_packed_bytes(N, K, nS) - (N // 4) * nS // 256 * 256
        codes, trits, rows = gpu_unpack(pm)
        assert np.array_equal(codes, oracle.pack(c["trits"]))
        assert np.array_equal(trits, c["trits"])
        if nS:
            assert np.array_equal(rows, oracle.resid_rows(c["idx"], N))


@pytest.mark.parametrize("B", [1, 2, 4, 5, 8, 16])
def test_e4m3_per_matrix_dyadic_exact(B):
    for N, K, nS in SHAPES[:4]:
        _report(f"per-matrix dyadic B={B} N={N} K={K} nS={nS}")
        c = e4m3_dyadic_case(11 + B, N, K, B, nS)
        y = gpu_gemm(gpu_pack_e4m3(c), c["x"])
        ref, _ = oracle_rows(c, need_wmax=False)
        assert np.array_equal(y.astype(np.float64), ref), (B, N, K, nS)


@pytest.mark.parametrize("B", [1, 3, 8, 9, 16])
def test_e4m3_grouped_dyadic_exact(B):
    _report(f"grouped dyadic B={B}")
    cases = [e4m3_dyadic_case(40 + i, N, K, B, nS) for i, (N, K, nS) in enumerate(SHAPES)]
    ys, _ = _grouped([gpu_pack_e4m3(c) for c in cases], cases, B)
    for c, y in zip(cases, ys):
        ref, _ = oracle_rows(c, need_wmax=False)
        assert np.array_equal(y.astype(np.float64), ref), (B, c["N"], c["K"])


@pytest.mark.parametrize("B", [1, 4, 16])
def test_e4m3_synth_tolerance(B):
    shapes = [(6144, 4096), (4096, 14336), (1040, 999)]
    cases = [e4m3_synth_case(5, N, K, B, mat=i) for i, (N, K) in enumerate(shapes)]
    mats = [gpu_pack_e4m3(c) for c in cases]
    for c, pm in zip(cases, mats):
        _report(f"per-matrix synth B={B} N={c['N']} K={c['K']}")
        ref, wmax = oracle_rows(c)
        y = gpu_gemm(pm, c["x"])
        assert_close(y, ref, c["x"], wmax, f"e4m3 per-matrix B={B}")
        assert_precise(y, ref, f"e4m3 per-matrix B={B}")
    _report(f"grouped synth B={B}")
    ys, _ = _grouped(mats, cases, B)
    for c, y in zip(cases, ys):
        ref, wmax = oracle_rows(c)
        assert_close(y, ref, c["x"], wmax, f"e4m3 grouped B={B}")
        assert_precise(y, ref, f"e4m3 grouped B={B}")


@pytest.mark.parametrize("B", [1, 4, 12])
def test_e4m3_matches_fp16_storage(B):
    """The same residual values stored as fp16 (layout 2) give the same
    outputs bit for bit, per matrix and grouped: the E4M3 decode on the GPU
    is exact."""
    shapes = [(4096, 4096), (1024, 5000)]
    cases = [e4m3_synth_case(9, N, K, B, mat=i) for i, (N, K) in enumerate(shapes)]
    m8 = [gpu_pack_e4m3(c) for c in cases]
    m16 = [gpu_pack(c) for c in cases]
    for c, a, b in zip(cases, m8, m16):
        _report(f"e4m3 vs fp16 per-matrix B={B} N={c['N']} K={c['K']}")
        assert np.array_equal(gpu_gemm(a, c["x"]), gpu_gemm(b, c["x"]))
    y8, _ = _grouped(m8, cases, B)
    y16, _ = _grouped(m16, cases, B)
    for a, b in zip(y8, y16):
        assert np.array_equal(a, b)


def test_e4m3_pack_errors():
    import torch

    import paper_2609_00224_amd as q

    c = e4m3_dyadic_case(1, 64, 100, 1, 5)
    N, K, nS = 64, 100, 5
    bm = synth.column_bitmap(c["S"], K)
    dev = lambda a: to_dev(a)
    # the value and position arrays always have n rows (the pack reads n of each)
    idx_rows = lambda n: np.ascontiguousarray(np.resize(c["idx"], (n, N // 4)))
    args = lambda bitmap, n, r8: (dev(c["trits"]), dev(c["alpha"]), dev(c["v"]), dev(bitmap), n, dev(r8),
                                  dev(idx_rows(n)))
    for what, bitmap, n, r8 in [
        ("NaN value code 0x7f", bm, nS, np.where(np.arange(c["R8"].size).reshape(c["R8"].shape) == 7, 0x7f, c["R8"])),
        ("NaN value code 0xff", bm, nS, np.full_like(c["R8"], 0xff)),
        ("bitmap bit past K", np.array([*bm[:-1], bm[-1] | (1 << 10)], dtype=np.int32), nS + 1,
         np.concatenate([c["R8"], c["R8"][:1]])),
        ("bitmap count below n_salient", bm, nS + 1, np.concatenate([c["R8"], c["R8"][:1]])),
        ("bitmap count above n_salient", bm, nS - 1, c["R8"][:-1]),
    ]:
        _report(f"pack error: {what}")
        r8 = np.ascontiguousarray(r8.astype(np.uint8))
        assert r8.shape == (n, N // 4)
        with pytest.raises(q.QteaError) as e:
            q.pack_matrix_e4m3(*args(bitmap, n, r8))
        assert e.value.status == q.QTEA_ERR_BAD_RESIDUAL, what
    # one plan, one residual layout
    _report("grouped plan mixing layouts")
    a, b = gpu_pack_e4m3(c), gpu_pack(c)
    x = to_dev(c["x"])
    y1 = torch.empty((1, N), dtype=torch.float32, device="cuda")
    y2 = torch.empty((1, N), dtype=torch.float32, device="cuda")
    with pytest.raises(q.QteaError) as e:
        q.plan_grouped([a, b], [x, x], [y1, y2], batch=1)
    assert e.value.status == q.QTEA_ERR_INVALID_ARG


@pytest.mark.parametrize("frac", [Fraction(12, 100), Fraction(25, 100)])
def test_e4m3_dense_salient_grouped(frac):
    """Slices with more than 16 and more than 32 salient columns (the staged
    and the direct-load residual paths of the batch-1 kernel)."""
    for B in (1, 4):
        shapes = [(4096, 4096), (1024, 3000)]
        cases = [e4m3_synth_case(21, N, K, B, frac=frac, mat=i) for i, (N, K) in enumerate(shapes)]
        _report(f"grouped dense salient frac={frac} B={B}")
        ys, _ = _grouped([gpu_pack_e4m3(c) for c in cases], cases, B)
        for c, y in zip(cases, ys):
            ref, wmax = oracle_rows(c)
            assert_close(y, ref, c["x"], wmax, f"e4m3 frac={frac} B={B}")
            assert_precise(y, ref, f"e4m3 frac={frac} B={B}")
