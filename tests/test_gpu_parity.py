"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Integer work (packing, decode, residual positions) must match bit for bit;
floating-point outputs must match within the tolerance of gpu_cases, and
bit for bit on dyadic inputs where every partial sum is exact in fp32.
"""
from __future__ import annotations

import ctypes
from fractions import Fraction

import numpy as np
import pytest

import oracle
from tests.gpu_cases import (assert_close, assert_precise, dyadic_case, gpu_gemm, gpu_pack, gpu_unpack, oracle_rows,
                             synth_case, to_dev)
from tests.golden import load_worked_example

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch

    import paper_2609_00224_amd as q

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    q.load()


def _report(what):
    print(f"[case] {what}", flush=True)


# ---------------------------------------------------------------------------
# Hand-worked example and exhaustive code table: exact.
# ---------------------------------------------------------------------------
def test_worked_example_exact():
    w = load_worked_example()
    pm = gpu_pack(w)
    codes, trits, rows = gpu_unpack(pm)
    assert np.array_equal(codes, w["codes"])
    assert np.array_equal(trits, w["trits"])
    assert np.array_equal(rows, oracle.resid_rows(w["idx"], w["N"]))
    y = gpu_gemm(pm, w["x"])
    assert np.array_equal(y.astype(np.float64), w["y"])


def test_exhaustive_codes_exact():
    N, K = 256, 5
    trits = np.zeros((N, K), np.int8)
    for c in range(243):
        trits[c] = oracle.decode_code(c)
    case = {
        "N": N, "K": K, "trits": trits,
        "alpha": (2.0 ** -(np.arange(N) % 4)).astype(np.float16),
        "v": np.array([0.5, 1.0, 1.5, 2.0, 0.5], np.float16),
        "S": np.zeros(0, np.int32), "R": np.zeros((0, N // 4), np.float16),
        "idx": np.zeros((0, N // 4), np.uint8),
        "x": np.array([[1.0, -2.0, 0.25, 4.0, -0.75]], np.float16),
    }
    pm = gpu_pack(case)
    codes, _, _ = gpu_unpack(pm)
    assert np.array_equal(codes[:243, 0], np.arange(243))
    assert np.all(codes[243:, 0] == 121)
    y = gpu_gemm(pm, case["x"])
    ref, _ = oracle_rows(case)
    assert np.array_equal(y.astype(np.float64), ref)


# ---------------------------------------------------------------------------
# Decode: bit-exact over edge shapes.
# ---------------------------------------------------------------------------
DECODE_SHAPES = [(4, 1, 0), (4, 4, 1), (8, 5, 1), (16, 6, 2), (60, 9, 3), (64, 10, 10), (68, 79, 4),
                 (128, 80, 80), (196, 81, 7), (260, 319, 6), (1028, 320, 9), (4, 321, 321),
                 (4096, 4097, 82), (1024, 14336, 287)]


@pytest.mark.parametrize("N,K,nS", DECODE_SHAPES)
def test_decode_bit_exact(N, K, nS):
    _report(f"decode N={N} K={K} nS={nS}")
    case = synth_case(11, N, K, 1, nS=nS)
    pm = gpu_pack(case)
    codes, trits, rows = gpu_unpack(pm)
    assert np.array_equal(codes, oracle.pack(case["trits"]))
    assert np.array_equal(trits, case["trits"])
    assert np.array_equal(rows, oracle.resid_rows(case["idx"], N))
    assert codes.max() < 243


# ---------------------------------------------------------------------------
# Dyadic inputs: GPU == oracle bit for bit.
# ---------------------------------------------------------------------------
DYADIC = [(4, 1, 1, 0), (8, 7, 1, 2), (64, 80, 2, 5), (68, 81, 3, 4), (196, 319, 1, 9),
          (260, 1601, 4, 20), (1028, 1601, 5, 33), (4096, 4097, 1, 82), (2048, 4100, 8, 60),
          (512, 14336, 16, 287), (28672, 4096, 1, 82)]


@pytest.mark.parametrize("N,K,B,nS", DYADIC)
def test_dyadic_bit_exact(N, K, B, nS):
    _report(f"dyadic N={N} K={K} B={B} nS={nS}")
    case = dyadic_case(N * 7 + K, N, K, B, nS)
    pm = gpu_pack(case)
    y = gpu_gemm(pm, case["x"])
    ref, _ = oracle_rows(case, need_wmax=False)
    assert np.array_equal(y.astype(np.float64), ref)


# ---------------------------------------------------------------------------
# Random inputs of the workload distributions: within tolerance.
# ---------------------------------------------------------------------------
RANDOM = [(4, 1, 1, None), (64, 10, 1, None), (128, 999, 2, None), (196, 4096, 1, None),
          (4096, 4096, 1, None), (4096, 4096, 4, None), (6144, 4096, 1, None), (4096, 14336, 1, None),
          (1024, 5120, 8, None), (512, 17408, 16, None), (2048, 8192, 3, 0), (1024, 4096, 16, 4096)]


@pytest.mark.parametrize("N,K,B,nS", RANDOM)
def test_random_within_tolerance(N, K, B, nS):
    _report(f"random N={N} K={K} B={B} nS={nS}")
    case = synth_case(5 + N + K, N, K, B, nS=nS)
    pm = gpu_pack(case)
    y = gpu_gemm(pm, case["x"])
    ref, wmax = oracle_rows(case)
    assert_close(y, ref, case["x"], wmax, f"N={N} K={K} B={B}")
    assert_precise(y, ref, f"N={N} K={K} B={B}")


@pytest.mark.parametrize("B", list(range(1, 17)))
def test_every_batch_size(B):
    _report(f"batch B={B}")
    case = synth_case(100 + B, 320, 2005, B, frac=Fraction(3, 100))
    pm = gpu_pack(case)
    y = gpu_gemm(pm, case["x"])
    ref, wmax = oracle_rows(case)
    assert_close(y, ref, case["x"], wmax, f"B={B}")
    assert_precise(y, ref, f"B={B}")


# ---------------------------------------------------------------------------
# Special cases.
# ---------------------------------------------------------------------------
def test_zero_trits_give_exact_zero():
    case = synth_case(3, 256, 1000, 2, nS=0)
    case["trits"][:] = 0
    y = gpu_gemm(gpu_pack(case), case["x"])
    assert np.all(y == 0.0)


def test_single_trit_one_rounding():
    case = synth_case(4, 128, 777, 1, nS=0)
    case["trits"][:] = 0
    case["trits"][77, 500] = -1
    y = gpu_gemm(gpu_pack(case), case["x"])
    ref, _ = oracle_rows(case)
    assert np.array_equal(y, ref.astype(np.float32))
    assert np.count_nonzero(y) == 1


def test_residual_only():
    case = synth_case(6, 256, 640, 3, nS=12)
    case["trits"][:] = 0
    y = gpu_gemm(gpu_pack(case), case["x"])
    ref, wmax = oracle_rows(case)
    assert_close(y, ref, case["x"], wmax, "residual only")
    assert_precise(y, ref, "residual only")
    assert np.array_equal(y != 0, ref != 0)


# ---------------------------------------------------------------------------
# Entry-point semantics.
# ---------------------------------------------------------------------------
def test_gemv_equals_lowbatch_b1_and_deterministic():
    case = synth_case(8, 4096, 4096, 1)
    pm = gpu_pack(case)
    y1 = gpu_gemm(pm, case["x"], use_gemv=True)
    y2 = gpu_gemm(pm, case["x"])
    y3 = gpu_gemm(pm, case["x"])
    assert np.array_equal(y1, y2) and np.array_equal(y2, y3)


def test_workspace_shared_across_matrices():
    """Counters return to zero after every call: one workspace serves a
    stream-ordered sequence of different matrices and batch sizes."""
    import torch

    import paper_2609_00224_amd as q

    cases = [synth_case(20 + i, N, K, B) for i, (N, K, B) in
             enumerate([(4096, 4096, 1), (1024, 14336, 2), (6144, 4096, 1), (512, 5120, 4)])]
    pms = [gpu_pack(c) for c in cases]
    need = max(q.qtea_workspace_bytes(pm.desc, c["x"].shape[0]) for pm, c in zip(pms, cases))
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    for rep in range(2):
        for pm, c in zip(pms, cases):
            y = gpu_gemm(pm, c["x"], ws=ws)
            ref, wmax = oracle_rows(c)
            assert_close(y, ref, c["x"], wmax, f"shared ws rep {rep}")
            assert_precise(y, ref, f"shared ws rep {rep}")
    # the panels' arrival counters (the workspace's first 256 bytes here)
    counters = ws[:256].cpu().numpy()
    assert np.all(counters == 0)


def test_error_statuses():
    import torch

    import paper_2609_00224_amd as q

    case = synth_case(9, 64, 100, 1)
    bad = dict(case)
    bad["trits"] = case["trits"].copy()
    bad["trits"][3, 7] = 2
    with pytest.raises(q.QteaError) as e:
        gpu_pack(bad)
    assert e.value.status == q.QTEA_ERR_BAD_TRIT
    bad = dict(case)
    bad["idx"] = case["idx"].copy()
    bad["idx"][0, 1] = 4
    with pytest.raises(q.QteaError) as e:
        gpu_pack(bad)
    assert e.value.status == q.QTEA_ERR_BAD_RESIDUAL
    bad = dict(case)
    bad["S"] = case["S"][::-1].copy()
    with pytest.raises(q.QteaError) as e:
        gpu_pack(bad)
    assert e.value.status == q.QTEA_ERR_BAD_RESIDUAL
    for v in (np.inf, -np.inf, np.nan):  # a residual value that is not finite
        bad = dict(case)
        bad["R"] = case["R"].copy()
        bad["R"][-1, -1] = v
        with pytest.raises(q.QteaError) as e:
            gpu_pack(bad)
        assert e.value.status == q.QTEA_ERR_BAD_RESIDUAL, v
    pm = gpu_pack(case)
    X = to_dev(np.zeros((17, 100), np.float16))
    Y = torch.empty((17, 64), dtype=torch.float32, device="cuda")
    ws = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
    for b in (0, 17):
        with pytest.raises(q.QteaError) as e:
            q.qtea_gemm_lowbatch(pm.desc, pm.packed, X, b, Y, ws)
        assert e.value.status == q.QTEA_ERR_BATCH
    need = q.qtea_workspace_bytes(pm.desc, 1)
    small = torch.zeros(max(need - 4, 0), dtype=torch.uint8, device="cuda")
    if need > 4:
        with pytest.raises(q.QteaError) as e:
            q.qtea_gemv(pm.desc, pm.packed, X, Y, small)
        assert e.value.status == q.QTEA_ERR_WORKSPACE
    packed = torch.empty(q.qtea_packed_bytes(64, 100, case["S"].size) - 256, dtype=torch.uint8,
                         device="cuda")
    with pytest.raises(q.QteaError) as e:
        q.qtea_pack(to_dev(case["trits"]), to_dev(case["alpha"]), to_dev(case["v"]), to_dev(case["S"]),
                    to_dev(case["R"]), to_dev(case["idx"]), packed)
    assert e.value.status == q.QTEA_ERR_WORKSPACE


def test_workspace_init_zeroes():
    import torch

    import paper_2609_00224_amd as q

    ws = torch.full((1027,), 7, dtype=torch.uint8, device="cuda")
    q.qtea_workspace_init(ws)
    torch.cuda.synchronize()
    assert int(ws.sum().item()) == 0
