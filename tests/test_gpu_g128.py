"""GPU parity of the paper's grouped format (128-column quantization groups
with a scale and a bias per row and group, 26-byte packs, E4M3 residual
values and a salient bitmap): packing read back bit for bit, the grouped
batch-1 GEMV against the fp64 oracle (bit for bit on dyadic inputs, within
the tolerance of gpu_cases on synthetic ones at the 8B shapes), the
per-matrix call, and batches above one (the rows one after another
through the batch-1 kernel)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from tests.gpu_cases import (assert_close, assert_precise, g128_dyadic_case, g128_synth_case, gpu_pack_g128,
                             gpu_unpack, oracle_rows_g128, to_dev)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch

    import paper_2609_00224_amd as q

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    q.load()


def _report(what):
    print(f"[case] {what}", flush=True)


def _grouped(mats, cases):
    import torch

    import paper_2609_00224_amd as q

    xs = [to_dev(c["x"]) for c in cases]
    ys = [torch.full((1, c["N"]), float("nan"), dtype=torch.float32, device="cuda") for c in cases]
    gp = q.plan_grouped(mats, xs, ys, batch=1)
    gp.run()
    torch.cuda.synchronize()
    return [y.cpu().numpy() for y in ys], gp


SHAPES = [(256, 1000, 50), (4160, 640, 32), (64, 5, 1), (1024, 14336, 300), (192, 130, 0), (512, 4096, 205),
          (4, 1, 1), (12, 300, 15), (68, 129, 3)]


def test_g128_layout_decode_bit_exact():
    import paper_2609_00224_amd as q

    for N, K, nS in SHAPES:
        _report(f"decode N={N} K={K} nS={nS}")
        c = g128_dyadic_case(3, N, K, 1, nS)
        pm = gpu_pack_g128(c)
        d = pm.desc
        assert d.layout == q.QTEA_LAYOUT_G128 and d.n_packs == 26 * ((K + 127) // 128)
        assert d.bytes_total == q.qtea_packed_bytes_g128(N, K, nS)
        codes, trits, rows = gpu_unpack(pm)
        assert np.array_equal(codes, oracle.pack128(c["trits"]))
        assert np.array_equal(trits, c["trits"])
        if nS:
            assert np.array_equal(rows, oracle.resid_rows(c["idx"], N))


def test_g128_grouped_dyadic_exact():
    cases = [g128_dyadic_case(40 + i, N, K, 1, nS) for i, (N, K, nS) in enumerate(SHAPES)]
    _report("grouped dyadic, batch 1")
    ys, gp = _grouped([gpu_pack_g128(c) for c in cases], cases)
    for c, y in zip(cases, ys):
        ref, _ = oracle_rows_g128(c, need_wmax=False)
        assert np.array_equal(y.astype(np.float64), ref), (c["N"], c["K"])


def test_g128_grouped_single_problem_and_repeat():
    c = g128_dyadic_case(9, 2048, 3000, 1, 150)
    pm = gpu_pack_g128(c)
    import torch

    import paper_2609_00224_amd as q

    _report("grouped dyadic single problem, three runs")
    y = torch.full((1, 2048), float("nan"), dtype=torch.float32, device="cuda")
    gp = q.plan_grouped([pm], [to_dev(c["x"])], [y], batch=1)
    ref, _ = oracle_rows_g128(c, need_wmax=False)
    for _ in range(3):
        y.fill_(float("nan"))
        gp.run()
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy().astype(np.float64), ref)
    assert int(gp.workspace[:4].view(torch.int32).item()) == 0


def test_g128_synth_8b_shapes():
    shapes = [(6144, 4096), (4096, 4096), (28672, 4096), (4096, 14336)]
    cases = [g128_synth_case(5, N, K, 1, mat=i) for i, (N, K) in enumerate(shapes)]
    _report("grouped synth, 8B layer shapes")
    ys, _ = _grouped([gpu_pack_g128(c) for c in cases], cases)
    rng = np.random.default_rng(0)
    for c, y in zip(cases, ys):
        N = c["N"]
        rows = np.unique(np.concatenate([np.arange(64), np.arange(N - 64, N), rng.choice(N, 512, replace=False)]))
        ref, wmax = oracle_rows_g128(c, rows=rows)
        assert_close(y[:, rows], ref, c["x"], wmax, f"g128 {N}x{c['K']}")
        assert_precise(y[:, rows], ref, f"g128 {N}x{c['K']}")


def test_g128_per_matrix_gemv_dyadic_exact():
    """qtea_gemv takes the grouped format at batch 1 (the table kernel on one
    problem); bit-exact on dyadic inputs, twice on one workspace."""
    import torch

    import paper_2609_00224_amd as q

    for i, (N, K, nS) in enumerate(SHAPES):
        c = g128_dyadic_case(60 + i, N, K, 1, nS)
        _report(f"per-matrix gemv, grouped format, dyadic {N}x{K} nS={nS}")
        pm = gpu_pack_g128(c)
        x = to_dev(c["x"])
        ws = q.new_workspace(pm.desc, 1)
        ref, _ = oracle_rows_g128(c, need_wmax=False)
        for _ in range(2):
            y = torch.full((1, N), float("nan"), dtype=torch.float32, device="cuda")
            q.qtea_gemv(pm.desc, pm.packed, x, y, ws)
            torch.cuda.synchronize()
            assert np.array_equal(y.cpu().numpy().astype(np.float64), ref), (N, K)


@pytest.mark.parametrize("B", [2, 4, 16])
def test_g128_batch_above_one_dyadic_exact(B):
    """At batch B the grouped format runs its rows through the batch-1 table
    kernel: per-matrix (qtea_gemm_lowbatch, B launches) and grouped (B batch-1
    problems per matrix), bit for bit against the fp64 oracle on dyadic
    inputs, every batch row."""
    import torch

    import paper_2609_00224_amd as q

    cases = [g128_dyadic_case(80 + i + B, N, K, B, nS) for i, (N, K, nS) in enumerate(SHAPES[:4])]
    mats = [gpu_pack_g128(c) for c in cases]
    refs = [oracle_rows_g128(c, need_wmax=False)[0] for c in cases]
    for c, pm, ref in zip(cases, mats, refs):
        N, K = c["N"], c["K"]
        _report(f"per-matrix lowbatch, grouped format, dyadic {N}x{K} B={B}")
        assert ref.shape == (B, N)
        ws = q.new_workspace(pm.desc, B)
        assert q.qtea_workspace_bytes(pm.desc, B) == q.qtea_workspace_bytes(pm.desc, 1)
        for _ in range(2):
            y = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
            q.qtea_gemm_lowbatch(pm.desc, pm.packed, to_dev(c["x"]), B, y, ws)
            torch.cuda.synchronize()
            assert np.array_equal(y.cpu().numpy().astype(np.float64), ref), (N, K, B)
    _report(f"grouped, grouped format, dyadic, B={B}")
    xs = [to_dev(c["x"]) for c in cases]
    ys = [torch.full((B, c["N"]), float("nan"), dtype=torch.float32, device="cuda") for c in cases]
    gp = q.plan_grouped(mats, xs, ys, batch=B)
    assert gp.info.batch == 1 and gp.info.n_problems == B * len(cases)
    for _ in range(2):
        for y in ys:
            y.fill_(float("nan"))
        gp.run()
        torch.cuda.synchronize()
        for c, y, ref in zip(cases, ys, refs):
            assert np.array_equal(y.cpu().numpy().astype(np.float64), ref), (c["N"], c["K"], B)
    assert q.qtea_grouped_status(gp.workspace) == 0


def test_g128_batch_4_synth_8b_shapes():
    """The 8B layer's four shapes in the grouped format at batch 4 through
    qtea_gemm_lowbatch, sampled rows of every batch row within tolerance."""
    import torch

    import paper_2609_00224_amd as q

    shapes = [(6144, 4096), (4096, 4096), (28672, 4096), (4096, 14336)]
    rng = np.random.default_rng(1)
    for i, (N, K) in enumerate(shapes):
        c = g128_synth_case(6, N, K, 4, mat=i)
        _report(f"per-matrix lowbatch, grouped format, synth {N}x{K} B=4")
        pm = gpu_pack_g128(c)
        y = torch.full((4, N), float("nan"), dtype=torch.float32, device="cuda")
        q.qtea_gemm_lowbatch(pm.desc, pm.packed, to_dev(c["x"]), 4, y, q.new_workspace(pm.desc, 4))
        torch.cuda.synchronize()
        rows = np.unique(np.concatenate([np.arange(64), np.arange(N - 64, N), rng.choice(N, 256, replace=False)]))
        ref, wmax = oracle_rows_g128(c, rows=rows)
        got = y.cpu().numpy()[:, rows]
        assert_close(got, ref, c["x"], wmax, f"g128 B=4 {N}x{K}")
        assert_precise(got, ref, f"g128 B=4 {N}x{K}")
