"""GPU parity of the grouped low-batch GEMM (qtea_grouped_plan with 2 <= batch
<= 16, the matrix-core kernel): every problem of the group against the fp64
oracle, bit for bit on dyadic inputs (every product and partial sum exact in
fp32, and every a_j = v_j x_j exact in fp16) and within the tolerance of
gpu_cases on synthetic inputs.  Groups are sized so that panels are split
between workgroups (the reduce kernel), with ragged rows and columns, parts
with more than 32 salient columns (several residual blocks), and a slice whose
activations exceed the fp16 range after rescaling (the scaled slow path).
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np
import pytest

from synth.workloads import WORKLOADS
from tests.gpu_cases import (assert_close, assert_precise, dyadic_case, fine_case, gpu_pack, oracle_rows,
                             synth_case, to_dev)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch

    import paper_2609_00224_amd as q

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    q.load()


def _report(what):
    print(f"[case] {what}", flush=True)


def _run_group(cases, B, runs=1):
    import torch

    import paper_2609_00224_amd as q

    mats = [gpu_pack(c) for c in cases]
    xs = [to_dev(c["x"]) for c in cases]
    ys = [torch.full((B, c["N"]), float("nan"), dtype=torch.float32, device="cuda") for c in cases]
    gp = q.plan_grouped(mats, xs, ys, batch=B)
    outs = []
    for _ in range(runs):
        for y in ys:
            y.fill_(float("nan"))
        gp.run()
        torch.cuda.synchronize()
        outs.append([y.cpu().numpy() for y in ys])
    return outs, gp


DYADIC_GROUP = [(64, 5, 0), (256, 1003, 7), (1024, 640, 20), (4096, 4096, 82), (512, 14336, 287),
                (4160, 700, 40), (192, 81, 3), (2048, 3200, 300)]


@pytest.mark.parametrize("B", [2, 3, 8, 9, 16])
def test_grouped_batch_dyadic_exact(B):
    cases = [dyadic_case(500 + 13 * B + i, N, K, B, nS) for i, (N, K, nS) in enumerate(DYADIC_GROUP)]
    _report(f"grouped batch {B} dyadic {DYADIC_GROUP}")
    (outs,), gp = _run_group(cases, B)
    assert gp.info.batch == B
    # the matrix-core workgroup shape: 1024 threads (rows per panel) up to
    # batch 8, 768 above
    assert gp.info.rows_per_panel == (1024 if B <= 8 else 768)
    assert gp.info.n_split_panels > 0, "the group should split panels between workgroups"
    for c, y in zip(cases, outs):
        ref, _ = oracle_rows(c, need_wmax=False)
        bad = np.argwhere(y.astype(np.float64) != ref)
        assert bad.size == 0, f"{c['N']}x{c['K']} B={B}: {len(bad)} outputs differ, first {bad[:4].tolist()}"


FINE_GROUP = [(256, 1000), (4160, 640), (1024, 999), (64, 7)]


@pytest.mark.parametrize("B", [2, 5, 8, 9, 16])
def test_grouped_batch_both_halves_exact(B):
    # a_j needs both fp16 halves (hi and lo): the result is still exact
    cases = [fine_case(900 + 7 * B + i, N, K, B) for i, (N, K) in enumerate(FINE_GROUP)]
    _report(f"grouped batch {B}, activations split in two halves, {FINE_GROUP}")
    (outs,), _ = _run_group(cases, B)
    for c, y in zip(cases, outs):
        ref, _ = oracle_rows(c, need_wmax=False)
        bad = np.argwhere(y.astype(np.float64) != ref)
        assert bad.size == 0, f"{c['N']}x{c['K']} B={B}: {len(bad)} outputs differ, first {bad[:4].tolist()}"


def test_grouped_batch_single_small_problem():
    c = dyadic_case(41, 64, 1, 4, 1)
    _report("grouped batch 4, 64x1")
    (outs,), _ = _run_group([c], 4)
    ref, _ = oracle_rows(c, need_wmax=False)
    assert np.array_equal(outs[0].astype(np.float64), ref)


def _synth(layers, B, name="llama3_8b_stack", seed=7):
    wl = WORKLOADS[name]
    cases = []
    for layer, mat, role, N, K in wl.matrices():
        if layer >= layers:
            break
        c = synth_case(seed, N, K, B, p0=wl.p0, frac=wl.frac, layer=layer, mat=mat)
        c["N"], c["K"] = N, K
        cases.append(c)
    return cases


@pytest.mark.parametrize("B,name", [(4, "llama3_8b_stack"), (8, "qwen3_14b_stack"), (16, "qwen3_14b_stack")])
def test_grouped_batch_synth_layer(B, name):
    cases = _synth(1, B, name)
    _report(f"grouped batch {B} synthetic {name} layer")
    (outs,), _ = _run_group(cases, B)
    for c, y in zip(cases, outs):
        ref, wmax = oracle_rows(c)
        assert_close(y, ref, c["x"], wmax, f"grouped B={B} {c['N']}x{c['K']}")
        assert_precise(y, ref, f"grouped B={B} {c['N']}x{c['K']}")


def test_grouped_batch_deterministic_and_queue_left_zero():
    import torch

    cases = _synth(1, 5, seed=9)
    _report("grouped batch 5, 3 runs")
    outs, gp = _run_group(cases, 5, runs=3)
    for r in (1, 2):
        for a, b in zip(outs[0], outs[r]):
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), "not deterministic"
    assert int(gp.workspace[:4].view(torch.int32).item()) == 0


def test_grouped_batch_large_activations():
    # one slice's activations beyond the fp16 range of v_j x_j: scaled path
    B = 3
    c = dyadic_case(77, 512, 960, B, 9)
    c["x"][1, 333] = np.float16(60000.0)
    c["v"][333] = np.float16(2.0)
    c["x"][2, 700] = np.float16(-40000.0)
    c["v"][700] = np.float16(1.5)
    _report("grouped batch 3 with |v x| beyond fp16")
    (outs,), _ = _run_group([c], B)
    ref, wmax = oracle_rows(c)
    assert np.all(np.isfinite(outs[0]))
    assert_close(outs[0], ref, c["x"], wmax, "large activations")
