"""GPU parity of the grouped GEMV (qtea_grouped_plan / qtea_grouped_gemv):
every problem of the group against the fp64 oracle, bit for bit on dyadic
inputs (every partial sum exact in fp32) and within the tolerance of
gpu_cases on synthetic inputs.  Groups are sized so that panels are split
between workgroups (the cross-workgroup reduction) and so that both panel
heights (512 and 1024 rows) are used.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np
import pytest

from synth.workloads import WORKLOADS
from tests.gpu_cases import assert_close, assert_precise, dyadic_case, gpu_pack, oracle_rows, synth_case, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch

    import paper_2609_00224_amd as q

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    q.load()


def _report(what):
    print(f"[case] {what}", flush=True)


def _run_group(cases, runs=1):
    """Pack every case, plan one grouped GEMV over all of them, run it
    `runs` times; returns (outputs of each run, plan, packed matrices)."""
    import torch

    import paper_2609_00224_amd as q

    mats = [gpu_pack(c) for c in cases]
    xs = [to_dev(c["x"]) for c in cases]
    ys = [torch.full((1, c["N"]), float("nan"), dtype=torch.float32, device="cuda") for c in cases]
    gp = q.plan_grouped(mats, xs, ys)
    outs = []
    for _ in range(runs):
        for y in ys:
            y.fill_(float("nan"))
        gp.run()
        torch.cuda.synchronize()
        outs.append([y.cpu().numpy() for y in ys])
    return outs, gp, mats


DYADIC_GROUP = [
    # (N, K, nS): ragged rows and columns, no salient columns, K spanning many slices
    (64, 5, 0), (256, 1003, 7), (1024, 640, 20), (4096, 4096, 82), (512, 14336, 287),
    (4160, 700, 40), (192, 81, 3),
]


def test_grouped_dyadic_exact():
    cases = [dyadic_case(300 + i, N, K, 1, nS) for i, (N, K, nS) in enumerate(DYADIC_GROUP)]
    _report(f"grouped dyadic {DYADIC_GROUP}")
    (outs,), gp, _ = _run_group(cases)
    assert gp.info.max_parts >= 2, "the group should split panels between workgroups"
    for c, y in zip(cases, outs):
        ref, _ = oracle_rows(c, need_wmax=False)
        assert np.array_equal(y.astype(np.float64), ref), f"{c['N']}x{c['K']}: not bit-exact"


def test_grouped_minimum_problem():
    c = dyadic_case(11, 64, 1, 1, 1)
    _report("grouped 64x1")
    (outs,), gp, _ = _run_group([c])
    ref, _ = oracle_rows(c, need_wmax=False)
    assert np.array_equal(outs[0].astype(np.float64), ref)


def test_grouped_dense_salient_slice():
    # every column salient: a slice holds 640 salient columns, far more than
    # the per-lane batch of residual loads
    c = dyadic_case(12, 512, 1280, 1, 1280)
    _report("grouped all-salient 512x1280")
    (outs,), _, _ = _run_group([c])
    ref, _ = oracle_rows(c, need_wmax=False)
    assert np.array_equal(outs[0].astype(np.float64), ref)


def _synth_group(layers, seed=7):
    wl = WORKLOADS["llama3_8b_stack"]
    cases = []
    for layer, mat, role, N, K in wl.matrices():
        if layer >= layers:
            break
        c = synth_case(seed, N, K, 1, p0=wl.p0, frac=wl.frac, layer=layer, mat=mat)
        c["N"], c["K"] = N, K
        cases.append(c)
    return cases


def test_grouped_synth_8b_layer():
    cases = _synth_group(1)
    _report("grouped synthetic 8B layer (4 matrices)")
    (outs,), gp, _ = _run_group(cases)
    for c, y in zip(cases, outs):
        ref, wmax = oracle_rows(c)
        assert_close(y, ref, c["x"], wmax, f"grouped {c['N']}x{c['K']}")
        assert_precise(y, ref, f"grouped {c['N']}x{c['K']}")


def test_grouped_synth_8b_eight_layers():
    cases = _synth_group(8)
    _report("grouped synthetic 8B stack, 8 layers (32 matrices)")
    (outs,), gp, _ = _run_group(cases)
    assert gp.info.rows_per_panel == 1024
    for c, y in zip(cases, outs):
        ref, wmax = oracle_rows(c)
        assert_close(y, ref, c["x"], wmax, f"grouped {c['N']}x{c['K']}")
        assert_precise(y, ref, f"grouped {c['N']}x{c['K']}")


def test_grouped_matches_gemv_and_is_deterministic():
    import torch

    import paper_2609_00224_amd as q

    cases = _synth_group(2, seed=9)
    _report("grouped vs qtea_gemv, 2 layers, 3 runs")
    outs, gp, mats = _run_group(cases, runs=3)
    for r in range(1, 3):
        for a, b in zip(outs[0], outs[r]):
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), "grouped run not deterministic"
    queue = gp.workspace[:4].view(torch.int32)
    assert int(queue.item()) == 0, "chunk queue counter not left at zero"
    for c, m, y in zip(cases, mats, outs[0]):
        X = to_dev(c["x"])
        Y = torch.empty((1, c["N"]), dtype=torch.float32, device="cuda")
        q.qtea_gemv(m.desc, m.packed, X, Y, q.new_workspace(m.desc, 1))
        torch.cuda.synchronize()
        ref, wmax = oracle_rows(c)
        assert_close(Y.cpu().numpy(), ref, c["x"], wmax, "gemv")
        assert_close(y, ref, c["x"], wmax, "grouped")
        assert_precise(y, ref, "grouped")


def test_grouped_graph_replay():
    import torch

    import paper_2609_00224_amd as q

    cases = _synth_group(1, seed=13)
    _report("grouped in a HIP graph, 3 replays")
    mats = [gpu_pack(c) for c in cases]
    xs = [to_dev(c["x"]) for c in cases]
    ys = [torch.zeros((1, c["N"]), dtype=torch.float32, device="cuda") for c in cases]
    gp = q.plan_grouped(mats, xs, ys)
    gp.run()
    torch.cuda.synchronize()
    eager = [y.clone() for y in ys]
    stream = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        gp.run(stream=stream)
        stream.synchronize()
        with torch.cuda.graph(g, stream=stream):
            gp.run(stream=stream)
    stream.synchronize()
    for rep in range(3):
        for y in ys:
            y.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        junk = torch.randn(1 << 20, device="cuda").sum()  # eager work between replays
        torch.cuda.synchronize()
        assert torch.isfinite(junk)
        for a, b in zip(ys, eager):
            assert torch.equal(a, b), f"replay {rep} differs from the eager result"


def test_grouped_errors():
    import torch

    import paper_2609_00224_amd as q

    c = dyadic_case(21, 256, 100, 1, 2)
    m = gpu_pack(c)
    x = to_dev(c["x"])
    y = torch.empty((1, 256), dtype=torch.float32, device="cuda")
    plan = torch.empty(q.qtea_grouped_plan_bytes(1), dtype=torch.uint8, device="cuda")
    for bad in (0, 17):
        with pytest.raises(q.QteaError) as e:
            q.qtea_grouped_plan([m.desc], [m.packed], [x], [y], bad, plan)
        assert e.value.status == q.QTEA_ERR_BATCH
    with pytest.raises(q.QteaError) as e:
        q.qtea_grouped_plan([m.desc], [m.packed], [x], [y], 1, plan[:16])
    assert e.value.status == q.QTEA_ERR_WORKSPACE
    info = q.qtea_grouped_plan([m.desc], [m.packed], [x], [y], 1, plan)
    small = torch.zeros(4, dtype=torch.uint8, device="cuda")
    with pytest.raises(q.QteaError) as e:
        q.qtea_grouped_gemv(info, plan, small)
    assert e.value.status == q.QTEA_ERR_WORKSPACE


def test_grouped_queue_left_over_counter_is_flagged():
    """A chunk-queue counter that does not start at zero (as after a call
    that did not complete, or a workspace that was not zero-filled) is set
    from the host: the launch stays in bounds, reports the condition through
    qtea_grouped_status, and leaves the counters at zero, so the next call
    (after the workspace is zero-filled, which clears the flags) is exact."""
    import torch

    import paper_2609_00224_amd as q

    cases = _synth_group(2, seed=9)
    _report("grouped queue: left-over counters (8 matrices)")
    mats = [gpu_pack(c) for c in cases]
    xs = [to_dev(c["x"]) for c in cases]
    ys = [torch.full((1, c["N"]), float("nan"), dtype=torch.float32, device="cuda") for c in cases]
    gp = q.plan_grouped(mats, xs, ys)
    info, ws = gp.info, gp.workspace
    assert info.n_chunks > 2 * info.grid, "the plan should hand out chunks from the queue"

    def run_clean():
        for y in ys:
            y.fill_(float("nan"))
        gp.run()
        torch.cuda.synchronize()
        assert q.qtea_grouped_status(ws) == 0
        return [y.cpu().numpy() for y in ys]

    first = run_clean()
    for c, y in zip(cases, first):
        ref, wmax = oracle_rows(c)
        assert_close(y, ref, c["x"], wmax, f"grouped {c['N']}x{c['K']}")
    # workspace words: [0] take counter, [1] flags, [2:4] the exit word (finished
    # workgroups in its top 16 bits, the tags of the chunks they ran below)
    words = ws[:16].view(torch.int32)
    exitw = ws[8:16].view(torch.int64)
    for start_take, start_exit in ((5, 0), (-(2 ** 31), 0), (0, 3 << 48), (0, 7)):
        _report(f"grouped queue: take counter {start_take & 0xffffffff}, exit word {start_exit:#x}")
        words[0] = start_take
        exitw[0] = start_exit
        torch.cuda.synchronize()
        gp.run()
        flags = q.qtea_grouped_status(ws)
        assert flags & (q.QTEA_QUEUE_STALE | q.QTEA_QUEUE_COUNT), "left-over counters not reported"
        if start_take < 0:
            assert flags & q.QTEA_QUEUE_STALE
        if start_exit == 0:
            assert words[0].item() == 0 and exitw[0].item() == 0, "counters not reset"
        ws.zero_()
        again = run_clean()
        for a, b in zip(first, again):
            assert np.array_equal(a, b)


