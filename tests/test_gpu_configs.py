"""GPU parity on the five benchmark configurations, at their full matrix
shapes and batch sizes, in the launch configuration bench.py times (one
grouped call over the whole set of matrices):

  single 4096x4096 GEMV, batch 1                      (all rows)
  one Llama-3-8B-shaped layer, batch 1                (all rows)
  32-layer Llama-3-8B-shaped stack, batch 1 and 4     (all 128 matrices)
  Qwen3-14B-shaped layers, 3% salient, batch 1, 8, 16 (two layers)
  Llama-3-70B-shaped layers, P(0)=0.5, batch 1, 16    (two layers)

The 14B- and 70B-shaped stacks are taken two layers deep (every matrix shape
of the layer at full size; the kernels see the same shapes as in the full
stacks).  Outputs: every row of the single GEMV and of the single layer,
and of the stacks' matrices up to 4096 x 14336 elements, else the first and
last 64 rows and 1024 random rows, against the fp64 oracle
within the tolerance of gpu_cases.  Decode: the first layer's packed codes
and residual rows read back bit-exactly.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import synth
from synth.workloads import WORKLOADS
from tests.gpu_cases import REL_L2, REL_L2_PRECISE, ROW_ABS, to_dev

pytestmark = pytest.mark.gpu

CONFIGS = [
    ("gemv_4096x4096", None, (1,)),
    ("llama3_8b_layer", None, (1,)),
    ("llama3_8b_stack", None, (1, 4)),
    ("qwen3_14b_stack", 2, (1, 8, 16)),
    ("llama3_70b_stack", 2, (1, 16)),
]
SEED = 20260224
_cache = {}


def _report(what):
    print(f"[case] {what}", flush=True)


def _stack(name, layers):
    """Packed matrices of the workload (kept for the batches of one config)."""
    import torch

    import paper_2609_00224_amd as q

    key = (name, layers)
    if key in _cache:
        return _cache[key]
    _cache.clear()
    torch.cuda.empty_cache()
    wl = WORKLOADS[name]
    mats = []
    for layer, mat, role, N, K in wl.matrices():
        if layers is not None and layer >= layers:
            break
        L = synth.layer_inputs(SEED, layer, mat, N, K, p0=wl.p0, frac=wl.frac)
        pm = q.pack_matrix(to_dev(L["trits"]), to_dev(L["alpha"]), to_dev(L["v"]), to_dev(L["S"]),
                           to_dev(L["R"]), to_dev(L["idx"]))
        if layer == 0:  # decode check on the first layer
            codes = torch.empty((N, pm.desc.n_packs), dtype=torch.uint8, device="cuda")
            rows = torch.empty((max(int(L["S"].size), 1), N // 4), dtype=torch.int32, device="cuda")
            q.qtea_debug_unpack(pm.desc, pm.packed, canon_codes=codes,
                                resid_row=rows if L["S"].size else None)
            torch.cuda.synchronize()
            assert np.array_equal(codes.cpu().numpy(), oracle.pack(L["trits"])), f"{name} {role}: codes"
            if L["S"].size:
                assert np.array_equal(rows.cpu().numpy(), oracle.resid_rows(L["idx"], N)), f"{name} {role}: resid"
        del L
        mats.append({"layer": layer, "mat": mat, "role": role, "N": N, "K": K, "pm": pm})
    torch.cuda.synchronize()
    _cache[key] = (wl, mats)
    return wl, mats


FULL_ROWS = ("gemv_4096x4096", "llama3_8b_layer")


def _sample_rows(N, K, rng, full=False):
    if full or N * K <= 4096 * 14336:
        return np.arange(N, dtype=np.int64)
    rnd = rng.choice(np.arange(64, N - 64), size=1024, replace=False)
    return np.unique(np.concatenate([np.arange(64), np.arange(N - 64, N), rnd])).astype(np.int64)


@pytest.mark.parametrize("name,layers,B", [(n, l, b) for n, l, bs in CONFIGS for b in bs])
def test_config_grouped_parity(name, layers, B):
    import torch

    import paper_2609_00224_amd as q

    _report(f"{name} layers={layers or 'all'} batch {B}")
    wl, mats = _stack(name, layers)
    xs, ys = [], []
    for m in mats:
        xs.append(to_dev(synth.activations(SEED, m["layer"], m["mat"], B, m["K"])))
        ys.append(torch.full((B, m["N"]), float("nan"), dtype=torch.float32, device="cuda"))
    gp = q.plan_grouped([m["pm"] for m in mats], xs, ys, batch=B)
    gp.run()
    torch.cuda.synchronize()
    rng = np.random.default_rng(B * 1000 + len(mats))
    worst = 0.0
    for m, x, y in zip(mats, xs, ys):
        N, K = m["N"], m["K"]
        rows = _sample_rows(N, K, rng, full=name in FULL_ROWS)
        L = synth.layer_inputs(SEED, m["layer"], m["mat"], N, K, p0=wl.p0, frac=wl.frac, rows=rows)
        codes = oracle.pack(L["trits"])
        xh = x.cpu().numpy()
        args = (N, K, codes, L["alpha"], L["v"], L["S"], L["R"], L["idx"])
        ref = oracle.gemv(*args, xh, rows=rows)
        wmax = np.empty(rows.size)
        for i in range(0, rows.size, 512):  # max |W_eff| per row, a block of rows at a time
            sl = slice(i, i + 512)
            wmax[sl] = np.abs(oracle.dense_rows(N, K, codes[sl], *args[3:], rows=rows[sl])).max(axis=1)
        got = y.cpu().numpy()[:, rows].astype(np.float64)
        assert np.all(np.isfinite(got)), f"{m['role']} layer {m['layer']}: non-finite outputs"
        xl1 = np.abs(xh.astype(np.float64)).sum(axis=1)
        for b in range(B):
            d = np.abs(got[b] - ref[b])
            rel = np.linalg.norm(d) / np.linalg.norm(ref[b])
            worst = max(worst, rel)
            assert rel <= REL_L2, f"{m['role']} layer {m['layer']} batch row {b}: relative L2 {rel:.3e}"
            assert rel <= REL_L2_PRECISE, f"{m['role']} layer {m['layer']} batch row {b}: relative L2 {rel:.3e}"
            bad = np.nonzero(d > ROW_ABS * xl1[b] * wmax)[0]
            assert bad.size == 0, f"{m['role']} layer {m['layer']} batch row {b}: row bound at rows {rows[bad[:5]]}"
    print(f"[case] {name} batch {B}: {len(mats)} matrices, worst relative L2 {worst:.2e}", flush=True)
