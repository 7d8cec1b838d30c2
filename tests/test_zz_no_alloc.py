"""The allocation-free entry point (qtea_gemm_lowbatch_noalloc) against the
workspace entry point it shares its kernels with (qtea_gemm_lowbatch),
through the C ABI: the outputs are the same bit for bit (same kernels, same
launch shape, same summation order), on two calls in a row of which the
second has the smaller input, then the first again (the scratch's counters
are left at zero by every completed call); batch 16 on a large matrix fits
the fixed scratch; a call whose workspace would not fit it is refused on the
host."""
from __future__ import annotations

import numpy as np
import pytest

from tests.gpu_cases import gpu_pack, synth_case, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch

    import paper_2609_00224_amd as q

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    q.load()


def _report(what):
    print(f"[case] {what}", flush=True)


def _both(pm, x, B):
    import torch

    import paper_2609_00224_amd as q

    N = pm.desc.N
    X = to_dev(x)
    ws = q.new_workspace(pm.desc, B)
    y_ws = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    q.qtea_gemm_lowbatch(pm.desc, pm.packed, X, B, y_ws, ws)
    y_na = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    q.qtea_gemm_lowbatch_noalloc(pm.desc, pm.packed, X, B, y_na)
    torch.cuda.synchronize()
    return y_ws.cpu().numpy(), y_na.cpu().numpy()


def test_noalloc_matches_workspace_entry_point():
    big = synth_case(31, 4096, 14336, 2)
    small = synth_case(32, 512, 1000, 1)
    pm_big, pm_small = gpu_pack(big), gpu_pack(small)
    for tag, pm, c in (("4096x14336 batch 2", pm_big, big), ("512x1000 batch 1 (smaller, second)", pm_small, small),
                       ("4096x14336 batch 2 again", pm_big, big)):
        _report(f"noalloc {tag}")
        a, b = _both(pm, c["x"], c["x"].shape[0])
        assert np.isfinite(a).all()
        assert np.array_equal(a, b), tag


def test_noalloc_large_matrix_batch_1_and_16_and_refusal():
    import torch

    import paper_2609_00224_amd as q

    c = synth_case(33, 16384, 5120, 16)
    pm = gpu_pack(c)
    for B in (1, 16):
        _report(f"noalloc 16384x5120 batch {B}")
        # batch 16: 2 x 256 workgroups x 512 rows x 16 x 4 bytes of partial
        # rows, which the fixed scratch holds
        assert q.qtea_workspace_bytes(pm.desc, B) <= q.QTEA_NOALLOC_SCRATCH_BYTES
        a, b = _both(pm, c["x"][:B], B)
        assert np.isfinite(a).all()
        assert np.array_equal(a, b)
    # 16385 panels of 512 rows need more arrival counters than the scratch
    # keeps (4 bytes each, 65536 bytes): refused before any launch
    tall = synth_case(34, 16385 * 512, 5, 1)
    pt = gpu_pack(tall)
    _report("noalloc refusal, 8389120x5 batch 1")
    X = to_dev(tall["x"])
    Y = torch.zeros((1, tall["trits"].shape[0]), dtype=torch.float32, device="cuda")
    with pytest.raises(q.QteaError) as e:
        q.qtea_gemm_lowbatch_noalloc(pt.desc, pt.packed, X, 1, Y)
    assert e.value.status == q.QTEA_ERR_WORKSPACE
