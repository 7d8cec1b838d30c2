"""The debug build (libqtea_debug.so, loaded when QTEA_DEBUG=1): the rows of
every decode table for the byte values 243..255, which no base-3 code of
five trits takes, read NaN.  A packed byte corrupted into such a value must
turn exactly its output row into NaN, through the batch-1 table kernel and
the matrix-core kernel, per matrix and grouped, while every other row keeps
the oracle's value bit for bit (dyadic inputs), and the uncorrupted matrix
gives the oracle's output everywhere.  The corruption is written from the
host into a copy of the packed buffer; no kernel is made to fault."""
from __future__ import annotations

import os

import numpy as np
import pytest

from tests.gpu_cases import dyadic_case, gpu_pack, oracle_rows, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def debug_lib():
    import torch

    import paper_2609_00224_amd as q

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    q.load()
    assert os.path.exists(q.DEBUG_LIB_PATH), "the debug build is missing (run __graft_entry__.build())"
    return q.open_library(q.DEBUG_LIB_PATH)


def _one_byte_of(q, c, r0, j0):
    """Offset of the packed byte that holds trit (r0, j0): the one byte of
    the packed-trit region (16 bytes per row and group of 16 packs) in
    which two packings differing only in that trit differ."""
    import torch

    pm = gpu_pack(c)
    t2 = c["trits"].copy()
    t2[r0, j0] = (t2[r0, j0] + 2) % 3 - 1
    pm2 = gpu_pack(dict(c, trits=t2))
    d = pm.desc
    lo, hi = int(d.off_trits), int(d.off_trits + d.n_pad * d.n_groups * 16)
    diff = torch.nonzero(pm.packed[lo:hi] != pm2.packed[lo:hi]).flatten()
    assert diff.numel() == 1, diff.numel()
    return pm, lo + int(diff[0].item())


@pytest.mark.parametrize("B", [1, 4])
def test_debug_build_nan_rows_for_invalid_codes(debug_lib, B):
    import torch

    import paper_2609_00224_amd as q

    N, K, r0, j0 = 256, 333, 101, 200
    c = dyadic_case(77 + B, N, K, B, 5)
    pm, off = _one_byte_of(q, c, r0, j0)
    bad = pm.packed.clone()
    bad[off] = 250
    ref, _ = oracle_rows(c, need_wmax=False)
    x = to_dev(c["x"])
    print(f"[case] debug build, B={B}, byte {off} set to 250", flush=True)
    saved = q._lib
    q._lib = debug_lib
    try:
        for packed, corrupt in ((pm.packed, False), (bad, True)):
            m = q.PackedMatrix(pm.desc, packed)
            y1 = torch.full((B, N), 7.0, dtype=torch.float32, device="cuda")
            q.qtea_gemm_lowbatch(pm.desc, packed, x, B, y1, q.new_workspace(pm.desc, B))
            yg = torch.full((B, N), 7.0, dtype=torch.float32, device="cuda")
            gp = q.plan_grouped([m], [x], [yg], batch=B)
            gp.run()
            torch.cuda.synchronize()
            for what, y in (("per matrix", y1), ("grouped", yg)):
                got = y.cpu().numpy().astype(np.float64)
                others = np.arange(N) != r0
                assert np.array_equal(got[:, others], ref[:, others]), (what, corrupt)
                if corrupt:
                    assert np.all(np.isnan(got[:, r0])), (what, got[:, r0])
                else:
                    assert np.array_equal(got[:, r0], ref[:, r0]), what
    finally:
        q._lib = saved
