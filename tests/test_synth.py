"""The seeded generator: published SplitMix64 outputs, determinism, and the
distributions the workloads ask for."""
from __future__ import annotations

from fractions import Fraction

import numpy as np
import pytest

import synth
from synth.workloads import WORKLOADS


def test_splitmix64_published_sequence():
    # First outputs of SplitMix64 seeded with 0 (the reference C code of
    # Steele et al. / Vigna's splitmix64.c): counter-mode element i equals
    # the (i+1)-th sequential output.
    assert synth.sm64_at(0, 0) == 0xE220A8397B1DCDAF
    assert synth.sm64_at(0, 1) == 0x6E789E6AA1B965F4
    assert synth.sm64_at(0, 2) == 0x06C45D188009454F


def test_thresholds_and_counts():
    assert synth.trit_thresholds(Fraction(2, 5)) == (1288490188, 3006477107)
    assert synth.trit_thresholds(Fraction(1, 2)) == (1073741824, 3221225472)
    for K, f, n in [(4096, Fraction(2, 100), 82), (14336, Fraction(2, 100), 287),
                    (5120, Fraction(3, 100), 154), (17408, Fraction(3, 100), 522),
                    (8192, Fraction(2, 100), 164), (28672, Fraction(2, 100), 573)]:
        assert synth.n_salient(K, f) == n


def test_deterministic_and_row_subsets():
    a = synth.trits(1, 2, 3, 64, 77, Fraction(2, 5))
    b = synth.trits(1, 2, 3, 64, 77, Fraction(2, 5))
    assert np.array_equal(a, b)
    rows = np.array([63, 0, 5, 5], np.int64)
    assert np.array_equal(synth.trits(1, 2, 3, 64, 77, Fraction(2, 5), rows=rows), a[rows])
    c = synth.trits(1, 2, 4, 64, 77, Fraction(2, 5))
    assert not np.array_equal(a, c)
    d = synth.trits(1, 3, 3, 64, 77, Fraction(2, 5))
    assert not np.array_equal(a, d)


@pytest.mark.parametrize("p0", [Fraction(2, 5), Fraction(1, 2)])
def test_trit_distribution(p0):
    t = synth.trits(9, 0, 0, 512, 1000, p0)
    n = t.size
    z = np.count_nonzero(t == 0) / n
    assert set(np.unique(t).tolist()) == {-1, 0, 1}
    assert abs(z - float(p0)) < 5 * np.sqrt(float(p0) * (1 - float(p0)) / n)
    pm = (1 - float(p0)) / 2
    assert abs(np.count_nonzero(t == 1) / n - pm) < 5 * np.sqrt(pm * (1 - pm) / n)


def test_layer_inputs_shapes_and_ranges():
    L = synth.layer_inputs(1, 0, 0, 256, 4096)
    assert L["S"].size == 82 and np.all(np.diff(L["S"]) > 0)
    assert L["S"].min() >= 0 and L["S"].max() < 4096
    assert L["R"].shape == (82, 64) and L["idx"].shape == (82, 64)
    assert L["idx"].max() <= 3 and np.unique(L["idx"]).size == 4
    a = L["alpha"].astype(np.float64)
    v = L["v"].astype(np.float64)
    assert a.min() >= 0.0099 and a.max() <= 0.0301
    assert v.min() >= 0.799 and v.max() <= 1.201
    assert abs(L["R"].astype(np.float64).std() - 0.01) < 0.001
    x = synth.activations(1, 0, 0, 4, 4096).astype(np.float64)
    assert x.shape == (4, 4096)
    assert abs(x.mean()) < 0.05 and abs(x.std() - 1.0) < 0.05


def st_shapes():
    return WORKLOADS["llama3_8b_stack"].shapes


def test_workload_table():
    assert [w for w in WORKLOADS] == ["gemv_4096x4096", "llama3_8b_layer", "llama3_8b_stack",
                                      "qwen3_14b_stack", "llama3_70b_stack", "llama3_8b_stack_e4m3",
                                      "llama3_8b_stack_g128"]
    g = WORKLOADS["llama3_8b_stack_g128"]
    assert g.groups == 128 and g.resid == "e4m3" and g.frac == Fraction(5, 100)
    e8 = WORKLOADS["llama3_8b_stack_e4m3"]
    assert e8.resid == "e4m3" and e8.frac == Fraction(5, 100) and e8.shapes == st_shapes()
    assert all(WORKLOADS[n].resid == "fp16" for n in list(WORKLOADS)[:5])
    st = WORKLOADS["llama3_8b_stack"]
    assert st.layers == 32 and len(list(st.matrices())) == 128
    assert WORKLOADS["llama3_70b_stack"].p0 == Fraction(1, 2)
    assert WORKLOADS["qwen3_14b_stack"].frac == Fraction(3, 100)


def test_e4m3_residual_inputs():
    import oracle

    L = synth.layer_inputs(3, 1, 2, 256, 4096, frac=Fraction(5, 100), resid="e4m3")
    nS = synth.n_salient(4096, Fraction(5, 100))
    assert nS == 205 and L["S"].size == nS and "R" not in L
    assert L["R8"].dtype == np.uint8 and L["R8"].shape == (nS, 64)
    assert not np.any((L["R8"] & 0x7F) == 0x7F)  # no NaN codes
    assert L["bitmap"].dtype == np.int32 and L["bitmap"].size == 128
    assert np.array_equal(oracle.bitmap_to_list(L["bitmap"], 4096), L["S"])
    # the codes are the fp64 draw rounded to E4M3: within half an E4M3 step
    # of the fp16 rounding of the same draw
    R16 = synth.layer_inputs(3, 1, 2, 256, 4096, frac=Fraction(5, 100))["R"].astype(np.float64)
    R8 = oracle.e4m3_decode(L["R8"])
    step = np.maximum(2.0 ** (np.floor(np.log2(np.maximum(np.abs(R16), 2.0 ** -6))) - 3), 2.0 ** -9)
    assert np.all(np.abs(R8 - R16) <= 0.5 * step + 2.0 ** -12)


def test_group128_inputs():
    L = synth.layer_inputs(4, 0, 1, 64, 300, groups=128)
    assert L["alpha_g"].shape == (64, 3) and L["beta_g"].shape == (64, 3)
    a, b = L["alpha_g"].astype(np.float64), L["beta_g"].astype(np.float64)
    assert a.min() >= 0.0099 and a.max() <= 0.0301
    assert b.min() >= -0.00501 and b.max() <= 0.00501 and (b < 0).any() and (b > 0).any()
    assert np.array_equal(L["trits"], synth.layer_inputs(4, 0, 1, 64, 300)["trits"])
