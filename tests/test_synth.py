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


def test_workload_table():
    assert [w for w in WORKLOADS] == ["gemv_4096x4096", "llama3_8b_layer", "llama3_8b_stack",
                                      "qwen3_14b_stack", "llama3_70b_stack"]
    st = WORKLOADS["llama3_8b_stack"]
    assert st.layers == 32 and len(list(st.matrices())) == 128
    assert WORKLOADS["llama3_70b_stack"].p0 == Fraction(1, 2)
    assert WORKLOADS["qwen3_14b_stack"].frac == Fraction(3, 100)
