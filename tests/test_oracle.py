"""Pins of the fp64 CPU oracle against facts fixed by the paper and by
mathematics, never against the oracle itself.

Paper passages: "Efficient Ternary Computation" (Eq. 10, Eq. 11, the 3^5 < 2^8
packing, the sign symmetry of the table, the residual storage format), the
experimental setup (1.7 bits per weight) and the hardware appendix (26 bytes
per 128 columns, 9.85x smaller than FP16).
"""
from __future__ import annotations

import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from tests.golden import load_worked_example


# --------------------------------------------------------------------------
# fp16 -> fp64 conversion: every one of the 65536 bit patterns against
# numpy's binary16 (a library routine).
# --------------------------------------------------------------------------
def test_half_to_double_all_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([oracle.half_to_double(int(b)) for b in bits])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # signed zeros keep their sign
    assert math.copysign(1.0, oracle.half_to_double(0x8000)) == -1.0


# --------------------------------------------------------------------------
# Base-3 byte codes (3^5 = 243 < 256 five-trit patterns per byte).
# --------------------------------------------------------------------------
ALL_PATTERNS = list(itertools.product((-1, 0, 1), repeat=5))


def test_all_243_codes_round_trip():
    seen = set()
    for t in ALL_PATTERNS:
        c = oracle.encode5(np.array(t, np.int8))
        assert 0 <= c < 243
        seen.add(c)
        back = oracle.decode_code(c)
        assert tuple(int(v) for v in back) == t
    assert seen == set(range(243))  # a bijection onto 0..242
    for c in range(243):
        assert set(int(v) for v in oracle.decode_code(c)) <= {-1, 0, 1}


@pytest.mark.parametrize("c", list(range(243, 256)) + [-1, 1000])
def test_invalid_codes_rejected(c):
    with pytest.raises(oracle.OracleError) as e:
        oracle.decode_code(c)
    assert e.value.rc == oracle.ERR_CODE


def test_code_closed_forms():
    # the all-zero pattern is code 121 = 1 + 3 + 9 + 27 + 81
    assert oracle.encode5(np.zeros(5, np.int8)) == 121
    # sign symmetry of the table: pattern -p has code 242 - code(p)
    for t in ALL_PATTERNS:
        c = oracle.encode5(np.array(t, np.int8))
        cn = oracle.encode5(-np.array(t, np.int8))
        assert cn == 242 - c
    # digit order: column 5p + i is base-3 digit i (least significant first)
    assert oracle.encode5(np.array([1, 0, 0, 0, 0], np.int8)) == 122
    assert oracle.encode5(np.array([0, 0, 0, 0, 1], np.int8)) == 121 + 81
    assert oracle.encode5(np.array([-1] * 5, np.int8)) == 0
    assert oracle.encode5(np.array([1] * 5, np.int8)) == 242
    assert oracle.encode5(np.array([0, -1, 0, 0, 0], np.int8)) == 121 - 3


def test_bad_trit_rejected():
    assert oracle.encode5(np.array([0, 2, 0, 0, 0], np.int8)) == oracle.ERR_TRIT
    with pytest.raises(oracle.OracleError) as e:
        oracle.pack(np.array([[0, 0, -2]], np.int8))
    assert e.value.rc == oracle.ERR_TRIT


@pytest.mark.parametrize("K", [1, 2, 4, 5, 6, 9, 10, 11, 37])
def test_pack_padding_is_zero_trit(K):
    rng = np.random.default_rng(K)
    T = rng.integers(-1, 2, size=(3, K)).astype(np.int8)
    P = oracle.pack(T)
    assert P.shape == (3, (K + 4) // 5)
    # brute force: integer base-3 sum with the zero trit in the padding
    for r in range(3):
        for p in range(P.shape[1]):
            digits = [(int(T[r, 5 * p + i]) if 5 * p + i < K else 0) + 1 for i in range(5)]
            assert P[r, p] == sum(d * 3 ** i for i, d in enumerate(digits))
    assert np.array_equal(oracle.unpack(P, K), T)


def test_single_column_codes():
    # K = 1: one byte whose upper four digits are the padding zero trit
    assert oracle.pack(np.array([[1]], np.int8))[0, 0] == 122
    assert oracle.pack(np.array([[0]], np.int8))[0, 0] == 121
    assert oracle.pack(np.array([[-1]], np.int8))[0, 0] == 120


def test_unpack_rejects_nonzero_padding_and_bad_bytes():
    # K = 6: second byte may only use digit 0; 121 + 3 puts a +1 in column 6
    with pytest.raises(oracle.OracleError) as e:
        oracle.unpack(np.array([[121, 124]], np.uint8), 6)
    assert e.value.rc == oracle.ERR_CODE
    with pytest.raises(oracle.OracleError) as e:
        oracle.unpack(np.array([[243]], np.uint8), 5)
    assert e.value.rc == oracle.ERR_CODE


# --------------------------------------------------------------------------
# Hand-worked example (tests/golden), Eq. 10 + Eq. 11.
# --------------------------------------------------------------------------
def test_worked_example_codes_and_output():
    w = load_worked_example()
    P = oracle.pack(w["trits"])
    assert np.array_equal(P, w["codes"])
    args = (w["N"], w["K"], P, w["alpha"], w["v"], w["S"], w["R"], w["idx"], w["x"])
    assert np.array_equal(oracle.gemv(*args), w["y"])
    assert np.array_equal(oracle.gemv_lut(*args), w["y"])


# --------------------------------------------------------------------------
# Residual storage: one value and one 2-bit position per group of four
# entries of a salient column.
# --------------------------------------------------------------------------
def test_resid_rows_one_per_group():
    rng = np.random.default_rng(7)
    N, nS = 64, 5
    idx = rng.integers(0, 4, size=(nS, N // 4)).astype(np.uint8)
    rows = oracle.resid_rows(idx, N)
    for s in range(nS):
        for g in range(N // 4):
            assert 4 * g <= rows[s, g] < 4 * g + 4
            assert rows[s, g] - 4 * g == idx[s, g]
        # each group contributes exactly one row: the rows are distinct
        assert len(set(rows[s].tolist())) == N // 4
    idx[2, 3] = 4
    with pytest.raises(oracle.OracleError) as e:
        oracle.resid_rows(idx, N)
    assert e.value.rc == oracle.ERR_RESID


def test_salient_list_checks():
    assert oracle.check_salient([0, 3, 9], 10) == oracle.OK
    assert oracle.check_salient([], 10) == oracle.OK
    assert oracle.check_salient([3, 3], 10) == oracle.ERR_RESID
    assert oracle.check_salient([4, 2], 10) == oracle.ERR_RESID
    assert oracle.check_salient([10], 10) == oracle.ERR_RESID
    assert oracle.check_salient([-1], 10) == oracle.ERR_RESID


# --------------------------------------------------------------------------
# Brute force in exact rational arithmetic on tiny dyadic inputs: the plain
# route and the table route of the oracle both equal the exact value.
# --------------------------------------------------------------------------
def _dyadic_case(rng, N, K, B, nS):
    T = rng.integers(-1, 2, size=(N, K)).astype(np.int8)
    alpha = (2.0 ** -rng.integers(0, 6, size=N)).astype(np.float16)
    v = rng.choice([0.5, 1.0, 1.5, 2.0], size=K).astype(np.float16)
    x = (rng.integers(-8, 9, size=(B, K)) / 4.0).astype(np.float16)
    S = np.sort(rng.choice(K, size=nS, replace=False)).astype(np.int32)
    R = (rng.integers(-64, 65, size=(nS, N // 4)) / 64.0).astype(np.float16)
    idx = rng.integers(0, 4, size=(nS, N // 4)).astype(np.uint8)
    return T, alpha, v, x, S, R, idx


def _exact(T, alpha, v, x, S, R, idx):
    """Eq. 10 (one group, beta = 0) plus Eq. 11 in Python Fractions."""
    N, K = T.shape
    F = lambda h: Fraction(float(h))
    out = []
    for b in range(x.shape[0]):
        yb = []
        for r in range(N):
            tern = sum(int(T[r, j]) * F(v[j]) * F(x[b, j]) for j in range(K))
            res = sum(F(R[s, r // 4]) * F(x[b, S[s]]) for s in range(len(S)) if idx[s, r // 4] == r % 4)
            yb.append(F(alpha[r]) * tern + res)
        out.append(yb)
    return out


@pytest.mark.parametrize("N,K,B,nS", [(4, 1, 1, 0), (4, 5, 2, 1), (8, 7, 3, 2), (8, 12, 1, 3),
                                      (12, 37, 2, 5), (16, 10, 4, 10)])
def test_brute_force_exact(N, K, B, nS):
    rng = np.random.default_rng(N * 1000 + K)
    T, alpha, v, x, S, R, idx = _dyadic_case(rng, N, K, B, nS)
    P = oracle.pack(T)
    exact = _exact(T, alpha, v, x, S, R, idx)
    y = oracle.gemv(N, K, P, alpha, v, S, R, idx, x)
    yl = oracle.gemv_lut(N, K, P, alpha, v, S, R, idx, x)
    for b in range(B):
        for r in range(N):
            assert Fraction(y[b, r]) == exact[b][r]
            assert Fraction(yl[b, r]) == exact[b][r]


def test_exhaustive_code_shape():
    """K = 5, N = 256: rows 0..242 carry codes 0..242, rows 243..255 are zero.
    With dyadic v, x and no residual, y_r = alpha_r * sum_i t_i(r) v_i x_i."""
    N, K = 256, 5
    P = np.full((N, 1), 121, np.uint8)
    P[:243, 0] = np.arange(243, dtype=np.uint8)
    alpha = (2.0 ** -(np.arange(N) % 4)).astype(np.float16)
    v = np.array([0.5, 1.0, 1.5, 2.0, 0.5], np.float16)
    x = np.array([[1.0, -2.0, 0.25, 4.0, -0.75]], np.float16)
    empty = np.zeros(0, np.int32)
    y = oracle.gemv(N, K, P, alpha, v, empty, np.zeros((0, N // 4)), np.zeros((0, N // 4)), x)
    for r in range(N):
        c = int(P[r, 0])
        t = [(c // 3 ** i) % 3 - 1 for i in range(5)]
        exact = Fraction(float(alpha[r])) * sum(t[i] * Fraction(float(v[i])) * Fraction(float(x[0, i]))
                                                for i in range(5))
        assert Fraction(y[0, r]) == exact


# --------------------------------------------------------------------------
# Textbook special cases.
# --------------------------------------------------------------------------
def _none(N):
    return np.zeros(0, np.int32), np.zeros((0, N // 4), np.float16), np.zeros((0, N // 4), np.uint8)


def test_zero_trits_no_residual_gives_zero():
    rng = np.random.default_rng(3)
    N, K = 16, 23
    P = oracle.pack(np.zeros((N, K), np.int8))
    alpha = rng.uniform(0.01, 0.03, N).astype(np.float16)
    v = rng.uniform(0.8, 1.2, K).astype(np.float16)
    x = rng.standard_normal((2, K)).astype(np.float16)
    y = oracle.gemv(N, K, P, alpha, v, *_none(N), x)
    assert np.all(y == 0.0)


def test_single_trit_is_one_product():
    N, K = 8, 13
    T = np.zeros((N, K), np.int8)
    T[5, 9] = -1
    alpha = np.full(N, 0.0234, np.float16)
    v = np.full(K, 1.1, np.float16)
    x = np.full((1, K), 0.7, np.float16)
    y = oracle.gemv(N, K, oracle.pack(T), alpha, v, *_none(N), x)
    expect = -float(alpha[5]) * float(v[9]) * float(x[0, 9])
    assert y[0, 5] == expect
    assert np.count_nonzero(y) == 1


def test_all_plus_one_sums_x():
    N, K = 4, 31
    rng = np.random.default_rng(11)
    x = rng.standard_normal((1, K)).astype(np.float16)
    y = oracle.gemv(N, K, oracle.pack(np.ones((N, K), np.int8)), np.ones(N, np.float16),
                    np.ones(K, np.float16), *_none(N), x)
    assert np.all(y == math.fsum(float(t) for t in x[0]))


def test_residual_alone_not_scaled_by_alpha_or_v():
    N, K = 12, 9
    S = np.array([6], np.int32)
    R = np.zeros((1, N // 4), np.float16)
    idx = np.zeros((1, N // 4), np.uint8)
    R[0, 2], idx[0, 2] = 0.375, 3  # group 2 -> row 11
    alpha = np.full(N, 0.25, np.float16)
    v = np.full(K, 1.5, np.float16)
    x = np.arange(1, K + 1, dtype=np.float16).reshape(1, K)
    y = oracle.gemv(N, K, oracle.pack(np.zeros((N, K), np.int8)), alpha, v, S, R, idx, x)
    assert y[0, 11] == 0.375 * 7.0
    assert np.count_nonzero(y) == 1


def test_matches_blas_on_dense_rows():
    """numpy's BLAS matrix-vector product on the oracle's dense rows."""
    rng = np.random.default_rng(5)
    N, K, B, nS = 40, 53, 3, 4
    T = rng.integers(-1, 2, size=(N, K)).astype(np.int8)
    alpha = rng.uniform(0.01, 0.03, N).astype(np.float16)
    v = rng.uniform(0.8, 1.2, K).astype(np.float16)
    x = rng.standard_normal((B, K)).astype(np.float16)
    S = np.sort(rng.choice(K, nS, replace=False)).astype(np.int32)
    R = (rng.standard_normal((nS, N // 4)) * 0.01).astype(np.float16)
    idx = rng.integers(0, 4, (nS, N // 4)).astype(np.uint8)
    P = oracle.pack(T)
    W = oracle.dense_rows(N, K, P, alpha, v, S, R, idx)
    # the dense rows themselves: alpha v t everywhere but the residual spots
    rr = oracle.resid_rows(idx, N)
    mask = np.ones((N, K), bool)
    for s in range(nS):
        mask[rr[s], S[s]] = False
    base = alpha.astype(np.float64)[:, None] * v.astype(np.float64)[None, :] * T
    assert np.array_equal(W[mask], base[mask])
    y = oracle.gemv(N, K, P, alpha, v, S, R, idx, x)
    ref = x.astype(np.float64) @ W.T
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-14)
    # non-square: transposing W would not even conform
    rows = np.array([39, 0, 17], np.int64)
    ys = oracle.gemv(N, K, P[rows], alpha, v, S, R, idx, x, rows=rows)
    assert np.array_equal(ys, y[:, rows])


# --------------------------------------------------------------------------
# Storage arithmetic printed in the paper.
# --------------------------------------------------------------------------
def test_bits_per_weight_paper_figures():
    # setup section: 1.6 bpw ternary + 5% columns x 8-bit value / 4 = 1.7
    assert oracle.bpw_paper(0.05, 8) == pytest.approx(1.7, abs=1e-12)
    # appendix: 26 one-byte packs per 128-column group -> 1.625 bpw, 9.85x vs FP16
    assert oracle.num_packs(128) == 26
    assert round(16 / (8 * oracle.num_packs(128) / 128), 2) == 9.85
    # 5% of columns at one value per four entries is 1.25% of the weights
    assert 0.05 / 4 == pytest.approx(0.0125)


def test_bits_per_weight_full_accounting():
    # all terms counted: trits, residual value + position, bitmap, alpha, v
    N, K, nS = 4096, 4096, 82
    bits = 8 * N * 820 + (N // 4) * nS * 18 + K + 16 * N + 16 * K
    assert oracle.bpw_full(N, K, nS) == pytest.approx(bits / (N * K), rel=1e-15)
    assert round(oracle.bpw_full(N, K, nS), 4) == 1.6997
    # no salient columns and K a multiple of 5: trits + scales only
    assert oracle.bpw_full(100, 1000, 0) == pytest.approx((8 * 100 * 200 + 1000 + 1600 + 16000) / 1e5)


@pytest.mark.parametrize("N,K,nS,expect", [
    (6144, 4096, 82, 5_342_280), (4096, 4096, 82, 3_564_360), (28672, 4096, 82, 24_899_400),
    (4096, 14336, 287, 12_446_588), (7168, 5120, 154, 7_986_152), (5120, 5120, 154, 5_707_496),
    (34816, 5120, 154, 38_748_008), (5120, 17408, 522, 19_378_344), (10240, 8192, 164, 17_765_520),
    (8192, 8192, 164, 14_215_824), (57344, 8192, 164, 99_408_528), (8192, 28672, 573, 49_697_524),
])
def test_algorithmic_bytes_per_shape(N, K, nS, expect):
    assert oracle.algorithmic_bytes(N, K, nS) == expect


# ---------------------------------------------------------------------------
# The paper's residual storage: FP8 E4M3 values and a salient column bitmap.
# ---------------------------------------------------------------------------
def test_e4m3_matches_library_routine_all_codes():
    """All 256 codes against torch's float8_e4m3fn (an independent
    implementation of the same OCP format)."""
    import torch

    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = oracle.e4m3_decode(codes)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert set(np.flatnonzero(nan)) == {0x7F, 0xFF}
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def test_e4m3_closed_forms():
    f = oracle.e4m3_to_double
    assert f(0x00) == 0.0 and math.copysign(1.0, f(0x80)) == -1.0
    assert f(0x38) == 1.0          # exponent field 7 = bias: 2^0
    assert f(0x3C) == 1.5          # mantissa 4/8
    assert f(0x7E) == 448.0        # largest finite: 1.75 * 2^8
    assert f(0x08) == 2.0 ** -6    # smallest normal
    assert f(0x01) == 2.0 ** -9    # smallest subnormal: 1/8 * 2^-6
    assert f(0x07) == 7 * 2.0 ** -9
    assert f(0xB8) == -1.0


def test_e4m3_order_sign_and_fp16_exactness():
    pos = oracle.e4m3_decode(np.arange(0x7F, dtype=np.uint8))  # 0x00..0x7e, finite
    assert np.all(np.diff(pos) > 0)  # strictly increasing with the code
    neg = oracle.e4m3_decode(np.arange(0x80, 0xFF, dtype=np.uint8))
    assert np.array_equal(neg, -pos)
    # every finite value is an fp16 value
    h = oracle.e4m3_as_half(np.arange(0x7F, dtype=np.uint8))
    assert np.array_equal(h.astype(np.float64), pos)
    with pytest.raises(oracle.OracleError):
        oracle.e4m3_as_half(np.array([0x7F], dtype=np.uint8))


@pytest.mark.parametrize("K", [1, 31, 32, 33, 100, 4096, 14337])
def test_bitmap_to_list_brute_force(K):
    rng = np.random.default_rng(K)
    S = np.sort(rng.choice(K, size=max(1, K // 20), replace=False)).astype(np.int32)
    words = np.zeros((K + 31) // 32, dtype=np.uint32)
    for j in S:  # brute force, one bit at a time
        words[j // 32] |= np.uint32(1) << np.uint32(j % 32)
    assert np.array_equal(oracle.bitmap_to_list(words, K), S)
    assert np.array_equal(oracle.bitmap_to_list(np.zeros_like(words), K), np.zeros(0, np.int32))


def test_bitmap_bit_past_K_rejected():
    with pytest.raises(oracle.OracleError):
        oracle.bitmap_to_list(np.array([1 << 5], dtype=np.uint32), 5)
    assert np.array_equal(oracle.bitmap_to_list(np.array([1 << 4], dtype=np.uint32), 5), [4])


def test_e4m3_storage_bytes():
    # one byte per value instead of two: the residual value bytes halve
    for N, K, nS in [(4096, 4096, 205), (28672, 4096, 205), (4096, 14336, 717)]:
        b16, b8 = oracle.algorithmic_bytes_vb(N, K, nS, 2), oracle.algorithmic_bytes_vb(N, K, nS, 1)
        assert b16 == oracle.algorithmic_bytes(N, K, nS)
        assert b16 - b8 == (N // 4) * nS
    # the paper's setting: 5% of columns, 8-bit values, one per four entries
    assert oracle.bpw_paper(0.05, 8) == pytest.approx(1.7, abs=1e-12)


# ---------------------------------------------------------------------------
# The paper's 128-column quantization groups: per-group alpha and beta,
# 26 bytes per row and group.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("K", [1, 5, 127, 128, 129, 300, 1000])
def test_pack128_round_trip_and_padding(K):
    rng = np.random.default_rng(K)
    T = rng.integers(-1, 2, size=(3, K)).astype(np.int8)
    P = oracle.pack128(T)
    ng = (K + 127) // 128
    assert P.shape == (3, 26 * ng) and P.max() < 243
    assert np.array_equal(oracle.unpack128(P, K), T)
    # byte 25 of a group holds its columns 125..127 and two zero trits: digits 3, 4 are 1
    assert np.all(P[:, 25::26] // 27 == 4)
    # columns past K are zero trits: a group with none of its columns left
    # never occurs, and a fully padded byte is the all-zero code 121
    for g in range(ng):
        for p in range(26):
            if 128 * g + 5 * p >= K:
                assert np.all(P[:, 26 * g + p] == 121)
    # first byte of every group: its columns 0..4 in base 3, least significant first
    for g in range(ng):
        cols = [128 * g + i for i in range(5)]
        want = sum((int(T[0, j]) + 1 if j < K else 1) * 3 ** i for i, j in enumerate(cols))
        assert P[0, 26 * g] == want


def test_pack128_bits_per_weight():
    # 26 one-byte packs per 128 columns: 1.625 bits per weight, 9.85x below fp16
    assert oracle.pack128(np.zeros((1, 128), np.int8)).shape[1] == 26
    assert 8 * 26 / 128 == 1.625 and round(16 / 1.625, 2) == 9.85


def _g128_dyadic(seed, N, K, B, nS):
    rng = np.random.default_rng(seed)
    ng = (K + 127) // 128
    S = np.sort(rng.choice(K, size=nS, replace=False)).astype(np.int32) if nS else np.zeros(0, np.int32)
    return {
        "T": rng.integers(-1, 2, size=(N, K)).astype(np.int8),
        "alpha": (2.0 ** -rng.integers(0, 6, size=(N, ng))).astype(np.float16),
        "beta": (rng.integers(-8, 9, size=(N, ng)) / 64.0).astype(np.float16),
        "v": rng.choice([0.5, 1.0, 1.5, 2.0], size=K).astype(np.float16),
        "S": S,
        "R": (rng.integers(-64, 65, size=(nS, N // 4)) / 64.0).astype(np.float16),
        "idx": rng.integers(0, 4, size=(nS, N // 4)).astype(np.uint8),
        "x": (rng.integers(-8, 9, size=(B, K)) / 4.0).astype(np.float16),
    }


def _g128(c, N, K, **kw):
    return oracle.gemv128(N, K, oracle.pack128(c["T"]), c["alpha"], c["beta"], c["v"], c["S"], c["R"],
                          c["idx"], c["x"], **kw)


@pytest.mark.parametrize("N,K,B,nS", [(8, 130, 2, 3), (4, 128, 1, 0), (12, 300, 3, 5), (4, 7, 2, 1)])
def test_gemv128_brute_force_exact(N, K, B, nS):
    """Exact rational arithmetic, term by term from Eq. 10 and Eq. 11."""
    c = _g128_dyadic(N * K + B, N, K, B, nS)
    Fr = lambda h: Fraction(float(h))
    want = np.zeros((B, N), dtype=object)
    for b in range(B):
        for r in range(N):
            tot = Fraction(0)
            for g in range((K + 127) // 128):
                cols = range(128 * g, min(128 * g + 128, K))
                tv = sum(int(c["T"][r, j]) * Fr(c["v"][j]) * Fr(c["x"][b, j]) for j in cols)
                xs = sum(Fr(c["x"][b, j]) for j in cols)
                tot += Fr(c["alpha"][r, g]) * tv + Fr(c["beta"][r, g]) * xs
            for s in range(nS):
                if c["idx"][s, r // 4] == r % 4:
                    tot += Fr(c["R"][s, r // 4]) * Fr(c["x"][b, c["S"][s]])
            want[b, r] = tot
    got = _g128(c, N, K)
    assert all(Fraction(got[b, r]) == want[b, r] for b in range(B) for r in range(N))


def test_gemv128_one_scale_per_row_is_the_single_group_product():
    """alpha_{r,g} = alpha_r for every g and beta = 0 reduces to Eq. 10 with
    one group: the single-group oracle (other packing, other sum order) gives
    the same values exactly on dyadic inputs."""
    N, K, B, nS = 16, 1000, 2, 9
    c = _g128_dyadic(5, N, K, B, nS)
    c["alpha"] = np.repeat(c["alpha"][:, :1], c["alpha"].shape[1], axis=1)
    c["beta"] = np.zeros_like(c["beta"])
    y128 = _g128(c, N, K)
    y1 = oracle.gemv(N, K, oracle.pack(c["T"]), c["alpha"][:, 0], c["v"], c["S"], c["R"], c["idx"], c["x"])
    assert np.array_equal(y128, y1)


def test_gemv128_bias_alone_is_the_group_sums():
    N, K, B = 8, 300, 2
    c = _g128_dyadic(6, N, K, B, 0)
    c["T"][:] = 0
    y = _g128(c, N, K)
    xg = np.zeros((B, 3))
    xpad = np.zeros((B, 384))
    xpad[:, :K] = c["x"].astype(np.float64)
    xg = xpad.reshape(B, 3, 128).sum(axis=2)  # per-group activation sums
    want = xg @ c["beta"].astype(np.float64).T
    assert np.array_equal(y, want)


def test_gemv128_rows_subset_and_sign():
    N, K, B, nS = 12, 260, 2, 4
    c = _g128_dyadic(8, N, K, B, nS)
    full = _g128(c, N, K)
    rows = np.array([11, 0, 5], dtype=np.int64)
    part = oracle.gemv128(N, K, oracle.pack128(c["T"][rows]), c["alpha"], c["beta"], c["v"], c["S"], c["R"],
                          c["idx"], c["x"], rows=rows)
    assert np.array_equal(part, full[:, rows])
    neg = dict(c, alpha=-c["alpha"], beta=-c["beta"], R=-c["R"])
    assert np.array_equal(_g128(neg, N, K), -full)


def test_algorithmic_bytes128():
    # 8B-shaped gate_up, 5% E4M3 residual: 26 bytes per row and group plus 4 bytes of scales
    N, K, nS = 28672, 4096, 205
    b = oracle.algorithmic_bytes128(N, K, nS, 1)
    assert b == N * 32 * 26 + 4 * N * 32 + (N // 4) * nS + ((N // 4) * nS * 2 + 7) // 8 + 2 * K + 4 * nS
