"""Pins of the quantizer oracle (oracle/quantizer.py) against facts that do
not come from the oracle itself:

  * the GPTQ propagation (Cholesky factor, lazy blocks, decay) against an
    independent sequential form that re-derives the inverse Hessian of the
    remaining columns by a fresh matrix inverse at every column;
  * lambda = 0 reduces error decay to the plain GPTQ update (the paper's
    own statement), gamma at the first column of a block is 1 and gamma at
    the middle of a block with d equal to the mean is exp(-lambda / 2);
  * with an identity Hessian nothing propagates: every code is the nearest
    of the three points, found by brute force;
  * a matrix that is exactly beta + c alpha t is reproduced exactly;
  * the E4M3 rounding against torch's float8_e4m3fn conversion and the
    format's tie and saturation rules;
  * the salient score of Eq. 3 on hand-derived cases whose choice flips
    under a mean over rows, diag(H) to the first power, or |W| in place of
    W^2; the salient set is the subset of that size with the largest score
    sum (brute force over subsets) and is invariant under row permutations
    and positive scalings;
  * the Hessian against explicit sums; the 1:4 residual structure; and the
    GPTQ result's Hessian-weighted error below round-to-nearest.
"""
from __future__ import annotations

import itertools
import math

import numpy as np
import pytest

import oracle
from oracle import quantizer as qz


def _spd(rng, K, n=None):
    """A correlated positive definite Hessian from synthetic calibration rows."""
    n = n or 4 * K
    mix = rng.normal(size=(K, K)) * 0.3 + np.eye(K)
    X = rng.normal(size=(n, K)) @ mix
    return qz.hessian(X)


def _obs_quantize(W, H, n_salient, lam, iters, group):
    """Sequential form: at column j the inverse Hessian of the remaining
    columns is inv(H[j:, j:]) (the Schur-complement identity), computed
    afresh; the error and its decayed update follow from it directly."""
    W = np.array(W, dtype=np.float64, copy=True)
    N, K = W.shape
    S = qz.select_salient(qz.salient_scores(W, H), n_salient)
    Hd, _, dead = qz.inv_hessian_factor(H)
    W[:, dead] = 0.0
    dfac = np.array([math.sqrt(np.linalg.inv(Hd[j:, j:])[0, 0]) for j in range(K)])
    T = np.zeros((N, K), np.int8)
    Q = np.zeros((N, K))
    v = np.ones(K)
    for b0 in range(0, K, group):
        b1 = min(K, b0 + group)
        ab = [qz.group_params(W[r, b0:b1]) for r in range(N)]
        al = np.array([a for a, _ in ab])
        be = np.array([b for _, b in ab])
        dmean = dfac[b0:b1].mean()
        for j in range(b0, b1):
            Hinv = np.linalg.inv(Hd[j:, j:])
            w = W[:, j].copy()
            t, vj, q, _, _ = qz.quantize_column(w, al, be, iters, j in set(S.tolist()))
            T[:, j], v[j], Q[:, j] = t, vj, q
            gamma = math.exp(-lam * (dfac[j] / dmean) * ((j - b0) / (b1 - b0)))
            W[:, j + 1:] -= gamma * np.outer((w - q) / Hinv[0, 0], Hinv[0, 1:])
    return T, Q, v


@pytest.mark.parametrize("lam,iters,nS", [(0.0, 0, 0), (0.0, 2, 2), (1.0, 2, 2), (3.0, 1, 3), (1e6, 2, 0)])
def test_gptq_matches_sequential_inverse_form(lam, iters, nS):
    rng = np.random.default_rng(7 + int(lam) + 10 * iters + 100 * nS)
    N, K, group = 8, 13, 4
    W = rng.normal(size=(N, K)) * 0.02
    H = _spd(rng, K)
    out = qz.quantize(W, H, nS, lam=lam, iters=iters, group=group)
    T, Q, v = _obs_quantize(W, H, nS, lam, iters, group)
    np.testing.assert_array_equal(out["T"], T)
    np.testing.assert_array_equal(out["v"], v)
    np.testing.assert_allclose(out["Q"], Q, rtol=0, atol=1e-12)


def test_decay_closed_forms():
    assert qz.decay(0.0, 3.0, 1.0, 100, 128) == 1.0  # lambda = 0: the GPTQ update
    assert qz.decay(5.0, 3.0, 1.0, 0, 128) == 1.0    # first column of a block
    assert qz.decay(1.0, 2.0, 2.0, 64, 128) == pytest.approx(0.6065306597126334, abs=1e-15)  # e^-1/2
    g = [qz.decay(1.0, 1.0, 1.0, i, 128) for i in range(128)]
    assert all(a > b for a, b in zip(g, g[1:]))


def test_decay_large_lambda_stops_all_but_first_column():
    """lambda -> infinity: only each block's first column still propagates
    (gamma = 1 there); the result matches the sequential form and differs
    from the undecayed one."""
    rng = np.random.default_rng(3)
    N, K, group = 8, 8, 4
    H = _spd(rng, K)
    W = rng.normal(size=(N, K)) * 0.02
    out_big = qz.quantize(W, H, 0, lam=1e9, iters=2, group=group)
    # the same quantization with propagation only from columns 0 and 4
    T, Q, _ = _obs_quantize(W, H, 0, 1e9, 2, group)
    np.testing.assert_array_equal(out_big["T"], T)
    np.testing.assert_allclose(out_big["Q"], Q, rtol=0, atol=1e-12)
    assert np.abs(out_big["Q"] - qz.quantize(W, H, 0, lam=0.0, iters=2, group=group)["Q"]).max() > 0


def test_identity_hessian_is_nearest_point():
    rng = np.random.default_rng(11)
    N, K = 16, 40
    W = rng.normal(size=(N, K)) * 0.02
    out = qz.quantize(W, np.eye(K) * 2.0, 0, lam=1.0, iters=2, group=16)
    for j in range(K):
        g = j // 16
        for r in range(N):
            a, b, vj = out["alpha"][r, g], out["beta"][r, g], out["v"][j]
            pts = [b - vj * a, b, b + vj * a]
            dist = [abs(W[r, j] - p) for p in pts]
            assert out["T"][r, j] == int(np.argmin(dist)) - 1
            assert out["Q"][r, j] == pts[out["T"][r, j] + 1]


def test_exact_ternary_matrix_is_reproduced():
    """W = beta + 0.75 alpha t with fp16-exact alpha, beta and every group
    holding each code equally often (so the first assignment is already t):
    zero error, no propagation, even with a full Hessian."""
    rng = np.random.default_rng(5)
    N, K, group = 8, 24, 6
    G = K // group
    al = 2.0 ** -rng.integers(4, 8, size=(N, G))
    be = rng.integers(-8, 9, size=(N, G)) * 2.0 ** -10
    t = np.concatenate([np.stack([rng.permutation([-1, -1, 0, 0, 1, 1]) for _ in range(G)]).reshape(-1)
                        for _ in range(N)]).reshape(N, K)
    W = np.repeat(be, group, axis=1) + 0.75 * np.repeat(al, group, axis=1) * t
    out = qz.quantize(W, _spd(rng, K), 0, lam=1.0, iters=2, group=group)
    np.testing.assert_array_equal(out["T"], t)
    np.testing.assert_array_equal(out["alpha"], 0.75 * al)
    np.testing.assert_array_equal(out["beta"], be)
    np.testing.assert_array_equal(out["v"], np.ones(K))
    np.testing.assert_array_equal(out["Q"], W)


def test_group_params_least_squares_given_codes():
    """The fitted alpha, beta are the least-squares solution (library
    routine) of w ~ alpha t + beta for the codes of the last fit, and the
    stored pair is that solution rounded to fp16."""
    rng = np.random.default_rng(9)
    for k in range(20):
        w = rng.normal(size=128) * 0.02 + 0.003 * k
        a, b, t = qz.group_fit(w)
        assert t is not None
        sol = np.linalg.lstsq(np.column_stack([t, np.ones_like(t)]), w, rcond=None)[0]
        assert a == pytest.approx(sol[0], rel=1e-12) and b == pytest.approx(sol[1], rel=1e-12, abs=1e-15)
        assert qz.group_params(w) == (float(np.float16(a)), float(np.float16(b)))


def test_e4m3_round_against_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(1)
    xs = np.concatenate([rng.normal(size=4000) * 0.01, rng.normal(size=2000) * 10,
                         rng.uniform(-448, 448, size=2000), [0.0, 1.0, -1.0, 448.0, -448.0, 2.0 ** -9, 2.0 ** -10]])
    xs = xs.astype(np.float32).astype(np.float64)  # exact in float32: no double rounding in torch's cast
    ref = torch.from_numpy(xs.astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = np.array([qz.e4m3_round(x) for x in xs], np.uint8)
    # torch keeps the sign of a zero result the same way
    np.testing.assert_array_equal(got, ref)


def test_e4m3_round_ties_and_saturation():
    assert oracle.e4m3_to_double(qz.e4m3_round(1.0625)) == 1.0     # halfway 1 and 1.125: even code
    assert oracle.e4m3_to_double(qz.e4m3_round(1.1875)) == 1.25    # halfway 1.125 and 1.25: even code
    assert qz.e4m3_round(1e6) == 0x7E and qz.e4m3_round(-1e6) == 0xFE
    assert qz.e4m3_round(464.0) == 0x7E
    assert qz.e4m3_round(2.0 ** -10) == 0x00                           # halfway 0 and 2^-9: even (zero)
    assert qz.e4m3_round(-3 * 2.0 ** -11) == 0x81                      # nearest is -2^-9


def test_salient_is_best_subset_and_invariant():
    rng = np.random.default_rng(21)
    N, K, k = 8, 9, 3
    W = rng.normal(size=(N, K))
    H = _spd(rng, K)
    s = qz.salient_scores(W, H)
    S = qz.select_salient(s, k)
    best = max(itertools.combinations(range(K), k), key=lambda c: sum(s[list(c)]))
    assert tuple(S.tolist()) == tuple(sorted(best))
    assert list(S) == sorted(S)
    perm = rng.permutation(N)
    np.testing.assert_array_equal(qz.select_salient(qz.salient_scores(W[perm], H), k), S)
    np.testing.assert_array_equal(qz.select_salient(qz.salient_scores(3.0 * W, 0.5 * H), k), S)
    W2 = W.copy()
    W2[2, 7] = 1e3
    assert 7 in qz.select_salient(qz.salient_scores(W2, H), 1)
    # ties go to the lower column
    np.testing.assert_array_equal(qz.select_salient(np.array([1.0, 2.0, 2.0, 2.0]), 2), [1, 2])


def test_salient_score_hand_derived_eq3():
    """Eq. 3, s_j = max_i W_ij^2 diag(H)_j^2, on three hand-made cases whose
    expected salient column flips under each plausible misreading.  Every
    value below is derived by hand from the formula, not by the oracle.

    Case A, maximum over rows (not the mean), W squared (a negative entry):
      H = I (diag 1, 1); column 0 = (-3, 0, 0, 0), column 1 = (2, 2, 2, 2).
      max_i W^2 d^2:  col 0: 9 * 1 = 9,     col 1: 4 * 1 = 4      -> {0}
      mean_i W^2 d^2: col 0: 9/4 = 2.25,    col 1: 4              -> {1}
      max_i W d^2 (no square): col 0: 0,    col 1: 2              -> {1}
    Case B, diag(H) squared (not to the first power, not left out):
      diag H = (1, 3); column 0 = (2, 0, 0, 0), column 1 = (1, 0, 0, 0).
      W^2 d^2: col 0: 4 * 1 = 4,  col 1: 1 * 9 = 9                 -> {1}
      W^2 d:   col 0: 4,          col 1: 1 * 3 = 3                 -> {0}
      W^2:     col 0: 4,          col 1: 1                         -> {0}
    Case C, W squared (not |W|):
      diag H = (1, 1.5); column 0 = (0, 2, 0, 0), column 1 = (0, 0, -1, 0).
      W^2 d^2: col 0: 4 * 1 = 4,  col 1: 1 * 2.25 = 2.25           -> {0}
      |W| d^2: col 0: 2 * 1 = 2,  col 1: 1 * 2.25 = 2.25           -> {1}
    Off-diagonal entries of H are set large in B and C: a score that read
    a row or column of H instead of its diagonal changes the picture.
    """
    WA = np.array([[-3.0, 2.0], [0.0, 2.0], [0.0, 2.0], [0.0, 2.0]])
    HA = np.eye(2)
    WB = np.array([[2.0, 1.0], [0.0, 0.0], [0.0, 0.0], [0.0, 0.0]])
    HB = np.array([[1.0, 0.9], [0.9, 3.0]])
    WC = np.array([[0.0, 0.0], [2.0, 0.0], [0.0, -1.0], [0.0, 0.0]])
    HC = np.array([[1.0, 1.2], [1.2, 1.5]])
    for W, H, scores, chosen in ((WA, HA, [9.0, 4.0], [0]),
                                 (WB, HB, [4.0, 9.0], [1]),
                                 (WC, HC, [4.0, 2.25], [0])):
        np.testing.assert_array_equal(qz.salient_scores(W, H), scores)
        np.testing.assert_array_equal(qz.select_salient(qz.salient_scores(W, H), 1), chosen)
    # the same choice through the whole quantizer (one salient column, one
    # four-row residual group): case A's column 0, on a positive-definite H
    out = qz.quantize(WA, HA, 1, lam=1.0, iters=2, group=2)
    np.testing.assert_array_equal(out["S"], [0])
    out = qz.quantize(WB, HB, 1, lam=1.0, iters=2, group=2)
    np.testing.assert_array_equal(out["S"], [1])


def test_hessian_explicit_sums():
    rng = np.random.default_rng(2)
    X = rng.normal(size=(5, 4))
    H = qz.hessian(X)
    for a in range(4):
        for b in range(4):
            assert H[a, b] == pytest.approx(2.0 / 5 * sum(X[t, a] * X[t, b] for t in range(5)), rel=1e-14)


def test_residual_structure_identity_hessian():
    rng = np.random.default_rng(4)
    N, K, nS = 16, 20, 4
    W = rng.normal(size=(N, K)) * 0.02
    W[:, 3] *= 20
    out = qz.quantize(W, np.eye(K), nS, lam=1.0, iters=2, group=8)
    assert 3 in out["S"]
    for s, j in enumerate(out["S"]):
        g8 = j // 8
        qt = out["beta"][:, g8] + out["v"][j] * out["alpha"][:, g8] * out["T"][:, j]
        for g in range(N // 4):
            rows = slice(4 * g, 4 * g + 4)
            k = int(np.argmax(np.abs(W[rows, j] - qt[rows])))
            assert out["ridx"][s, g] == k
            diff = out["Q"][rows, j] - qt[rows]
            assert np.count_nonzero(diff) <= 1
            assert diff[k] == oracle.e4m3_to_double(int(out["rval"][s, g]))
            assert abs(W[4 * g + k, j] - out["Q"][4 * g + k, j]) <= abs(W[4 * g + k, j] - qt[4 * g + k])


def test_gptq_lowers_hessian_weighted_error():
    rng = np.random.default_rng(8)
    N, K = 16, 64
    H = _spd(rng, K)
    W = rng.normal(size=(N, K)) * 0.02
    err = lambda Q: float(np.trace((W - Q) @ H @ (W - Q).T))
    gptq = qz.quantize(W, H, 0, lam=0.0, iters=2, group=32)["Q"]
    rtn = qz.quantize(W, np.eye(K), 0, lam=0.0, iters=2, group=32)["Q"]
    assert err(gptq) < 0.9 * err(rtn)
