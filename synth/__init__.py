"""Seeded synthetic inputs for the QTEA ternary GEMV workloads.

This package draws random numbers and nothing else: it produces the dense
inputs of one compressed linear layer (ternary codes T, row scales alpha,
column rescales v, the salient column set S, the 1:4 residual values R and
their 2-bit in-group positions) and the activations x.  It holds none of the
method's arithmetic (no packing, no scaling, no lookup tables), so the CPU
oracle and the GPU path can both take their inputs from here without sharing
code with each other.

Value recipe (stands in for QTEA-quantized checkpoints, which are not
available; shapes follow Llama-3-8B, Qwen3-14B and Llama-3-70B linears):
  * T i.i.d.: P(0) = p0, P(+1) = P(-1) = (1 - p0) / 2, via integer thresholds
    on the top 32 bits of each draw;
  * alpha ~ U(0.01, 0.03), v ~ U(0.8, 1.2), x ~ N(0, 1), R ~ N(0, 0.01)
    (sigma = 0.01), each drawn in float64 and rounded to fp16 (RNE);
  * |S| = floor(f * K + 1/2) columns chosen uniformly without replacement,
    sorted ascending;
  * one residual per (salient column, group of 4 consecutive output rows), at
    a uniformly drawn position 0..3 in the group;
  * for the paper's residual storage (resid="e4m3"): the same R draw rounded
    to FP8 E4M3 (RNE, by torch's float8_e4m3fn conversion) and given as
    codes, and the salient set given as a column bitmap;
  * for the paper's 128-column quantization groups (groups=128): a scale
    alpha[r][g] ~ U(0.01, 0.03) and a bias beta[r][g] ~ U(-0.005, 0.005)
    per row and group, rounded to fp16.

Quantizer inputs (quant_inputs; stand in for a full-precision linear layer
and its calibration activations, which are not available): weights
W ~ N(0, 0.02) in fp64 with 1% of the columns scaled by 4 (outlier input
channels); calibration rows X = Z M in fp32 with Z ~ N(0, 1) [n][K] and
M = I + N(0, 0.1 / sqrt(K)) [K][K] (correlated channels), 2% of the channels
scaled by 5 (high-energy activations); numpy's PCG64 generator seeded by
`seed`.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from fractions import Fraction

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth_gen.c")
_LIB = os.path.join(_HERE, "libsynth.so")

# Field tags of the per-(seed, layer, matrix) streams.
FIELD_TRITS, FIELD_SALIENT, FIELD_RIDX, FIELD_RVAL, FIELD_ALPHA, FIELD_V, FIELD_X, FIELD_BETA = range(1, 9)

DEFAULT_SEED = 20260224


def build(force: bool = False) -> str:
    """Compile the generator with gcc (OpenMP); returns the library path."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11", "-o", tmp, _SRC, "-lm"]
        )
        os.replace(tmp, _LIB)
    return _LIB



def build_sanitized(out_dir: str) -> str:
    """Compile the same source with the host address and undefined-behaviour
    sanitizers into out_dir (load it through $QTEA_SYNTH_LIB, with the sanitizer
    runtime preloaded); returns the library path."""
    out = os.path.join(out_dir, "libsynth.so")
    subprocess.check_call(
        ["gcc", "-O1", "-g", "-fPIC", "-shared", "-fopenmp", "-std=c11",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
         "-o", out, _SRC, "-lm"]
    )
    return out


_lib = None


def _L():
    global _lib
    if _lib is None:
        path = os.environ.get("QTEA_SYNTH_LIB")  # another build of the same source (the sanitized one)
        if not path:
            if not os.path.exists(_LIB):
                build()
            path = _LIB
        lib = ctypes.CDLL(path)
        u64, i64, i32, dbl, vp = (ctypes.c_uint64, ctypes.c_int64, ctypes.c_int,
                                  ctypes.c_double, ctypes.c_void_p)
        lib.synth_sm64_at.restype = u64
        lib.synth_sm64_at.argtypes = [u64, u64]
        lib.synth_key.restype = u64
        lib.synth_key.argtypes = [u64, u64, u64, u64]
        lib.synth_trits.restype = None
        lib.synth_trits.argtypes = [u64, i64, i64, ctypes.c_uint32, ctypes.c_uint32, vp, i32]
        lib.synth_trits_rows.restype = None
        lib.synth_trits_rows.argtypes = [u64, i64, vp, i64, ctypes.c_uint32, ctypes.c_uint32, vp, i32]
        lib.synth_uniform.restype = None
        lib.synth_uniform.argtypes = [u64, i64, dbl, dbl, vp]
        lib.synth_normal.restype = None
        lib.synth_normal.argtypes = [u64, i64, dbl, dbl, vp]
        lib.synth_uint2.restype = None
        lib.synth_uint2.argtypes = [u64, i64, vp]
        lib.synth_choose_sorted.restype = i32
        lib.synth_choose_sorted.argtypes = [u64, i64, i64, vp]
        _lib = lib
    return _lib


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def sm64_at(key: int, i: int) -> int:
    """Element i of the counter-mode SplitMix64 stream keyed by `key`."""
    return int(_L().synth_sm64_at(key, i))


def key(seed: int, layer: int, mat: int, field: int) -> int:
    return int(_L().synth_key(seed, layer, mat, field))


def trit_thresholds(p0: Fraction | float) -> tuple[int, int]:
    """Integer thresholds (thr_neg, thr_zero) on a uniform u32 for P(0) = p0."""
    p0 = Fraction(p0).limit_denominator(10**6)
    pm = (1 - p0) / 2
    thr_neg = (pm * 2**32).__floor__()
    thr_zero = ((pm + p0) * 2**32).__floor__()
    return int(thr_neg), int(thr_zero)


def n_salient(K: int, frac: Fraction | float) -> int:
    """|S| = floor(f * K + 1/2) with f taken as an exact rational."""
    f = Fraction(frac).limit_denominator(10**6)
    return int((f * K + Fraction(1, 2)).__floor__())


def trits(seed, layer, mat, N, K, p0, rows=None) -> np.ndarray:
    """Ternary codes int8 [N][K] (or [len(rows)][K] for a row subset)."""
    k = key(seed, layer, mat, FIELD_TRITS)
    tn, tz = trit_thresholds(p0)
    lib = _L()
    if rows is None:
        out = np.empty((N, K), dtype=np.int8)
        lib.synth_trits(k, N, K, tn, tz, out.ctypes.data, _threads())
    else:
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        if rows.size and (rows.min() < 0 or rows.max() >= N):
            raise ValueError("row index out of range")
        out = np.empty((rows.size, K), dtype=np.int8)
        lib.synth_trits_rows(k, K, rows.ctypes.data, rows.size, tn, tz, out.ctypes.data, _threads())
    return out


def uniform_f16(k: int, n: int, lo: float, hi: float) -> np.ndarray:
    d = np.empty(n, dtype=np.float64)
    _L().synth_uniform(k, n, lo, hi, d.ctypes.data)
    return d.astype(np.float16)


def normal_f16(k: int, n: int, mu: float, sigma: float) -> np.ndarray:
    d = np.empty(n, dtype=np.float64)
    _L().synth_normal(k, n, mu, sigma, d.ctypes.data)
    return d.astype(np.float16)


def normal_e4m3(k: int, n: int, mu: float, sigma: float) -> np.ndarray:
    """FP8 E4M3 codes (uint8) of float64 normal draws, rounded to nearest even."""
    import torch

    d = np.empty(n, dtype=np.float64)
    _L().synth_normal(k, n, mu, sigma, d.ctypes.data)
    return torch.from_numpy(d).to(torch.float8_e4m3fn).view(torch.uint8).numpy().copy()


def column_bitmap(S, K: int) -> np.ndarray:
    """int32 [ceil(K/32)] words, bit j % 32 of word j / 32 set for j in S."""
    w = np.zeros((K + 31) // 32, dtype=np.uint32)
    S = np.asarray(S, dtype=np.int64)
    np.bitwise_or.at(w, S // 32, (np.uint32(1) << (S % 32).astype(np.uint32)))
    return w.view(np.int32)


def layer_inputs(seed, layer, mat, N, K, p0=Fraction(2, 5), frac=Fraction(2, 100),
                 with_trits=True, rows=None, resid="fp16", groups=0) -> dict:
    """All non-activation inputs of one compressed N x K matrix.

    Returns numpy arrays: trits int8 [N][K] (omitted if with_trits is False),
    alpha fp16 [N], v fp16 [K], S int32 [nS] (sorted), R fp16 [nS][N/4],
    idx uint8 [nS][N/4]; with resid="e4m3" R is replaced by R8, uint8 E4M3
    codes [nS][N/4], and bitmap, int32 [ceil(K/32)], is added; with
    groups=128, alpha_g and beta_g fp16 [N][ceil(K/128)] are added.
    """
    if N % 4:
        raise ValueError("N must be a multiple of 4 (1:4 residual groups)")
    nS = n_salient(K, frac)
    G = N // 4
    S = np.zeros(nS, dtype=np.int32)
    if nS:
        rc = _L().synth_choose_sorted(key(seed, layer, mat, FIELD_SALIENT), K, nS, S.ctypes.data)
        if rc != 0:
            raise RuntimeError("synth_choose_sorted failed")
    idx = np.empty(nS * G, dtype=np.uint8)
    _L().synth_uint2(key(seed, layer, mat, FIELD_RIDX), nS * G, idx.ctypes.data)
    out = {
        "N": N,
        "K": K,
        "alpha": uniform_f16(key(seed, layer, mat, FIELD_ALPHA), N, 0.01, 0.03),
        "v": uniform_f16(key(seed, layer, mat, FIELD_V), K, 0.8, 1.2),
        "S": S,
        "idx": idx.reshape(nS, G),
    }
    if groups:
        if groups != 128:
            raise ValueError("quantization groups of 128 columns only")
        ng = (K + 127) // 128
        out["alpha_g"] = uniform_f16(key(seed, layer, mat, FIELD_ALPHA), N * ng, 0.01, 0.03).reshape(N, ng)
        out["beta_g"] = uniform_f16(key(seed, layer, mat, FIELD_BETA), N * ng, -0.005, 0.005).reshape(N, ng)
    if resid == "e4m3":
        out["R8"] = normal_e4m3(key(seed, layer, mat, FIELD_RVAL), nS * G, 0.0, 0.01).reshape(nS, G)
        out["bitmap"] = column_bitmap(S, K)
    elif resid == "fp16":
        out["R"] = normal_f16(key(seed, layer, mat, FIELD_RVAL), nS * G, 0.0, 0.01).reshape(nS, G)
    else:
        raise ValueError(f"unknown residual storage {resid!r}")
    if with_trits:
        out["trits"] = trits(seed, layer, mat, N, K, p0, rows=rows)
    return out


def activations(seed, layer, mat, B, K) -> np.ndarray:
    """x fp16 [B][K], N(0, 1), independent per (matrix, batch row)."""
    return normal_f16(key(seed, layer, mat, FIELD_X), B * K, 0.0, 1.0).reshape(B, K)


def quant_inputs(seed: int, N: int, K: int, n_calib: int):
    """Full-precision weights W fp64 [N][K] and calibration rows X fp32
    [n_calib][K] for the offline quantizer (recipe in the module docstring)."""
    rng = np.random.default_rng(seed)
    W = rng.normal(0.0, 0.02, size=(N, K))
    n_out = max(1, K // 100)
    W[:, rng.choice(K, size=n_out, replace=False)] *= 4.0
    M = np.eye(K) + rng.normal(0.0, 0.1 / np.sqrt(K), size=(K, K))
    X = rng.normal(size=(n_calib, K)) @ M
    n_hot = max(1, K // 50)
    X[:, rng.choice(K, size=n_hot, replace=False)] *= 5.0
    return W, X.astype(np.float32)
