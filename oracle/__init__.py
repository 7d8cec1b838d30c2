"""Plain fp64 CPU oracle for the QTEA compressed ternary GEMV.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The GPU library never imports,
links or runs anything here, and this package never imports the GPU
library.  The arithmetic lives in ``qtea_oracle.c`` (plain C loops, fp64);
this module only marshals numpy arrays through ctypes.

Pins (tests/test_oracle.py): exhaustive code round trip, sign-symmetry and
zero-pattern closed forms, hand-worked example (tests/golden), brute force
in exact rational arithmetic on tiny inputs, textbook special cases, the
paper's bits-per-weight figures, the FP8 E4M3 decode against a library
routine and the format's closed forms, the salient bitmap against brute
force.  Every function is pinned; none is marked "parity unpinned".
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "qtea_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, ERR_ARG, ERR_TRIT, ERR_CODE, ERR_RESID, ERR_NOMEM = 0, -1, -2, -3, -4, -5


class OracleError(RuntimeError):
    def __init__(self, rc, what):
        super().__init__(f"oracle {what} failed with status {rc}")
        self.rc = rc


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (plain C, OpenMP over rows)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11", "-fno-fast-math",
             "-ffp-contract=off", "-o", tmp, _SRC, "-lm"]
        )
        os.replace(tmp, _LIB)
    return _LIB



def build_sanitized(out_dir: str) -> str:
    """Compile the same source with the host address and undefined-behaviour
    sanitizers into out_dir (load it through $QTEA_ORACLE_LIB, with the sanitizer
    runtime preloaded); returns the library path."""
    out = os.path.join(out_dir, "liboracle.so")
    subprocess.check_call(
        ["gcc", "-O1", "-g", "-fPIC", "-shared", "-fopenmp", "-std=c11", "-fno-fast-math", "-ffp-contract=off",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
         "-o", out, _SRC, "-lm"]
    )
    return out


_lib = None


def _L():
    global _lib
    if _lib is None:
        path = os.environ.get("QTEA_ORACLE_LIB")  # another build of the same source (the sanitized one)
        if not path:
            if not os.path.exists(_LIB):
                build()
            path = _LIB
        lib = ctypes.CDLL(path)
        i64, i32, vp, dbl = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_double
        lib.or_half_to_double.restype = dbl
        lib.or_half_to_double.argtypes = [ctypes.c_uint16]
        lib.or_num_packs.restype = i64
        lib.or_num_packs.argtypes = [i64]
        lib.or_encode5.restype = i32
        lib.or_encode5.argtypes = [vp]
        lib.or_decode_code.restype = i32
        lib.or_decode_code.argtypes = [i32, vp]
        lib.or_pack.restype = i32
        lib.or_pack.argtypes = [vp, i64, i64, vp]
        lib.or_unpack.restype = i32
        lib.or_unpack.argtypes = [vp, i64, i64, vp]
        lib.or_check_salient.restype = i32
        lib.or_check_salient.argtypes = [vp, i64, i64]
        lib.or_resid_rows.restype = i32
        lib.or_resid_rows.argtypes = [vp, i64, i64, vp]
        lib.or_dense_rows.restype = i32
        lib.or_dense_rows.argtypes = [i64, i64, vp, vp, i64, vp, vp, vp, i64, vp, vp, vp]
        lib.or_gemv_rows.restype = i32
        lib.or_gemv_rows.argtypes = [i64, i64, vp, vp, i64, vp, vp, vp, i64, vp, vp, vp, i64, vp, i32]
        lib.or_gemv_lut_rows.restype = i32
        lib.or_gemv_lut_rows.argtypes = [i64, i64, vp, vp, i64, vp, vp, vp, i64, vp, vp, vp, i64, vp]
        lib.or_bpw_full.restype = dbl
        lib.or_bpw_full.argtypes = [i64, i64, i64]
        lib.or_bpw_paper.restype = dbl
        lib.or_bpw_paper.argtypes = [dbl, dbl]
        lib.or_algorithmic_bytes.restype = i64
        lib.or_algorithmic_bytes.argtypes = [i64, i64, i64]
        lib.or_e4m3_to_double.restype = dbl
        lib.or_e4m3_to_double.argtypes = [ctypes.c_uint8]
        lib.or_bitmap_to_list.restype = i64
        lib.or_bitmap_to_list.argtypes = [vp, i64, vp, i64]
        lib.or_algorithmic_bytes_vb.restype = i64
        lib.or_algorithmic_bytes_vb.argtypes = [i64, i64, i64, i64]
        lib.or_num_groups128.restype = i64
        lib.or_num_groups128.argtypes = [i64]
        lib.or_pack128.restype = i32
        lib.or_pack128.argtypes = [vp, i64, i64, vp]
        lib.or_unpack128.restype = i32
        lib.or_unpack128.argtypes = [vp, i64, i64, vp]
        lib.or_gemv128_rows.restype = i32
        lib.or_gemv128_rows.argtypes = [i64, i64, vp, vp, i64, vp, vp, vp, vp, i64, vp, vp, vp, i64, vp, i32]
        lib.or_algorithmic_bytes128.restype = i64
        lib.or_algorithmic_bytes128.argtypes = [i64, i64, i64, i64]
        _lib = lib
    return _lib


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _bits16(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.float16:
        return a.view(np.uint16)
    return _c(a, np.uint16)


def threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def half_to_double(h: int) -> float:
    return float(_L().or_half_to_double(int(h) & 0xFFFF))


def num_packs(K: int) -> int:
    return int(_L().or_num_packs(K))


def encode5(t) -> int:
    t = _c(t, np.int8)
    assert t.size == 5
    return int(_L().or_encode5(t.ctypes.data))


def decode_code(c: int):
    t = np.zeros(5, dtype=np.int8)
    rc = _L().or_decode_code(int(c), t.ctypes.data)
    if rc:
        raise OracleError(rc, "decode_code")
    return t


def pack(trits) -> np.ndarray:
    t = _c(trits, np.int8)
    n, K = t.shape
    out = np.empty((n, num_packs(K)), dtype=np.uint8)
    rc = _L().or_pack(t.ctypes.data, n, K, out.ctypes.data)
    if rc:
        raise OracleError(rc, "pack")
    return out


def unpack(codes, K: int) -> np.ndarray:
    c = _c(codes, np.uint8)
    n = c.shape[0]
    if c.shape[1] != num_packs(K):
        raise ValueError("code row length must be ceil(K/5)")
    out = np.empty((n, K), dtype=np.int8)
    rc = _L().or_unpack(c.ctypes.data, n, K, out.ctypes.data)
    if rc:
        raise OracleError(rc, "unpack")
    return out


def check_salient(S, K: int) -> int:
    S = _c(S, np.int32)
    return int(_L().or_check_salient(S.ctypes.data, S.size, K))


def resid_rows(idx, N: int) -> np.ndarray:
    idx = _c(idx, np.uint8)
    nS = idx.shape[0]
    out = np.empty((nS, N // 4), dtype=np.int32)
    rc = _L().or_resid_rows(idx.ctypes.data, nS, N, out.ctypes.data)
    if rc:
        raise OracleError(rc, "resid_rows")
    return out


def _layer_args(N, K, alpha, v, S, R, idx):
    alpha, v = _bits16(alpha), _bits16(v)
    S = _c(S, np.int32)
    nS = S.size
    R = _bits16(R).reshape(nS, N // 4) if nS else np.zeros((0, N // 4), np.uint16)
    idx = _c(idx, np.uint8).reshape(nS, N // 4) if nS else np.zeros((0, N // 4), np.uint8)
    assert alpha.size == N and v.size == K
    keep = (alpha, v, S, R, idx)
    return keep, [alpha.ctypes.data, v.ctypes.data, S.ctypes.data, nS, R.ctypes.data, idx.ctypes.data]


def _rows_args(N, K, codes_rows, rows):
    rows = np.arange(N, dtype=np.int64) if rows is None else _c(rows, np.int64)
    P = _c(codes_rows, np.uint8)
    if P.shape != (rows.size, num_packs(K)):
        raise ValueError(f"codes_rows must be [{rows.size}][{num_packs(K)}], got {P.shape}")
    return P, rows


def dense_rows(N, K, codes_rows, alpha, v, S, R, idx, rows=None) -> np.ndarray:
    """fp64 dequantized rows (alpha_r v_j T_rj plus the stored residuals)."""
    P, rows = _rows_args(N, K, codes_rows, rows)
    keep, la = _layer_args(N, K, alpha, v, S, R, idx)
    W = np.empty((rows.size, K), dtype=np.float64)
    rc = _L().or_dense_rows(N, K, P.ctypes.data, rows.ctypes.data, rows.size, *la, W.ctypes.data)
    if rc:
        raise OracleError(rc, "dense_rows")
    return W


def gemv(N, K, codes_rows, alpha, v, S, R, idx, x, rows=None, nthreads=None) -> np.ndarray:
    """fp64 y[b][i] for output rows `rows` (default: all rows)."""
    P, rows = _rows_args(N, K, codes_rows, rows)
    keep, la = _layer_args(N, K, alpha, v, S, R, idx)
    x = _bits16(x).reshape(-1, K)
    B = x.shape[0]
    y = np.empty((B, rows.size), dtype=np.float64)
    rc = _L().or_gemv_rows(N, K, P.ctypes.data, rows.ctypes.data, rows.size, *la, x.ctypes.data,
                           B, y.ctypes.data, int(nthreads or threads()))
    if rc:
        raise OracleError(rc, "gemv")
    return y


def gemv_lut(N, K, codes_rows, alpha, v, S, R, idx, x, rows=None) -> np.ndarray:
    """fp64 y through per-pack 243-entry tables (same result as gemv)."""
    P, rows = _rows_args(N, K, codes_rows, rows)
    keep, la = _layer_args(N, K, alpha, v, S, R, idx)
    x = _bits16(x).reshape(-1, K)
    B = x.shape[0]
    y = np.empty((B, rows.size), dtype=np.float64)
    rc = _L().or_gemv_lut_rows(N, K, P.ctypes.data, rows.ctypes.data, rows.size, *la,
                               x.ctypes.data, B, y.ctypes.data)
    if rc:
        raise OracleError(rc, "gemv_lut")
    return y


def bpw_full(N, K, nS) -> float:
    return float(_L().or_bpw_full(N, K, nS))


def bpw_paper(f, value_bits) -> float:
    return float(_L().or_bpw_paper(float(f), float(value_bits)))


def algorithmic_bytes(N, K, nS) -> int:
    return int(_L().or_algorithmic_bytes(N, K, nS))


def e4m3_to_double(code: int) -> float:
    return float(_L().or_e4m3_to_double(int(code) & 0xFF))


def e4m3_decode(codes) -> np.ndarray:
    """fp64 values of FP8 E4M3 codes (any shape)."""
    c = _c(codes, np.uint8)
    table = np.array([e4m3_to_double(i) for i in range(256)], dtype=np.float64)
    return table[c]


def e4m3_as_half(codes) -> np.ndarray:
    """The same values as fp16 (every finite E4M3 value is one); raises if a
    code is NaN."""
    d = e4m3_decode(codes)
    if np.isnan(d).any():
        raise OracleError(ERR_RESID, "e4m3_as_half (NaN code)")
    h = d.astype(np.float16)
    assert np.array_equal(h.astype(np.float64), d)
    return h


def bitmap_to_list(words, K: int) -> np.ndarray:
    """Ascending salient columns marked in a column bitmap."""
    w = np.ascontiguousarray(words)
    if w.dtype.itemsize != 4:
        raise ValueError("bitmap words are 32-bit")
    w = w.view(np.uint32)
    if w.size != (K + 31) // 32:
        raise ValueError("a bitmap of ceil(K/32) words")
    S = np.empty(K, dtype=np.int32)
    n = int(_L().or_bitmap_to_list(w.ctypes.data, K, S.ctypes.data, K))
    if n < 0:
        raise OracleError(n, "bitmap_to_list")
    return S[:n].copy()


def algorithmic_bytes_vb(N, K, nS, value_bytes) -> int:
    return int(_L().or_algorithmic_bytes_vb(N, K, nS, value_bytes))


# The paper's 128-column quantization groups (Eq. 10 with alpha and beta per
# row and group; 26 bytes per row and group).
def num_groups128(K: int) -> int:
    return int(_L().or_num_groups128(K))


def pack128(trits) -> np.ndarray:
    t = _c(trits, np.int8)
    n, K = t.shape
    out = np.empty((n, 26 * num_groups128(K)), dtype=np.uint8)
    rc = _L().or_pack128(t.ctypes.data, n, K, out.ctypes.data)
    if rc:
        raise OracleError(rc, "pack128")
    return out


def unpack128(codes, K: int) -> np.ndarray:
    c = _c(codes, np.uint8)
    n = c.shape[0]
    if c.shape[1] != 26 * num_groups128(K):
        raise ValueError("code row length must be 26 * ceil(K/128)")
    out = np.empty((n, K), dtype=np.int8)
    rc = _L().or_unpack128(c.ctypes.data, n, K, out.ctypes.data)
    if rc:
        raise OracleError(rc, "unpack128")
    return out


def gemv128(N, K, codes_rows, alpha, beta, v, S, R, idx, x, rows=None, nthreads=None) -> np.ndarray:
    """fp64 y[b][i] with per-row, per-128-column-group alpha and beta
    ([N][ceil(K/128)] fp16) for output rows `rows` (default all)."""
    rows = np.arange(N, dtype=np.int64) if rows is None else _c(rows, np.int64)
    ng = num_groups128(K)
    P = _c(codes_rows, np.uint8)
    if P.shape != (rows.size, 26 * ng):
        raise ValueError(f"codes_rows must be [{rows.size}][{26 * ng}]")
    alpha, beta = _bits16(alpha).reshape(N, ng), _bits16(beta).reshape(N, ng)
    keep, la = _layer_args(N, K, np.zeros(N, np.uint16), v, S, R, idx)
    x = _bits16(x).reshape(-1, K)
    B = x.shape[0]
    y = np.empty((B, rows.size), dtype=np.float64)
    rc = _L().or_gemv128_rows(N, K, P.ctypes.data, rows.ctypes.data, rows.size, alpha.ctypes.data,
                              beta.ctypes.data, *la[1:], x.ctypes.data, B, y.ctypes.data,
                              int(nthreads or threads()))
    if rc:
        raise OracleError(rc, "gemv128")
    return y


def algorithmic_bytes128(N, K, nS, value_bytes) -> int:
    return int(_L().or_algorithmic_bytes128(N, K, nS, value_bytes))
