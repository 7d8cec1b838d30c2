"""MI355X (gfx950) compressed ternary GEMV: Python binding of libqtea.so.

The binding marshals arguments only: every step of the GEMV runs in the HIP
kernels of ``csrc/qtea.hip``, ``csrc/grouped.hip`` and ``csrc/grouped_mma.hip``
behind the C ABI of ``include/qtea.h``, and every step of the offline
quantizer in those of ``csrc/quant.hip`` behind ``include/qtea_quant.h``.  Torch
is used to allocate device memory and to name the current HIP stream.
There is no CPU fallback: if the library is not built, loading it raises.

Entry points carry the C names: qtea_packed_bytes, qtea_pack,
qtea_packed_bytes_e4m3, qtea_pack_e4m3, qtea_packed_bytes_g128, qtea_pack_g128,
qtea_workspace_bytes, qtea_workspace_init, qtea_gemv, qtea_gemm_lowbatch,
qtea_debug_unpack, qtea_read_ceiling, qtea_status_string, qtea_abi_version,
qtea_grouped_plan_bytes, qtea_grouped_plan, qtea_grouped_gemv, qtea_grouped_status,
qtea_quant_hessian, qtea_quant_workspace_bytes, qtea_quantize.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libqtea.so")
# The debug build (QTEA_DEBUG=1 in the environment when the library is
# loaded): every decode table's rows for the byte values 243..255, which no
# base-3 code takes, read NaN, so a corrupted packed byte shows as NaN in
# its output row.  Same ABI.
DEBUG_LIB_PATH = os.path.join(HERE, "libqtea_debug.so")

QTEA_OK = 0
QTEA_ERR_INVALID_ARG = -1
QTEA_ERR_BAD_TRIT = -2
QTEA_ERR_BAD_RESIDUAL = -3
QTEA_ERR_BATCH = -4
QTEA_ERR_WORKSPACE = -5
QTEA_ERR_HIP = -6
QTEA_ERR_NOT_POSITIVE = -7
QTEA_QUANT_GROUP = 128
QTEA_MAX_BATCH = 16
QTEA_ABI_VERSION = 9  # the header this binding mirrors
QTEA_DESC_MAGIC = 0x51544541

# Every function the header declares (checked by tests/test_abi.py).
EXPORTS = (
    "qtea_status_string", "qtea_abi_version", "qtea_packed_bytes", "qtea_pack",
    "qtea_workspace_bytes", "qtea_workspace_init", "qtea_gemv", "qtea_gemm_lowbatch",
    "qtea_debug_unpack", "qtea_grouped_plan_bytes", "qtea_grouped_plan", "qtea_grouped_gemv",
    "qtea_grouped_status", "qtea_gemm_lowbatch_noalloc",
    "qtea_packed_bytes_e4m3", "qtea_pack_e4m3", "qtea_packed_bytes_g128", "qtea_pack_g128",
    "qtea_read_ceiling", "qtea_quant_hessian", "qtea_quant_workspace_bytes", "qtea_quantize",
)
QTEA_LAYOUT_FP16 = 2  # residual values fp16
QTEA_LAYOUT_E4M3 = 3  # residual values FP8 E4M3
QTEA_LAYOUT_G128 = 4  # 128-column groups with scale and bias, E4M3 residual
QTEA_GROUPED_MAGIC = 0x51475250


class QteaDesc(ctypes.Structure):
    """Mirror of struct qtea_desc (include/qtea.h)."""
    _fields_ = [
        ("magic", ctypes.c_uint32), ("layout", ctypes.c_uint32),
        ("N", ctypes.c_int64), ("K", ctypes.c_int64), ("n_salient", ctypes.c_int64),
        ("n_packs", ctypes.c_int64), ("n_groups", ctypes.c_int64), ("n_pad", ctypes.c_int64),
        ("bytes_total", ctypes.c_int64),
        ("off_trits", ctypes.c_int64), ("off_alpha", ctypes.c_int64), ("off_v", ctypes.c_int64),
        ("off_salient", ctypes.c_int64), ("off_spos", ctypes.c_int64), ("off_rval", ctypes.c_int64),
        ("off_ridx", ctypes.c_int64),
    ]


class QteaGroupedInfo(ctypes.Structure):
    """Mirror of struct qtea_grouped_info (include/qtea.h)."""
    _fields_ = [
        ("magic", ctypes.c_uint32), ("n_problems", ctypes.c_int32), ("batch", ctypes.c_int32),
        ("grid", ctypes.c_int32), ("rows_per_panel", ctypes.c_int32), ("max_parts", ctypes.c_int32),
        ("n_chunks", ctypes.c_int32), ("n_split_panels", ctypes.c_int32),
        ("layout", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("n_units", ctypes.c_int64), ("plan_bytes", ctypes.c_int64), ("workspace_bytes", ctypes.c_int64),
    ]


class QteaQuantParams(ctypes.Structure):
    """Mirror of struct qtea_quant_params (include/qtea_quant.h)."""
    _fields_ = [
        ("n_salient", ctypes.c_int64), ("lambda_decay", ctypes.c_double), ("damp", ctypes.c_double),
        ("iters", ctypes.c_int32), ("reserved", ctypes.c_int32),
    ]


class QteaError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {qtea_status_string(status)} ({status})")
        self.status = status


_lib = None


def load(path: str = None):
    """Load the HIP library (the debug build when QTEA_DEBUG=1); raises if it
    has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if path is None:
        path = DEBUG_LIB_PATH if os.environ.get("QTEA_DEBUG") == "1" else LIB_PATH
    _lib = open_library(path)
    return _lib


def open_library(path: str):
    """Open one build of the library with the argument types of every entry
    point (load() keeps one as the binding's library)."""
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built (run __graft_entry__.build()); "
                          "there is no fallback path")
    lib = ctypes.CDLL(path)
    i64, i32, vp = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
    pdesc = ctypes.POINTER(QteaDesc)
    lib.qtea_status_string.restype = ctypes.c_char_p
    lib.qtea_status_string.argtypes = [i32]
    lib.qtea_abi_version.restype = i32
    lib.qtea_abi_version.argtypes = []
    lib.qtea_packed_bytes.restype = i32
    lib.qtea_packed_bytes.argtypes = [i64, i64, i64, ctypes.POINTER(i64)]
    lib.qtea_pack.restype = i32
    lib.qtea_pack.argtypes = [vp, i64, i64, vp, vp, vp, i64, vp, vp, vp, i64, pdesc, vp]
    lib.qtea_packed_bytes_e4m3.restype = i32
    lib.qtea_packed_bytes_e4m3.argtypes = [i64, i64, i64, ctypes.POINTER(i64)]
    lib.qtea_pack_e4m3.restype = i32
    lib.qtea_pack_e4m3.argtypes = [vp, i64, i64, vp, vp, vp, i64, vp, vp, vp, i64, pdesc, vp]
    lib.qtea_packed_bytes_g128.restype = i32
    lib.qtea_packed_bytes_g128.argtypes = [i64, i64, i64, ctypes.POINTER(i64)]
    lib.qtea_pack_g128.restype = i32
    lib.qtea_pack_g128.argtypes = [vp, i64, i64, vp, vp, vp, vp, i64, vp, vp, vp, i64, pdesc, vp]
    lib.qtea_workspace_bytes.restype = i32
    lib.qtea_workspace_bytes.argtypes = [pdesc, i32, ctypes.POINTER(i64)]
    lib.qtea_workspace_init.restype = i32
    lib.qtea_workspace_init.argtypes = [vp, i64, vp]
    lib.qtea_gemv.restype = i32
    lib.qtea_gemv.argtypes = [pdesc, vp, vp, vp, vp, i64, vp]
    lib.qtea_gemm_lowbatch.restype = i32
    lib.qtea_gemm_lowbatch.argtypes = [pdesc, vp, vp, i32, vp, vp, i64, vp]
    lib.qtea_read_ceiling.restype = i32
    lib.qtea_read_ceiling.argtypes = [vp, i64, vp, vp]
    lib.qtea_debug_unpack.restype = i32
    lib.qtea_debug_unpack.argtypes = [pdesc, vp, vp, vp, vp, vp]
    pinfo = ctypes.POINTER(QteaGroupedInfo)
    lib.qtea_grouped_plan_bytes.restype = i32
    lib.qtea_grouped_plan_bytes.argtypes = [i32, ctypes.POINTER(i64)]
    lib.qtea_grouped_plan.restype = i32
    lib.qtea_grouped_plan.argtypes = [pdesc, ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp),
                                      i32, i32, vp, i64, pinfo, vp]
    lib.qtea_grouped_gemv.restype = i32
    lib.qtea_grouped_gemv.argtypes = [pinfo, vp, vp, i64, vp]
    lib.qtea_gemm_lowbatch_noalloc.restype = i32
    lib.qtea_gemm_lowbatch_noalloc.argtypes = [pdesc, vp, vp, i32, vp, vp]
    lib.qtea_grouped_status.restype = i32
    lib.qtea_grouped_status.argtypes = [vp, ctypes.POINTER(ctypes.c_uint32), vp]
    lib.qtea_quant_hessian.restype = i32
    lib.qtea_quant_hessian.argtypes = [vp, i64, i64, vp, vp]
    lib.qtea_quant_workspace_bytes.restype = i32
    lib.qtea_quant_workspace_bytes.argtypes = [i64, i64, ctypes.POINTER(i64)]
    lib.qtea_quantize.restype = i32
    lib.qtea_quantize.argtypes = [vp, vp, i64, i64, ctypes.POINTER(QteaQuantParams),
                                  vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, i64, vp]
    return lib


def _stream(stream=None):
    import torch

    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check(status: int, what: str):
    if status != QTEA_OK:
        raise QteaError(status, what)


def _need_cuda(*tensors):
    for t in tensors:
        if t is not None and not t.is_cuda:
            raise ValueError("qtea entry points take device tensors")
        if t is not None and not t.is_contiguous():
            raise ValueError("qtea entry points take contiguous tensors")


# ---------------------------------------------------------------------------
# Entry points (same names as the C ABI).
# ---------------------------------------------------------------------------
def qtea_status_string(status: int) -> str:
    return load().qtea_status_string(int(status)).decode()


def qtea_abi_version() -> int:
    return int(load().qtea_abi_version())


def qtea_packed_bytes(N: int, K: int, n_salient: int) -> int:
    out = ctypes.c_int64(0)
    _check(load().qtea_packed_bytes(N, K, n_salient, ctypes.byref(out)), "qtea_packed_bytes")
    return out.value


def qtea_pack(trits, row_scale, col_rescale, salient, resid_val, resid_idx, packed,
              stream=None) -> QteaDesc:
    """Pack device tensors (int8 [N][K], fp16 [N], fp16 [K], int32 [nS],
    fp16 [nS][N/4], uint8 [nS][N/4]) into `packed` (uint8, >= qtea_packed_bytes)."""
    import torch

    _need_cuda(trits, row_scale, col_rescale, salient, resid_val, resid_idx, packed)
    assert trits.dtype == torch.int8 and row_scale.dtype == torch.float16
    assert col_rescale.dtype == torch.float16 and salient.dtype == torch.int32
    assert resid_val.dtype == torch.float16 and resid_idx.dtype == torch.uint8
    N, K = trits.shape
    nS = salient.numel()
    d = QteaDesc()
    st = load().qtea_pack(_ptr(trits), N, K, _ptr(row_scale), _ptr(col_rescale),
                          _ptr(salient) if nS else None, nS,
                          _ptr(resid_val) if nS else None, _ptr(resid_idx) if nS else None,
                          _ptr(packed), packed.numel() * packed.element_size(), ctypes.byref(d),
                          _stream(stream))
    _check(st, "qtea_pack")
    return d


def qtea_packed_bytes_e4m3(N: int, K: int, n_salient: int) -> int:
    out = ctypes.c_int64(0)
    _check(load().qtea_packed_bytes_e4m3(N, K, n_salient, ctypes.byref(out)), "qtea_packed_bytes_e4m3")
    return out.value


def qtea_pack_e4m3(trits, row_scale, col_rescale, salient_bitmap, n_salient: int, resid_val,
                   resid_idx, packed, stream=None) -> QteaDesc:
    """Pack with the paper's residual storage: int8 [N][K] trits, fp16 [N]
    and [K] scales, int32 [ceil(K/32)] salient column bitmap (bit j % 32 of
    word j / 32), uint8 [nS][N/4] E4M3 residual codes, uint8 [nS][N/4]
    positions, into `packed` (uint8, >= qtea_packed_bytes_e4m3)."""
    import torch

    _need_cuda(trits, row_scale, col_rescale, salient_bitmap, resid_val, resid_idx, packed)
    assert trits.dtype == torch.int8 and row_scale.dtype == torch.float16
    assert col_rescale.dtype == torch.float16 and salient_bitmap.dtype == torch.int32
    assert resid_val.dtype == torch.uint8 and resid_idx.dtype == torch.uint8
    N, K = trits.shape
    if salient_bitmap.numel() != (K + 31) // 32:
        raise ValueError("the salient bitmap has ceil(K/32) words")
    nS = int(n_salient)
    d = QteaDesc()
    st = load().qtea_pack_e4m3(_ptr(trits), N, K, _ptr(row_scale), _ptr(col_rescale), _ptr(salient_bitmap),
                               nS, _ptr(resid_val) if nS else None, _ptr(resid_idx) if nS else None,
                               _ptr(packed), packed.numel() * packed.element_size(), ctypes.byref(d),
                               _stream(stream))
    _check(st, "qtea_pack_e4m3")
    return d


def qtea_packed_bytes_g128(N: int, K: int, n_salient: int) -> int:
    out = ctypes.c_int64(0)
    _check(load().qtea_packed_bytes_g128(N, K, n_salient, ctypes.byref(out)), "qtea_packed_bytes_g128")
    return out.value


def qtea_pack_g128(trits, group_scale, group_bias, col_rescale, salient_bitmap, n_salient: int, resid_val,
                   resid_idx, packed, stream=None) -> QteaDesc:
    """Pack in the paper's grouped format: int8 [N][K] trits, fp16 [N][ceil(K/128)]
    group scales and biases, fp16 [K] rescales, int32 [ceil(K/32)] salient
    bitmap, uint8 [nS][N/4] E4M3 residual codes and positions."""
    import torch

    _need_cuda(trits, group_scale, group_bias, col_rescale, salient_bitmap, resid_val, resid_idx, packed)
    assert trits.dtype == torch.int8 and group_scale.dtype == torch.float16
    assert group_bias.dtype == torch.float16 and col_rescale.dtype == torch.float16
    assert salient_bitmap.dtype == torch.int32
    assert resid_val.dtype == torch.uint8 and resid_idx.dtype == torch.uint8
    N, K = trits.shape
    ng = (K + 127) // 128
    if tuple(group_scale.shape) != (N, ng) or tuple(group_bias.shape) != (N, ng):
        raise ValueError("group scales and biases are [N][ceil(K/128)]")
    if salient_bitmap.numel() != (K + 31) // 32:
        raise ValueError("the salient bitmap has ceil(K/32) words")
    nS = int(n_salient)
    d = QteaDesc()
    st = load().qtea_pack_g128(_ptr(trits), N, K, _ptr(group_scale), _ptr(group_bias), _ptr(col_rescale),
                               _ptr(salient_bitmap), nS, _ptr(resid_val) if nS else None,
                               _ptr(resid_idx) if nS else None, _ptr(packed),
                               packed.numel() * packed.element_size(), ctypes.byref(d), _stream(stream))
    _check(st, "qtea_pack_g128")
    return d


def qtea_workspace_bytes(desc: QteaDesc, batch: int) -> int:
    out = ctypes.c_int64(0)
    _check(load().qtea_workspace_bytes(ctypes.byref(desc), int(batch), ctypes.byref(out)),
           "qtea_workspace_bytes")
    return out.value


def qtea_workspace_init(workspace, stream=None):
    _need_cuda(workspace)
    _check(load().qtea_workspace_init(_ptr(workspace), workspace.numel() * workspace.element_size(),
                                      _stream(stream)), "qtea_workspace_init")


def qtea_gemv(desc: QteaDesc, packed, x, y, workspace, stream=None):
    _need_cuda(packed, x, y, workspace)
    _check(load().qtea_gemv(ctypes.byref(desc), _ptr(packed), _ptr(x), _ptr(y), _ptr(workspace),
                            workspace.numel() * workspace.element_size(), _stream(stream)),
           "qtea_gemv")


def qtea_gemm_lowbatch(desc: QteaDesc, packed, X, batch: int, Y, workspace, stream=None):
    _need_cuda(packed, X, Y, workspace)
    _check(load().qtea_gemm_lowbatch(ctypes.byref(desc), _ptr(packed), _ptr(X), int(batch), _ptr(Y),
                                     _ptr(workspace), workspace.numel() * workspace.element_size(),
                                     _stream(stream)), "qtea_gemm_lowbatch")


READ_CEILING_CHUNK = 65536  # QTEA_READ_CEILING_CHUNK


def read_ceiling_sink_words(nbytes: int) -> int:
    """Words of the sink qtea_read_ceiling needs for a buffer of nbytes."""
    return -(-int(nbytes) // READ_CEILING_CHUNK)


def qtea_read_ceiling(buf, sink, stream=None):
    """Stream the whole device buffer `buf` once; sink (device, 4-byte
    elements, at least read_ceiling_sink_words(bytes of buf)) receives one
    fold per chunk (see include/qtea.h)."""
    _need_cuda(buf, sink)
    nbytes = buf.numel() * buf.element_size()
    if sink.element_size() != 4 or sink.numel() < read_ceiling_sink_words(nbytes):
        raise ValueError("qtea_read_ceiling: sink needs one 4-byte word per 64 KiB chunk of buf")
    _check(load().qtea_read_ceiling(_ptr(buf), nbytes, _ptr(sink), _stream(stream)), "qtea_read_ceiling")


def qtea_debug_unpack(desc: QteaDesc, packed, canon_codes=None, trits=None, resid_row=None,
                      stream=None):
    _need_cuda(packed, canon_codes, trits, resid_row)
    _check(load().qtea_debug_unpack(ctypes.byref(desc), _ptr(packed), _ptr(canon_codes), _ptr(trits),
                                    _ptr(resid_row), _stream(stream)), "qtea_debug_unpack")


def qtea_grouped_plan_bytes(n_problems: int) -> int:
    out = ctypes.c_int64(0)
    _check(load().qtea_grouped_plan_bytes(int(n_problems), ctypes.byref(out)), "qtea_grouped_plan_bytes")
    return out.value


def qtea_grouped_plan(descs, packed, xs, ys, batch: int, plan, stream=None) -> QteaGroupedInfo:
    """Plan y_m = W_m x_m for independent problems m (lists of descriptors,
    packed buffers, fp16 activations, fp32 outputs: device tensors)."""
    n = len(descs)
    if not (len(packed) == len(xs) == len(ys) == n) or n < 1:
        raise ValueError("one descriptor, packed buffer, x and y per problem")
    _need_cuda(plan, *packed, *xs, *ys)
    darr = (QteaDesc * n)(*descs)
    parr = (ctypes.c_void_p * n)(*[t.data_ptr() for t in packed])
    xarr = (ctypes.c_void_p * n)(*[t.data_ptr() for t in xs])
    yarr = (ctypes.c_void_p * n)(*[t.data_ptr() for t in ys])
    info = QteaGroupedInfo()
    _check(load().qtea_grouped_plan(darr, parr, xarr, yarr, n, int(batch), _ptr(plan),
                                    plan.numel() * plan.element_size(), ctypes.byref(info),
                                    _stream(stream)), "qtea_grouped_plan")
    return info


def qtea_grouped_gemv(info: QteaGroupedInfo, plan, workspace, stream=None):
    _need_cuda(plan, workspace)
    _check(load().qtea_grouped_gemv(ctypes.byref(info), _ptr(plan), _ptr(workspace),
                                    workspace.numel() * workspace.element_size(), _stream(stream)),
           "qtea_grouped_gemv")


QTEA_NOALLOC_SCRATCH_BYTES = 16 * 1048576 + 65536


def qtea_gemm_lowbatch_noalloc(desc: QteaDesc, packed, X, batch: int, Y, stream=None):
    """qtea_gemm_lowbatch with the library's own fixed device workspace (no
    allocation; calls that overlap on one GPU race)."""
    _need_cuda(packed, X, Y)
    _check(load().qtea_gemm_lowbatch_noalloc(ctypes.byref(desc), _ptr(packed), _ptr(X), int(batch), _ptr(Y),
                                             _stream(stream)), "qtea_gemm_lowbatch_noalloc")


QTEA_QUEUE_STALE = 1  # a chunk-queue take found the counter past the plan's count
QTEA_QUEUE_COUNT = 2  # a launch's takes did not add up to the plan's count


def qtea_grouped_status(workspace, stream=None) -> int:
    """Error flags a grouped workspace has collected (0: none); synchronizes
    the stream.  Zero-filling the workspace clears them."""
    _need_cuda(workspace)
    out = ctypes.c_uint32(0)
    _check(load().qtea_grouped_status(_ptr(workspace), ctypes.byref(out), _stream(stream)), "qtea_grouped_status")
    return int(out.value)


@dataclass
class GroupedPlan:
    info: QteaGroupedInfo
    plan: object       # torch uint8 device tensor
    workspace: object  # torch uint8 device tensor (zero-filled)

    def run(self, stream=None):
        qtea_grouped_gemv(self.info, self.plan, self.workspace, stream=stream)


def plan_grouped(mats, xs, ys, batch: int = 1, stream=None) -> GroupedPlan:
    """Plan a grouped GEMV over PackedMatrix objects `mats` with activations
    `xs` and outputs `ys`; allocates the plan and a zeroed workspace."""
    import torch

    dev = mats[0].packed.device
    plan = torch.empty(qtea_grouped_plan_bytes(len(mats)), dtype=torch.uint8, device=dev)
    info = qtea_grouped_plan([m.desc for m in mats], [m.packed for m in mats], xs, ys, batch, plan,
                             stream=stream)
    ws = torch.zeros(max(int(info.workspace_bytes), 4), dtype=torch.uint8, device=dev)
    return GroupedPlan(info, plan, ws)


# ---------------------------------------------------------------------------
# Convenience: one packed matrix with its own device buffer.
# ---------------------------------------------------------------------------
@dataclass
class PackedMatrix:
    desc: QteaDesc
    packed: object  # torch uint8 device tensor

    @property
    def N(self):
        return self.desc.N

    @property
    def K(self):
        return self.desc.K


def pack_matrix(trits, alpha, v, S, R, idx, stream=None) -> PackedMatrix:
    """Allocate the packed buffer and pack (all arguments device tensors)."""
    import torch

    N, K = trits.shape
    nbytes = qtea_packed_bytes(N, K, S.numel())
    packed = torch.empty(nbytes, dtype=torch.uint8, device=trits.device)
    d = qtea_pack(trits, alpha, v, S, R, idx, packed, stream=stream)
    return PackedMatrix(d, packed)


def pack_matrix_e4m3(trits, alpha, v, bitmap, n_salient, R8, idx, stream=None) -> PackedMatrix:
    """Allocate the packed buffer and pack with E4M3 residual values and a
    salient column bitmap (all arguments device tensors)."""
    import torch

    N, K = trits.shape
    nbytes = qtea_packed_bytes_e4m3(N, K, int(n_salient))
    packed = torch.empty(nbytes, dtype=torch.uint8, device=trits.device)
    d = qtea_pack_e4m3(trits, alpha, v, bitmap, n_salient, R8, idx, packed, stream=stream)
    return PackedMatrix(d, packed)


def pack_matrix_g128(trits, alpha, beta, v, bitmap, n_salient, R8, idx, stream=None) -> PackedMatrix:
    """Allocate the packed buffer and pack in the paper's grouped format."""
    import torch

    N, K = trits.shape
    nbytes = qtea_packed_bytes_g128(N, K, int(n_salient))
    packed = torch.empty(nbytes, dtype=torch.uint8, device=trits.device)
    d = qtea_pack_g128(trits, alpha, beta, v, bitmap, n_salient, R8, idx, packed, stream=stream)
    return PackedMatrix(d, packed)


def algorithmic_bytes_g128(N: int, K: int, n_salient: int) -> int:
    """Weight bytes of one GEMV in the paper's grouped format: 26 bytes per
    row and 128-column group, fp16 scale and bias per row and group, one
    E4M3 byte and a 2-bit position per residual value, fp16 v, the int32
    salient list."""
    ng = (K + 127) // 128
    entries = (N // 4) * n_salient
    return N * ng * 26 + 4 * N * ng + entries + (2 * entries + 7) // 8 + 2 * K + 4 * n_salient


def new_workspace(desc: QteaDesc, batch: int, device="cuda"):
    """A zero-filled workspace for this matrix and batch size."""
    import torch

    n = qtea_workspace_bytes(desc, batch)
    return torch.zeros(max(n, 4), dtype=torch.uint8, device=device)


def algorithmic_bytes(N: int, K: int, n_salient: int, value_bytes: int = 2) -> int:
    """Weight bytes one GEMV must read in the paper's format: packed trits
    (ceil(K/5) bytes per row), residual values (fp16: 2 bytes, E4M3: 1)
    plus 2-bit positions for one entry per four rows of each salient column,
    fp16 alpha and v, and the int32 salient list."""
    entries = (N // 4) * n_salient
    return (N * ((K + 4) // 5) + value_bytes * entries + (2 * entries + 7) // 8 + 2 * N + 2 * K
            + 4 * n_salient)


# ---------------------------------------------------------------------------
# Offline quantizer (include/qtea_quant.h).
# ---------------------------------------------------------------------------
def qtea_quant_hessian(X, H, stream=None):
    """H [K][K] fp64 = (2/n) X^T X for X [n][K] fp32 (device tensors)."""
    import torch

    _need_cuda(X, H)
    if X.dtype != torch.float32 or H.dtype != torch.float64 or X.dim() != 2 or H.shape != (X.shape[1], X.shape[1]):
        raise ValueError("qtea_quant_hessian: X fp32 [n][K], H fp64 [K][K]")
    _check(load().qtea_quant_hessian(_ptr(X), X.shape[0], X.shape[1], _ptr(H), _stream(stream)), "qtea_quant_hessian")


def qtea_quant_workspace_bytes(N: int, K: int) -> int:
    out = ctypes.c_int64(0)
    _check(load().qtea_quant_workspace_bytes(N, K, ctypes.byref(out)), "qtea_quant_workspace_bytes")
    return int(out.value)


def qtea_quantize(W, H, params: QteaQuantParams, T, alpha, beta, v, S, bitmap, R8, idx, Q, workspace, stream=None):
    """Quantize W [N][K] (fp64) with Hessian H [K][K] (fp64) into the given
    output tensors (see include/qtea_quant.h); synchronizes the stream."""
    _need_cuda(W, H, T, alpha, beta, v, S, bitmap, R8, idx, Q, workspace)
    N, K = W.shape
    _check(load().qtea_quantize(_ptr(W), _ptr(H), N, K, ctypes.byref(params), _ptr(T), _ptr(alpha), _ptr(beta),
                                _ptr(v), _ptr(S), _ptr(bitmap), _ptr(R8), _ptr(idx), _ptr(Q), _ptr(workspace),
                                workspace.numel() * workspace.element_size(), _stream(stream)), "qtea_quantize")


def quantize_matrix(W, H, n_salient, lambda_decay=1.0, iters=2, damp=0.01, want_q=False, stream=None):
    """Allocate the outputs and a workspace and quantize one matrix; returns
    a dict of device tensors (T, alpha, beta, v, S, bitmap, R8, idx, Q)."""
    import torch

    if W.dtype != torch.float64 or H.dtype != torch.float64:
        raise ValueError("quantize_matrix: W and H are fp64")
    N, K = W.shape
    dev = W.device
    G = -(-K // QTEA_QUANT_GROUP)
    out = {
        "T": torch.empty((N, K), dtype=torch.int8, device=dev),
        "alpha": torch.empty((N, G), dtype=torch.float16, device=dev),
        "beta": torch.empty((N, G), dtype=torch.float16, device=dev),
        "v": torch.empty(K, dtype=torch.float16, device=dev),
        "S": torch.empty(max(int(n_salient), 1), dtype=torch.int32, device=dev),
        "bitmap": torch.empty(-(-K // 32), dtype=torch.int32, device=dev),
        "R8": torch.empty((max(int(n_salient), 1), N // 4), dtype=torch.uint8, device=dev),
        "idx": torch.empty((max(int(n_salient), 1), N // 4), dtype=torch.uint8, device=dev),
        "Q": torch.empty((N, K), dtype=torch.float64, device=dev) if want_q else None,
    }
    ws = torch.empty(qtea_quant_workspace_bytes(N, K), dtype=torch.uint8, device=dev)
    params = QteaQuantParams(int(n_salient), float(lambda_decay), float(damp), int(iters), 0)
    qtea_quantize(W, H, params, out["T"], out["alpha"], out["beta"], out["v"], out["S"], out["bitmap"], out["R8"],
                  out["idx"], out["Q"], ws, stream=stream)
    out["S"] = out["S"][:int(n_salient)]
    out["R8"] = out["R8"][:int(n_salient)]
    out["idx"] = out["idx"][:int(n_salient)]
    return out
