"""Python binding of libsherry (MI355X / gfx950) -- argument marshalling only.

Every function has the name of the C entry point it calls (see
include/sherry.h).  Host arrays are numpy; device buffers are torch tensors on
the current HIP device (torch supplies device memory and the stream; every
step of the computation runs in the library's kernels).  There is no CPU
fallback: importing this package raises if libsherry.so has not been built.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsherry.so")

SHERRY_OK = 0
SHERRY_E_INVALID = 1
SHERRY_E_SHAPE = 2
SHERRY_E_NOT_3_4 = 3
SHERRY_E_BUFSIZE = 4
SHERRY_E_ALIGN = 5
SHERRY_E_DEVICE = 6
SHERRY_KERNEL_AUTO = 0
SHERRY_KERNEL_GEMV = 1
SHERRY_KERNEL_MFMA = 2
SHERRY_KERNEL_SKINNY = 3
SHERRY_KERNEL_ALUT = 4
SHERRY_KERNEL_GEMV_TOK = 5
SHERRY_LAUNCH_GROUPS = 1 << 30  # flag of a grouped launch value: per-group scales
SHERRY_ALUT_MAX_K = 8192
SHERRY_MAX_K = 174720
SHERRY_MAX_M = 1 << 24
SHERRY_FUSED_MAX_K = 32768

EXPORTS = [
    "sherry_status_str", "sherry_version", "sherry_last_error", "sherry_packed_bytes", "sherry_pack",
    "sherry_unpack", "sherry_quantize_act", "sherry_gemv", "sherry_gemm", "sherry_gemm_ex",
    "sherry_gemm_kernel_for", "sherry_gemv_batched_prepare", "sherry_gemv_batched",
    "sherry_packed2_bytes", "sherry_pack2", "sherry_gemv2", "sherry_stream_read",
    "sherry_stream_read_groups", "sherry_gemv_f32", "sherry_gemv_f32_batched_prepare",
    "sherry_gemv_f32_batched", "sherry_gemm_batched_prepare", "sherry_gemm_batched",
    "sherry_gemm_channel", "sherry_gemv_f32_channel", "sherry_ternarize_pack",
    "sherry_gemm_group", "sherry_gemv_f32_group", "sherry_packed3_bytes", "sherry_pack3",
    "sherry_unpack3", "sherry_gemv3", "sherry_gemv2_batched_prepare", "sherry_gemv2_batched",
    "sherry_gemv3_batched_prepare", "sherry_gemv3_batched", "sherry_quantize_act_batched_prepare",
    "sherry_quantize_act_batched", "sherry_pack_il", "sherry_unpack_il",
    "sherry_gemv_f32_il_batched_prepare", "sherry_gemv_f32_il_batched",
    "sherry_gemm_il_batched_prepare", "sherry_gemm_il_batched", "sherry_interleave",
]


class SherryError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = "%s: %s (status %d)" % (where, _status_str(status), status)
        if status == SHERRY_E_DEVICE:
            msg += " [%s]" % lib.sherry_last_error().decode()
        super().__init__(msg)


class sherry_gemv_desc(ctypes.Structure):
    _fields_ = [
        ("w", ctypes.c_void_p), ("x", ctypes.c_void_p), ("x_scale", ctypes.c_void_p),
        ("y", ctypes.c_void_p), ("acc", ctypes.c_void_p), ("w_scales", ctypes.c_void_p),
        ("w_group_scales", ctypes.c_void_p), ("n", ctypes.c_int32), ("k", ctypes.c_int32),
        ("w_scale", ctypes.c_float), ("block_begin", ctypes.c_int32),
    ]


class sherry_gemv_f32_desc(ctypes.Structure):
    _fields_ = [
        ("w", ctypes.c_void_p), ("x", ctypes.c_void_p), ("x_scale", ctypes.c_void_p),
        ("y", ctypes.c_void_p), ("acc", ctypes.c_void_p), ("w_scales", ctypes.c_void_p),
        ("w_group_scales", ctypes.c_void_p), ("n", ctypes.c_int32), ("k", ctypes.c_int32),
        ("w_scale", ctypes.c_float), ("block_begin", ctypes.c_int32),
    ]


class sherry_gemm_desc(ctypes.Structure):
    _fields_ = [
        ("w", ctypes.c_void_p), ("x", ctypes.c_void_p), ("x_scale", ctypes.c_void_p),
        ("y", ctypes.c_void_p), ("acc", ctypes.c_void_p), ("w_scales", ctypes.c_void_p),
        ("w_group_scales", ctypes.c_void_p),
        ("n", ctypes.c_int32), ("k", ctypes.c_int32), ("m", ctypes.c_int32),
        ("w_scale", ctypes.c_float), ("block_begin", ctypes.c_int32),
        ("block_count", ctypes.c_int32),
    ]


class sherry_quant_desc(ctypes.Structure):
    _fields_ = [
        ("x", ctypes.c_void_p), ("q", ctypes.c_void_p), ("x_scale", ctypes.c_void_p),
        ("m", ctypes.c_int32), ("k", ctypes.c_int32), ("row_begin", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
    ]


def _load():
    # torch ships its own HIP runtime (same SONAME as the system's).  Loading
    # torch first makes libsherry bind to that runtime instead of mapping a
    # second HIP/HSA runtime into the process (which then sees no device).
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            "libsherry.so is not built (%s); run __graft_entry__.build() or "
            "python paper_2601_07892_amd/_build.py" % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, f32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_float
    i64p = ctypes.POINTER(ctypes.c_int64)
    sig = {
        "sherry_status_str": ([ctypes.c_int], ctypes.c_char_p),
        "sherry_version": ([], ctypes.c_char_p),
        "sherry_last_error": ([], ctypes.c_char_p),
        "sherry_packed_bytes": ([i64, i64], ctypes.c_size_t),
        "sherry_pack": ([vp, i64, i64, vp, ctypes.c_size_t, i64p], ctypes.c_int),
        "sherry_pack_il": ([vp, i64, i64, vp, ctypes.c_size_t, i64p], ctypes.c_int),
        "sherry_unpack_il": ([vp, ctypes.c_size_t, i64, i64, vp], ctypes.c_int),
        "sherry_interleave": ([vp, vp, i64, i64, vp], ctypes.c_int),
        "sherry_unpack": ([vp, ctypes.c_size_t, i64, i64, vp], ctypes.c_int),
        "sherry_quantize_act": ([vp, i64, i64, vp, vp, vp], ctypes.c_int),
        "sherry_gemv": ([vp, vp, vp, f32, vp, vp, i64, i64, vp], ctypes.c_int),
        "sherry_gemm": ([vp, vp, vp, f32, vp, vp, i64, i64, i64, vp], ctypes.c_int),
        "sherry_gemm_ex": ([vp, vp, vp, f32, vp, vp, i64, i64, i64, ctypes.c_int, vp],
                           ctypes.c_int),
        "sherry_gemm_kernel_for": ([i64, i64, i64], ctypes.c_int),
        "sherry_gemv_batched_prepare": ([ctypes.POINTER(sherry_gemv_desc), ctypes.c_int, i64p],
                                        ctypes.c_int),
        "sherry_gemv_batched": ([vp, ctypes.c_int, i64, vp], ctypes.c_int),
        "sherry_packed2_bytes": ([i64, i64], ctypes.c_size_t),
        "sherry_pack2": ([vp, i64, i64, vp, ctypes.c_size_t, i64p], ctypes.c_int),
        "sherry_gemv2": ([vp, vp, vp, f32, vp, vp, i64, i64, vp], ctypes.c_int),
        "sherry_stream_read": ([vp, ctypes.c_size_t, vp, vp], ctypes.c_int),
        "sherry_stream_read_groups": ([ctypes.c_size_t], i64),
        "sherry_gemv_f32": ([vp, vp, vp, f32, vp, vp, i64, i64, vp], ctypes.c_int),
        "sherry_gemv_f32_batched_prepare": ([ctypes.POINTER(sherry_gemv_f32_desc), ctypes.c_int,
                                             i64p], ctypes.c_int),
        "sherry_gemv_f32_il_batched_prepare": ([ctypes.POINTER(sherry_gemv_f32_desc), ctypes.c_int,
                                             i64p], ctypes.c_int),
        "sherry_gemv_f32_batched": ([vp, ctypes.c_int, i64, vp], ctypes.c_int),
        "sherry_gemv_f32_il_batched": ([vp, ctypes.c_int, i64, vp], ctypes.c_int),
        "sherry_gemm_batched_prepare": ([ctypes.POINTER(sherry_gemm_desc), ctypes.c_int, i64p,
                                         ctypes.POINTER(ctypes.c_int32)], ctypes.c_int),
        "sherry_gemm_batched": ([vp, ctypes.c_int, i64, ctypes.c_int32, vp], ctypes.c_int),
        "sherry_gemm_il_batched_prepare": ([ctypes.POINTER(sherry_gemm_desc), ctypes.c_int, i64p,
                                            ctypes.POINTER(ctypes.c_int32)], ctypes.c_int),
        "sherry_gemm_il_batched": ([vp, ctypes.c_int, i64, ctypes.c_int32, vp], ctypes.c_int),
        "sherry_gemm_channel": ([vp, vp, vp, vp, vp, vp, i64, i64, i64, ctypes.c_int, vp],
                                ctypes.c_int),
        "sherry_gemv_f32_channel": ([vp, vp, vp, vp, vp, vp, i64, i64, vp], ctypes.c_int),
        "sherry_ternarize_pack": ([vp, i64, i64, vp, ctypes.c_size_t, vp, vp], ctypes.c_int),
        "sherry_gemm_group": ([vp, vp, vp, vp, vp, vp, i64, i64, i64, ctypes.c_int, vp],
                              ctypes.c_int),
        "sherry_gemv_f32_group": ([vp, vp, vp, vp, vp, vp, i64, i64, vp], ctypes.c_int),
        "sherry_packed3_bytes": ([i64, i64], ctypes.c_size_t),
        "sherry_pack3": ([vp, i64, i64, vp, ctypes.c_size_t, i64p], ctypes.c_int),
        "sherry_unpack3": ([vp, ctypes.c_size_t, i64, i64, vp], ctypes.c_int),
        "sherry_gemv3": ([vp, vp, vp, f32, vp, vp, i64, i64, vp], ctypes.c_int),
        "sherry_gemv2_batched_prepare": ([ctypes.POINTER(sherry_gemv_desc), ctypes.c_int, i64p],
                                         ctypes.c_int),
        "sherry_gemv2_batched": ([vp, ctypes.c_int, i64, vp], ctypes.c_int),
        "sherry_gemv3_batched_prepare": ([ctypes.POINTER(sherry_gemv_desc), ctypes.c_int, i64p],
                                         ctypes.c_int),
        "sherry_gemv3_batched": ([vp, ctypes.c_int, i64, vp], ctypes.c_int),
        "sherry_quantize_act_batched_prepare": ([ctypes.POINTER(sherry_quant_desc), ctypes.c_int,
                                                 i64p, ctypes.POINTER(ctypes.c_int32)],
                                                ctypes.c_int),
        "sherry_quantize_act_batched": ([vp, ctypes.c_int, i64, ctypes.c_int32, vp],
                                        ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    return L


lib = _load()


def _status_str(st: int) -> str:
    return lib.sherry_status_str(int(st)).decode()


def _check(st: int, where: str):
    if st != SHERRY_OK:
        raise SherryError(st, where)


def _ptr(t) -> int | None:
    """Device pointer of a torch tensor (None passes through as NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is not None:
        return stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _host(a: np.ndarray, dtype) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != dtype:
        raise TypeError("expected %s, got %s" % (np.dtype(dtype), a.dtype))
    return a


def sherry_version() -> str:
    return lib.sherry_version().decode()


# ---- packing (host) ---------------------------------------------------------

def sherry_packed_bytes(n: int, k: int) -> int:
    return int(lib.sherry_packed_bytes(n, k))


def sherry_pack(t: np.ndarray, out: np.ndarray | None = None) -> np.ndarray:
    """int8 [n][k] ternary 3:4 -> uint8 packed bytes (host)."""
    t = _host(t, np.int8)
    n, k = t.shape
    nb = sherry_packed_bytes(n, k)
    if out is None:
        out = np.empty(max(nb, 1), np.uint8)
    bad = ctypes.c_int64(-1)
    st = lib.sherry_pack(t.ctypes.data, n, k, out.ctypes.data, out.nbytes, ctypes.byref(bad))
    if st == SHERRY_E_NOT_3_4:
        e = SherryError(st, "sherry_pack")
        e.bad_block = int(bad.value)
        raise e
    _check(st, "sherry_pack")
    return out


def sherry_unpack(p: np.ndarray, n: int, k: int) -> np.ndarray:
    p = _host(p, np.uint8)
    t = np.empty((n, k), np.int8)
    _check(lib.sherry_unpack(p.ctypes.data, p.nbytes, n, k, t.ctypes.data), "sherry_unpack")
    return t


def sherry_pack_il(t: np.ndarray, out: np.ndarray | None = None) -> np.ndarray:
    """int8 [n][k] ternary 3:4 -> uint8 packed bytes, lane-interleaved layout (host)."""
    t = _host(t, np.int8)
    n, k = t.shape
    nb = sherry_packed_bytes(n, k)
    if out is None:
        out = np.empty(max(nb, 1), np.uint8)
    bad = ctypes.c_int64(-1)
    st = lib.sherry_pack_il(t.ctypes.data, n, k, out.ctypes.data, out.nbytes, ctypes.byref(bad))
    if st == SHERRY_E_NOT_3_4:
        e = SherryError(st, "sherry_pack_il")
        e.bad_block = int(bad.value)
        raise e
    _check(st, "sherry_pack_il")
    return out


def sherry_unpack_il(p: np.ndarray, n: int, k: int) -> np.ndarray:
    p = _host(p, np.uint8)
    t = np.empty((n, k), np.int8)
    _check(lib.sherry_unpack_il(p.ctypes.data, p.nbytes, n, k, t.ctypes.data), "sherry_unpack_il")
    return t


def sherry_interleave(tiled, il, n: int, k: int, stream=None):
    """Device: tiled packed bytes -> lane-interleaved packed bytes."""
    _check(lib.sherry_interleave(_ptr(tiled), _ptr(il), n, k, _stream(stream)),
           "sherry_interleave")


def sherry_packed2_bytes(n: int, k: int) -> int:
    return int(lib.sherry_packed2_bytes(n, k))


def sherry_pack2(t: np.ndarray) -> np.ndarray:
    t = _host(t, np.int8)
    n, k = t.shape
    out = np.empty(max(sherry_packed2_bytes(n, k), 1), np.uint8)
    bad = ctypes.c_int64(-1)
    _check(lib.sherry_pack2(t.ctypes.data, n, k, out.ctypes.data, out.nbytes, ctypes.byref(bad)),
           "sherry_pack2")
    return out


def sherry_packed3_bytes(n: int, k: int) -> int:
    return int(lib.sherry_packed3_bytes(n, k))


def sherry_pack3(t: np.ndarray) -> np.ndarray:
    t = _host(t, np.int8)
    n, k = t.shape
    out = np.empty(max(sherry_packed3_bytes(n, k), 1), np.uint8)
    bad = ctypes.c_int64(-1)
    _check(lib.sherry_pack3(t.ctypes.data, n, k, out.ctypes.data, out.nbytes, ctypes.byref(bad)),
           "sherry_pack3")
    return out


def sherry_unpack3(p: np.ndarray, n: int, k: int) -> np.ndarray:
    p = _host(p, np.uint8)
    t = np.empty((n, k), np.int8)
    _check(lib.sherry_unpack3(p.ctypes.data, p.nbytes, n, k, t.ctypes.data), "sherry_unpack3")
    return t


# ---- device calls -------------------------------------------------------------

def sherry_quantize_act(x, q, x_scale, stream=None):
    """x fp32 [m][k] -> q int8 [m][k], x_scale fp32 [m] (device tensors)."""
    m, k = x.shape
    _check(lib.sherry_quantize_act(_ptr(x), m, k, _ptr(q), _ptr(x_scale), _stream(stream)),
           "sherry_quantize_act")


def sherry_gemv(w, x, x_scale, w_scale: float, y, acc, n: int, k: int, stream=None):
    _check(lib.sherry_gemv(_ptr(w), _ptr(x), _ptr(x_scale), float(w_scale), _ptr(y), _ptr(acc),
                           n, k, _stream(stream)), "sherry_gemv")


def sherry_gemm(w, x, x_scale, w_scale: float, y, acc, m: int, n: int, k: int, stream=None):
    _check(lib.sherry_gemm(_ptr(w), _ptr(x), _ptr(x_scale), float(w_scale), _ptr(y), _ptr(acc),
                           m, n, k, _stream(stream)), "sherry_gemm")


def sherry_gemm_ex(w, x, x_scale, w_scale: float, y, acc, m: int, n: int, k: int, kernel: int,
                   stream=None):
    _check(lib.sherry_gemm_ex(_ptr(w), _ptr(x), _ptr(x_scale), float(w_scale), _ptr(y),
                              _ptr(acc), m, n, k, int(kernel), _stream(stream)),
           "sherry_gemm_ex")


def sherry_gemm_channel(w, x, x_scale, w_scales, y, acc, m: int, n: int, k: int,
                        kernel: int = SHERRY_KERNEL_AUTO, stream=None):
    """sherry_gemm_ex with one weight scale per output channel (w_scales: fp32 [n])."""
    _check(lib.sherry_gemm_channel(_ptr(w), _ptr(x), _ptr(x_scale), _ptr(w_scales), _ptr(y),
                                   _ptr(acc), m, n, k, int(kernel), _stream(stream)),
           "sherry_gemm_channel")


def sherry_gemm_group(w, x, x_scale, w_group_scales, y, acc, m: int, n: int, k: int,
                      kernel: int = SHERRY_KERNEL_AUTO, stream=None):
    """Product with per-group weight scales (fp32 [n][ceil(k/128)])."""
    _check(lib.sherry_gemm_group(_ptr(w), _ptr(x), _ptr(x_scale), _ptr(w_group_scales), _ptr(y),
                                 _ptr(acc), m, n, k, int(kernel), _stream(stream)),
           "sherry_gemm_group")


def sherry_gemv_f32_group(w, x, x_scale, w_group_scales, y, acc, n: int, k: int, stream=None):
    """Fused quantization + M = 1 product with per-group weight scales."""
    _check(lib.sherry_gemv_f32_group(_ptr(w), _ptr(x), _ptr(x_scale), _ptr(w_group_scales),
                                     _ptr(y), _ptr(acc), n, k, _stream(stream)),
           "sherry_gemv_f32_group")


def sherry_ternarize_pack(w, n: int, k: int, packed, alpha=None, stream=None):
    """Sparse-AbsMean ternarization + packing of device fp32 w [n][k] into the
    device byte tensor packed; per-channel alpha into the fp32 [n] tensor alpha."""
    nbytes = packed.numel() * packed.element_size()
    _check(lib.sherry_ternarize_pack(_ptr(w), n, k, _ptr(packed), nbytes, _ptr(alpha),
                                     _stream(stream)), "sherry_ternarize_pack")


def sherry_quantize_act_batched_prepare(descs):
    """Fills row_begin of a ctypes array of sherry_quant_desc; returns (total_rows, max_k)."""
    total, kk = ctypes.c_int64(0), ctypes.c_int32(0)
    _check(lib.sherry_quantize_act_batched_prepare(descs, len(descs), ctypes.byref(total),
                                                   ctypes.byref(kk)),
           "sherry_quantize_act_batched_prepare")
    return int(total.value), int(kk.value)


def sherry_quantize_act_batched(descs_dev, count: int, total_rows: int, max_k: int,
                                stream=None):
    """descs_dev: device uint8 tensor holding a byte copy of prepared descriptors."""
    _check(lib.sherry_quantize_act_batched(_ptr(descs_dev), count, total_rows, max_k,
                                           _stream(stream)), "sherry_quantize_act_batched")


def sherry_gemm_kernel_for(m: int, n: int, k: int) -> int:
    return int(lib.sherry_gemm_kernel_for(m, n, k))


def sherry_gemv_batched_prepare(descs) -> int:
    """Fills block_begin of a ctypes array of sherry_gemv_desc; returns total blocks."""
    total = ctypes.c_int64(0)
    _check(lib.sherry_gemv_batched_prepare(descs, len(descs), ctypes.byref(total)),
           "sherry_gemv_batched_prepare")
    return int(total.value)


def sherry_gemv_batched(descs_dev, count: int, total_blocks: int, stream=None):
    """descs_dev: device uint8 tensor holding a byte copy of prepared descriptors."""
    _check(lib.sherry_gemv_batched(_ptr(descs_dev), count, total_blocks, _stream(stream)),
           "sherry_gemv_batched")


def sherry_gemv_f32(w, x, x_scale, w_scale: float, y, acc, n: int, k: int, stream=None):
    """Quantizes the fp32 activation row x and multiplies, in one launch."""
    _check(lib.sherry_gemv_f32(_ptr(w), _ptr(x), _ptr(x_scale), float(w_scale), _ptr(y),
                               _ptr(acc), n, k, _stream(stream)), "sherry_gemv_f32")


def sherry_gemv_f32_channel(w, x, x_scale, w_scales, y, acc, n: int, k: int, stream=None):
    """sherry_gemv_f32 with one weight scale per output channel."""
    _check(lib.sherry_gemv_f32_channel(_ptr(w), _ptr(x), _ptr(x_scale), _ptr(w_scales), _ptr(y),
                                       _ptr(acc), n, k, _stream(stream)),
           "sherry_gemv_f32_channel")


def sherry_gemv_f32_batched_prepare(descs) -> int:
    """Fills block_begin of a ctypes array of sherry_gemv_f32_desc; returns total blocks."""
    total = ctypes.c_int64(0)
    _check(lib.sherry_gemv_f32_batched_prepare(descs, len(descs), ctypes.byref(total)),
           "sherry_gemv_f32_batched_prepare")
    return int(total.value)


def sherry_gemv_f32_batched(descs_dev, count: int, total_blocks: int, stream=None):
    """descs_dev: device uint8 tensor holding a byte copy of prepared f32 descriptors."""
    _check(lib.sherry_gemv_f32_batched(_ptr(descs_dev), count, total_blocks, _stream(stream)),
           "sherry_gemv_f32_batched")


def sherry_gemv_f32_il_batched_prepare(descs) -> int:
    """As sherry_gemv_f32_batched_prepare, for lane-interleaved weights."""
    total = ctypes.c_int64(0)
    _check(lib.sherry_gemv_f32_il_batched_prepare(descs, len(descs), ctypes.byref(total)),
           "sherry_gemv_f32_il_batched_prepare")
    return int(total.value)


def sherry_gemv_f32_il_batched(descs_dev, count: int, total_blocks: int, stream=None):
    """Fused products on lane-interleaved weights (descriptors from the _il prepare)."""
    _check(lib.sherry_gemv_f32_il_batched(_ptr(descs_dev), count, total_blocks, _stream(stream)),
           "sherry_gemv_f32_il_batched")


def sherry_gemm_batched_prepare(descs) -> tuple[int, int]:
    """Fills block_begin and block_count of a ctypes array of sherry_gemm_desc
    (blocks numbered longest rows first); returns (total blocks, launch value)."""
    total = ctypes.c_int64(0)
    mm = ctypes.c_int32(0)
    _check(lib.sherry_gemm_batched_prepare(descs, len(descs), ctypes.byref(total),
                                           ctypes.byref(mm)), "sherry_gemm_batched_prepare")
    return int(total.value), int(mm.value)


def sherry_gemm_batched(descs_dev, count: int, total_blocks: int, max_m: int, stream=None):
    """descs_dev: device uint8 tensor holding a byte copy of prepared descriptors."""
    _check(lib.sherry_gemm_batched(_ptr(descs_dev), count, total_blocks, max_m, _stream(stream)),
           "sherry_gemm_batched")


def sherry_gemm_il_batched_prepare(descs) -> tuple[int, int]:
    """As sherry_gemm_batched_prepare, for lane-interleaved weights (m <= 16)."""
    total = ctypes.c_int64(0)
    mm = ctypes.c_int32(0)
    _check(lib.sherry_gemm_il_batched_prepare(descs, len(descs), ctypes.byref(total),
                                              ctypes.byref(mm)), "sherry_gemm_il_batched_prepare")
    return int(total.value), int(mm.value)


def sherry_gemm_il_batched(descs_dev, count: int, total_blocks: int, max_m: int, stream=None):
    _check(lib.sherry_gemm_il_batched(_ptr(descs_dev), count, total_blocks, max_m,
                                      _stream(stream)), "sherry_gemm_il_batched")


def sherry_gemv2(w2, x, x_scale, w_scale: float, y, acc, n: int, k: int, stream=None):
    _check(lib.sherry_gemv2(_ptr(w2), _ptr(x), _ptr(x_scale), float(w_scale), _ptr(y), _ptr(acc),
                            n, k, _stream(stream)), "sherry_gemv2")


def sherry_gemv3(w3, x, x_scale, w_scale: float, y, acc, n: int, k: int, stream=None):
    _check(lib.sherry_gemv3(_ptr(w3), _ptr(x), _ptr(x_scale), float(w_scale), _ptr(y), _ptr(acc),
                            n, k, _stream(stream)), "sherry_gemv3")


def sherry_gemv2_batched_prepare(descs) -> int:
    """As sherry_gemv_batched_prepare, for descriptors on the 2-bit layout."""
    total = ctypes.c_int64(0)
    _check(lib.sherry_gemv2_batched_prepare(descs, len(descs), ctypes.byref(total)),
           "sherry_gemv2_batched_prepare")
    return int(total.value)


def sherry_gemv2_batched(descs_dev, count: int, total_blocks: int, stream=None):
    _check(lib.sherry_gemv2_batched(_ptr(descs_dev), count, total_blocks, _stream(stream)),
           "sherry_gemv2_batched")


def sherry_gemv3_batched_prepare(descs) -> int:
    """As sherry_gemv_batched_prepare, for descriptors on the 1.67-bit layout."""
    total = ctypes.c_int64(0)
    _check(lib.sherry_gemv3_batched_prepare(descs, len(descs), ctypes.byref(total)),
           "sherry_gemv3_batched_prepare")
    return int(total.value)


def sherry_gemv3_batched(descs_dev, count: int, total_blocks: int, stream=None):
    _check(lib.sherry_gemv3_batched(_ptr(descs_dev), count, total_blocks, _stream(stream)),
           "sherry_gemv3_batched")


def sherry_stream_read(src, nbytes: int, sink, stream=None):
    _check(lib.sherry_stream_read(_ptr(src), nbytes, _ptr(sink), _stream(stream)),
           "sherry_stream_read")


def sherry_stream_read_groups(nbytes: int) -> int:
    return int(lib.sherry_stream_read_groups(nbytes))


def descs_to_bytes(descs) -> np.ndarray:
    """Raw bytes of a ctypes descriptor array (to copy to the device)."""
    return np.frombuffer(bytes(descs), dtype=np.uint8).copy()
