"""CPU oracle for the Sherry 3:4 ternary product -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never does, and
this package never imports the product: the two share no code.

The arithmetic lives in ``sherry_oracle.c`` (plain C, built with gcc); this
module only marshals numpy arrays through ctypes.  Each function names the
passage of the paper it follows; see the header of ``sherry_oracle.c``.

Parity status of each piece (what pins it, in ``tests/test_oracle.py``):

* code table         -- pinned: hand-derived table (tests/golden), exhaustive
                         counts (32 of 81 tuples, Sec. 3.1), mirror pairs
                         (16, Appendix C);
* pack / unpack      -- pinned: hand-derived byte fixtures (tests/golden),
                         round trips, 3:4 rejection;
* act. quantization  -- pinned: absmax -> +-127, exact multiples, RNE ties,
                         zero rows, clamp;
* product            -- pinned: numpy int64 matmul, pure-Python brute force,
                         one-hot / all-ones closed forms;
* epilogue           -- pinned: exactly representable scale products;
* ternarizer         -- pinned: brute force over all 32 patterns per block
                         (Appendix D) and least-squares alpha (Eq. 5);
* 2-bit codec        -- pinned: hand-derived bytes and round trips.
* 1.67-bit codec     -- pinned: hand-derived code table and bytes, 27 of the
                         32 codes used (3^3 triples, Sec. 2.3), mirror
                         code(-t) = 26 - code(t), rejection of the unused
                         codes, round trips.
* lane-interleaved   -- pinned: hand-derived bytes (tests/golden), round
  layout                 trips, the same multiset of codes per unit as the
                         tiled layout, 3:4 rejection.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sherry_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (plain -O2, no intrinsics)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call([
            "gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
            "-fno-fast-math", "-pthread", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = ctypes.CDLL(_LIB)
        i8p = ctypes.POINTER(ctypes.c_int8)
        u8p = ctypes.POINTER(ctypes.c_uint8)
        i64 = ctypes.c_int64
        L.oracle_code_table.argtypes = [i8p]
        L.oracle_code_table.restype = ctypes.c_int
        L.oracle_encode_block.argtypes = [i8p]
        L.oracle_encode_block.restype = ctypes.c_int
        L.oracle_decode_code.argtypes = [ctypes.c_int, i8p]
        L.oracle_decode_code.restype = None
        L.oracle_packed_bytes.argtypes = [i64, i64]
        L.oracle_packed_bytes.restype = i64
        L.oracle_pack.argtypes = [i8p, i64, i64, u8p]
        L.oracle_pack.restype = i64
        L.oracle_unpack.argtypes = [u8p, i64, i64, i8p]
        L.oracle_unpack.restype = ctypes.c_int
        L.oracle_quantize_act.argtypes = [ctypes.POINTER(ctypes.c_float), i64, i64, i8p,
                                          ctypes.POINTER(ctypes.c_float)]
        L.oracle_quantize_act.restype = None
        L.oracle_gemm_i32.argtypes = [i8p, i8p, i64, i64, i64,
                                      ctypes.POINTER(ctypes.c_int32), ctypes.c_int]
        L.oracle_gemm_i32.restype = None
        L.oracle_dot_i32.argtypes = [i8p, i8p, i64]
        L.oracle_dot_i32.restype = ctypes.c_int32
        L.oracle_epilogue.argtypes = [ctypes.POINTER(ctypes.c_int32),
                                      ctypes.POINTER(ctypes.c_float), ctypes.c_float,
                                      i64, i64, ctypes.POINTER(ctypes.c_double)]
        L.oracle_epilogue.restype = None
        L.oracle_ternarize.argtypes = [ctypes.POINTER(ctypes.c_float), i64, i64, i8p]
        L.oracle_ternarize.restype = ctypes.c_double
        L.oracle_ternarize_rows.argtypes = [ctypes.POINTER(ctypes.c_float), i64, i64, i8p,
                                            ctypes.POINTER(ctypes.c_double)]
        L.oracle_ternarize_rows.restype = None
        L.oracle_epilogue_rows.argtypes = [ctypes.POINTER(ctypes.c_int32),
                                           ctypes.POINTER(ctypes.c_float),
                                           ctypes.POINTER(ctypes.c_float), i64, i64,
                                           ctypes.POINTER(ctypes.c_double)]
        L.oracle_epilogue_rows.restype = None
        L.oracle_packed2_bytes.argtypes = [i64, i64]
        L.oracle_packed2_bytes.restype = i64
        L.oracle_pack2.argtypes = [i8p, i64, i64, u8p]
        L.oracle_pack2.restype = i64
        L.oracle_unpack2.argtypes = [u8p, i64, i64, i8p]
        L.oracle_unpack2.restype = ctypes.c_int
        L.oracle_code3_table.argtypes = [i8p]
        L.oracle_code3_table.restype = ctypes.c_int
        L.oracle_encode3.argtypes = [i8p]
        L.oracle_encode3.restype = ctypes.c_int
        L.oracle_packed3_bytes.argtypes = [i64, i64]
        L.oracle_packed3_bytes.restype = i64
        L.oracle_pack3.argtypes = [i8p, i64, i64, u8p]
        L.oracle_pack3.restype = i64
        L.oracle_unpack3.argtypes = [u8p, i64, i64, i8p]
        L.oracle_unpack3.restype = ctypes.c_int
        L.oracle_pack_il.argtypes = [i8p, i64, i64, u8p]
        L.oracle_pack_il.restype = i64
        L.oracle_unpack_il.argtypes = [u8p, i64, i64, i8p]
        L.oracle_unpack_il.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a: np.ndarray, ct):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.POINTER(ct))


class OracleError(ValueError):
    pass


# ---- (i) code table (Sec. 3.1 point 3) -----------------------------------

def code_table() -> np.ndarray:
    """int8 [32][4]: weights of each 5-bit code, built by enumeration."""
    t = np.zeros((32, 4), dtype=np.int8)
    n = lib().oracle_code_table(_p(t, ctypes.c_int8))
    if n != 32:
        raise OracleError("code table enumeration accepted %d tuples" % n)
    return t


def encode_block(w) -> int:
    a = np.ascontiguousarray(np.asarray(w, dtype=np.int8).reshape(4))
    return int(lib().oracle_encode_block(_p(a, ctypes.c_int8)))


def decode_code(c: int) -> np.ndarray:
    w = np.zeros(4, dtype=np.int8)
    lib().oracle_decode_code(int(c), _p(w, ctypes.c_int8))
    return w


# ---- (ii) packed layout (Appendix A, offline packing) --------------------

def packed_bytes(n: int, k: int) -> int:
    return int(lib().oracle_packed_bytes(n, k))


def pack(t: np.ndarray) -> np.ndarray:
    t = np.ascontiguousarray(t, dtype=np.int8)
    n, k = t.shape
    nb = packed_bytes(n, k)
    if nb == 0:
        raise OracleError("bad shape %s" % (t.shape,))
    out = np.zeros(nb, dtype=np.uint8)
    rc = lib().oracle_pack(_p(t, ctypes.c_int8), n, k, _p(out, ctypes.c_uint8))
    if rc != 0:
        raise OracleError("block %d is not 3:4" % (-rc - 1))
    return out


def pack_bad_block(t: np.ndarray):
    """Flat index of the first non-3:4 block, or None if T packs."""
    t = np.ascontiguousarray(t, dtype=np.int8)
    n, k = t.shape
    out = np.zeros(packed_bytes(n, k), dtype=np.uint8)
    rc = lib().oracle_pack(_p(t, ctypes.c_int8), n, k, _p(out, ctypes.c_uint8))
    return None if rc == 0 else int(-rc - 1)


def unpack(p: np.ndarray, n: int, k: int) -> np.ndarray:
    p = np.ascontiguousarray(p, dtype=np.uint8)
    if p.size < packed_bytes(n, k):
        raise OracleError("packed buffer too small")
    t = np.zeros((n, k), dtype=np.int8)
    if lib().oracle_unpack(_p(p, ctypes.c_uint8), n, k, _p(t, ctypes.c_int8)) != 0:
        raise OracleError("bad shape")
    return t


# ---- (ix) lane-interleaved layout (this project's own) ---------------------

def pack_il(t: np.ndarray) -> np.ndarray:
    t = np.ascontiguousarray(t, dtype=np.int8)
    n, k = t.shape
    nb = packed_bytes(n, k)
    if nb == 0:
        raise OracleError("bad shape %s" % (t.shape,))
    out = np.zeros(nb, dtype=np.uint8)
    rc = lib().oracle_pack_il(_p(t, ctypes.c_int8), n, k, _p(out, ctypes.c_uint8))
    if rc != 0:
        raise OracleError("block %d is not 3:4" % (-rc - 1))
    return out


def unpack_il(p: np.ndarray, n: int, k: int) -> np.ndarray:
    p = np.ascontiguousarray(p, dtype=np.uint8)
    if p.size < packed_bytes(n, k):
        raise OracleError("packed buffer too small")
    t = np.zeros((n, k), dtype=np.int8)
    if lib().oracle_unpack_il(_p(p, ctypes.c_uint8), n, k, _p(t, ctypes.c_int8)) != 0:
        raise OracleError("bad shape")
    return t


# ---- (iii) activation quantization ---------------------------------------

def quantize_act(x: np.ndarray):
    """fp32 [m][k] -> (int8 [m][k], fp32 sx [m]); absmax/127, RNE, clamp."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim == 1:
        x = x[None, :]
    m, k = x.shape
    q = np.zeros((m, k), dtype=np.int8)
    sx = np.zeros(m, dtype=np.float32)
    lib().oracle_quantize_act(_p(x, ctypes.c_float), m, k, _p(q, ctypes.c_int8),
                              _p(sx, ctypes.c_float))
    return q, sx


# ---- (iv) product of Eq. 2 on the unpacked T ------------------------------

def gemm_i32(x: np.ndarray, t: np.ndarray, threads: int = 1) -> np.ndarray:
    """acc [m][n] = x [m][k] . t[n][k]^T in exact integers."""
    x = np.ascontiguousarray(x, dtype=np.int8)
    t = np.ascontiguousarray(t, dtype=np.int8)
    if x.ndim == 1:
        x = x[None, :]
    m, k = x.shape
    n, k2 = t.shape
    if k != k2:
        raise OracleError("k mismatch")
    acc = np.zeros((m, n), dtype=np.int32)
    lib().oracle_gemm_i32(_p(x, ctypes.c_int8), _p(t, ctypes.c_int8), m, n, k,
                          _p(acc, ctypes.c_int32), int(threads))
    return acc


def dot_i32(x_row: np.ndarray, t_row: np.ndarray) -> int:
    x_row = np.ascontiguousarray(x_row, dtype=np.int8)
    t_row = np.ascontiguousarray(t_row, dtype=np.int8)
    return int(lib().oracle_dot_i32(_p(x_row, ctypes.c_int8), _p(t_row, ctypes.c_int8),
                                    x_row.size))


# ---- (v) epilogue (Eq. 2 scaling), fp64 -----------------------------------

def epilogue(acc: np.ndarray, sx: np.ndarray, sw: float) -> np.ndarray:
    acc = np.ascontiguousarray(acc, dtype=np.int32)
    sx = np.ascontiguousarray(sx, dtype=np.float32)
    m, n = acc.shape
    y = np.zeros((m, n), dtype=np.float64)
    lib().oracle_epilogue(_p(acc, ctypes.c_int32), _p(sx, ctypes.c_float),
                          ctypes.c_float(sw), m, n, _p(y, ctypes.c_double))
    return y


def epilogue_rows(acc: np.ndarray, sx: np.ndarray, sw: np.ndarray) -> np.ndarray:
    """Per-output-channel scales ([T alpha]_ij = T_ij alpha_j): y = acc*sx[m]*sw[n]."""
    acc = np.ascontiguousarray(acc, dtype=np.int32)
    sx = np.ascontiguousarray(sx, dtype=np.float32)
    sw = np.ascontiguousarray(sw, dtype=np.float32)
    m, n = acc.shape
    assert sx.shape == (m,) and sw.shape == (n,)
    y = np.zeros((m, n), dtype=np.float64)
    lib().oracle_epilogue_rows(_p(acc, ctypes.c_int32), _p(sx, ctypes.c_float),
                               _p(sw, ctypes.c_float), m, n, _p(y, ctypes.c_double))
    return y


GROUP = 128  # weights per scale group along K (the paper's group size 128)


def product_groups(x: np.ndarray, t: np.ndarray, sx: np.ndarray, s_groups: np.ndarray,
                   threads: int = 1):
    """Per-group weight scales (group size 128 along K, the paper's default
    granularity): y[m][n] = sx[m] * sum_g acc_g[m][n] * s[n][g], where acc_g
    is the exact integer product over K values [128 g, 128 g + 128).  fp64.

    Returns (y, mag, acc): mag[m][n] = sx[m] * sum_g |acc_g * s[n][g]| (the
    scale of the rounding error of any fp32 summation order) and acc the
    int32 sum over all groups."""
    x = np.ascontiguousarray(x, dtype=np.int8)
    t = np.ascontiguousarray(t, dtype=np.int8)
    if x.ndim == 1:
        x = x[None, :]
    m, k = x.shape
    n = t.shape[0]
    g_count = (k + GROUP - 1) // GROUP
    s_groups = np.asarray(s_groups, dtype=np.float32)
    if s_groups.shape != (n, g_count):
        raise OracleError("group scales must be [n][ceil(k/128)]")
    sx = np.asarray(sx, dtype=np.float32).astype(np.float64)
    y = np.zeros((m, n), dtype=np.float64)
    mag = np.zeros((m, n), dtype=np.float64)
    acc = np.zeros((m, n), dtype=np.int64)
    for g in range(g_count):
        lo, hi = g * GROUP, min(k, (g + 1) * GROUP)
        a = gemm_i32(x[:, lo:hi], t[:, lo:hi], threads=threads).astype(np.float64)
        term = a * s_groups[:, g].astype(np.float64)[None, :]
        y += term
        mag += np.abs(term)
        acc += a.astype(np.int64)
    return y * sx[:, None], mag * sx[:, None], acc.astype(np.int32)


# ---- (vi) Sparse-AbsMean ternarizer (Eq. 4, Eq. 5) -------------------------

def ternarize(w: np.ndarray):
    """fp32 [n][k] -> (int8 T [n][k], per-tensor alpha as float)."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    n, k = w.shape
    t = np.zeros((n, k), dtype=np.int8)
    alpha = lib().oracle_ternarize(_p(w, ctypes.c_float), n, k, _p(t, ctypes.c_int8))
    return t, float(alpha)


def ternarize_rows(w: np.ndarray):
    """fp32 [n][k] -> (int8 T [n][k], fp64 alpha [n]): Eq. 5 per output channel."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    n, k = w.shape
    t = np.zeros((n, k), dtype=np.int8)
    alpha = np.zeros(n, dtype=np.float64)
    lib().oracle_ternarize_rows(_p(w, ctypes.c_float), n, k, _p(t, ctypes.c_int8),
                                _p(alpha, ctypes.c_double))
    return t, alpha


# ---- (vii) 2-bit layout ----------------------------------------------------

def packed2_bytes(n: int, k: int) -> int:
    return int(lib().oracle_packed2_bytes(n, k))


def pack2(t: np.ndarray) -> np.ndarray:
    t = np.ascontiguousarray(t, dtype=np.int8)
    n, k = t.shape
    out = np.zeros(packed2_bytes(n, k), dtype=np.uint8)
    rc = lib().oracle_pack2(_p(t, ctypes.c_int8), n, k, _p(out, ctypes.c_uint8))
    if rc != 0:
        raise OracleError("bad weight at %d" % (-rc - 1))
    return out


def unpack2(p: np.ndarray, n: int, k: int) -> np.ndarray:
    p = np.ascontiguousarray(p, dtype=np.uint8)
    t = np.zeros((n, k), dtype=np.int8)
    if lib().oracle_unpack2(_p(p, ctypes.c_uint8), n, k, _p(t, ctypes.c_int8)) != 0:
        raise OracleError("bad 2-bit stream")
    return t


# ---- (viii) 1.67-bit layout (three weights per 5-bit code, Sec. 2.3) --------

def code3_table():
    """(27 x 3) int8 table: row c = the weights (t0, t1, t2) of code c, and
    the count of codes the enumeration used."""
    t = np.zeros((27, 3), dtype=np.int8)
    used = lib().oracle_code3_table(_p(t, ctypes.c_int8))
    return t, int(used)


def encode3(w) -> int:
    a = np.ascontiguousarray(np.asarray(w, dtype=np.int8))
    return int(lib().oracle_encode3(_p(a, ctypes.c_int8)))


def packed3_bytes(n: int, k: int) -> int:
    return int(lib().oracle_packed3_bytes(n, k))


def pack3(t: np.ndarray) -> np.ndarray:
    t = np.ascontiguousarray(t, dtype=np.int8)
    n, k = t.shape
    out = np.zeros(packed3_bytes(n, k), dtype=np.uint8)
    rc = lib().oracle_pack3(_p(t, ctypes.c_int8), n, k, _p(out, ctypes.c_uint8))
    if rc != 0:
        raise OracleError("bad weight at %d" % (-rc - 1))
    return out


def unpack3(p: np.ndarray, n: int, k: int) -> np.ndarray:
    p = np.ascontiguousarray(p, dtype=np.uint8)
    t = np.zeros((n, k), dtype=np.int8)
    if lib().oracle_unpack3(_p(p, ctypes.c_uint8), n, k, _p(t, ctypes.c_int8)) != 0:
        raise OracleError("bad 1.67-bit stream")
    return t


# ---- convenience: the whole path on the CPU --------------------------------

def linear(x_f32: np.ndarray, t: np.ndarray, sw: float, threads: int = 1):
    """Quantize x, multiply by T, scale: returns (q, sx, acc, y_fp64)."""
    q, sx = quantize_act(x_f32)
    acc = gemm_i32(q, t, threads)
    return q, sx, acc, epilogue(acc, sx, sw)
