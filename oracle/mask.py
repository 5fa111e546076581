"""Python face of the masking-compressor oracle (paper Sec. 3.1, App. F).

TEST INFRASTRUCTURE ONLY: the C definition in ``mask_oracle.c`` does the
work; this module marshals numpy arrays into it.  Arrays of bf16 values are
carried as their uint16 bit patterns.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

F32, BF16 = 0, 1


def _lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "_mask_oracle.so")
        if not os.path.exists(path):
            from . import build as _b
            _b.build()
        lib = C.CDLL(path)
        u64, u32, i32, i64 = C.c_uint64, C.c_uint32, C.c_int, C.c_int64
        lib.orc_mix64.restype = u64
        lib.orc_mix64.argtypes = [u64]
        lib.orc_fmix32.restype = u32
        lib.orc_fmix32.argtypes = [u32]
        lib.orc_mask_key.restype = u64
        lib.orc_mask_key.argtypes = [u64, u32, u64, u32, u32, u32, u32]
        lib.orc_row_key.restype = u64
        lib.orc_row_key.argtypes = [u64, u64]
        lib.orc_domain_bits.restype = i32
        lib.orc_domain_bits.argtypes = [u32]
        lib.orc_feistel.restype = u32
        lib.orc_feistel.argtypes = [u32, i32, u64]
        lib.orc_perm.restype = u32
        lib.orc_perm.argtypes = [u32, u32, u64]
        lib.orc_keep_count.restype = i32
        lib.orc_keep_count.argtypes = [i32, C.c_double, C.POINTER(i32)]
        lib.orc_row_indices.restype = i32
        lib.orc_row_indices.argtypes = [u64, u64, u32, u32, C.c_void_p]
        lib.orc_pack.restype = i32
        lib.orc_pack.argtypes = [C.c_void_p, i32, i64, i32, i64, i32, u64, i64, C.c_void_p, C.c_void_p]
        lib.orc_unpack.restype = i32
        lib.orc_unpack.argtypes = [C.c_void_p, C.c_void_p, i32, i64, i32, i32, u64, i64, C.c_float,
                                   C.c_void_p, i64]
        lib.orc_mask_dense.restype = i32
        lib.orc_mask_dense.argtypes = [i64, i32, i32, u64, i64, C.c_void_p]
        lib.orc_bern_threshold.restype = i32
        lib.orc_bern_threshold.argtypes = [C.c_double, C.POINTER(i32)]
        lib.orc_bern_kept.restype = i32
        lib.orc_bern_kept.argtypes = [u64, u32, i32]
        lib.orc_bern_row_ptr.restype = i32
        lib.orc_bern_row_ptr.argtypes = [u64, i64, i32, i32, i64, C.c_void_p]
        lib.orc_bern_pack.restype = i32
        lib.orc_bern_pack.argtypes = [C.c_void_p, i32, i64, i32, i64, i32, u64, i64, C.c_void_p, C.c_void_p,
                                      C.c_void_p]
        lib.orc_bern_unpack.restype = i32
        lib.orc_bern_unpack.argtypes = [C.c_void_p, C.c_void_p, i32, i64, i32, i32, u64, i64, C.c_void_p,
                                        C.c_float, C.c_void_p, i64]
        lib.orc_bf16_from_double.restype = C.c_uint16
        lib.orc_bf16_from_double.argtypes = [C.c_double]
        lib.orc_bf16_to_double.restype = C.c_double
        lib.orc_bf16_to_double.argtypes = [C.c_uint16]
        _LIB = lib
    return _LIB


def mix64(z: int) -> int:
    return int(_lib().orc_mix64(z & (2 ** 64 - 1)))


def fmix32(h: int) -> int:
    return int(_lib().orc_fmix32(h & 0xFFFFFFFF))


def mask_key(seed: int, layer: int, step: int, microbatch: int, B: int, S: int, H: int) -> int:
    """64-bit key of g(layer, step, B, S, H) with a seed and a microbatch id."""
    return int(_lib().orc_mask_key(seed, layer, step, microbatch, B, S, H))


def row_key(key: int, row: int) -> int:
    return int(_lib().orc_row_key(key, row))


def domain_bits(H: int) -> int:
    return int(_lib().orc_domain_bits(H))


def feistel(x: int, w: int, rk: int) -> int:
    return int(_lib().orc_feistel(x, w, rk))


def perm(i: int, H: int, rk: int) -> int:
    return int(_lib().orc_perm(i, H, rk))


def keep_count(H: int, keep: float) -> int:
    """K = round(keep * H) (Sec. 3.1), ties away from zero; ValueError if K is
    not in [1, H]."""
    k = C.c_int(0)
    if _lib().orc_keep_count(H, keep, C.byref(k)) != 0:
        raise ValueError(f"invalid keep={keep} for H={H}")
    return k.value


def row_indices(key: int, row: int, H: int, K: int) -> np.ndarray:
    out = np.zeros(K, dtype=np.uint32)
    if _lib().orc_row_indices(key, row, H, K, out.ctypes.data) != 0:
        raise ValueError("bad K")
    return out


def indices(key: int, rows: int, H: int, K: int, row0: int = 0) -> np.ndarray:
    """[rows, K] kept indices (ascending per row) for rows row0 .. row0+rows-1."""
    out = np.zeros((rows, K), dtype=np.uint32)
    for r in range(rows):
        out[r] = row_indices(key, row0 + r, H, K)
    return out


def mask_dense(key: int, rows: int, H: int, K: int, row0: int = 0) -> np.ndarray:
    m = np.zeros((rows, H), dtype=np.uint8)
    if _lib().orc_mask_dense(rows, H, K, key, row0, m.ctypes.data) != 0:
        raise ValueError("bad K")
    return m


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    raise TypeError("expected float32 values or uint16 bf16 bit patterns")


def pack(x: np.ndarray, K: int, key: int, row0: int = 0, with_idx: bool = True):
    """vals[r, i] = x[r, I_r[i]], idx[r, i] = I_r[i] (Sec. 3.1: only the K kept
    values of each token cross the boundary)."""
    x = np.ascontiguousarray(x)
    rows, H = x.shape
    vals = np.zeros((rows, K), dtype=x.dtype)
    idx = np.zeros((rows, K), dtype=np.uint16) if with_idx else None
    rc = _lib().orc_pack(x.ctypes.data, x.dtype.itemsize, rows, H, H, K, key, row0,
                         vals.ctypes.data, idx.ctypes.data if idx is not None else None)
    if rc != 0:
        raise ValueError("pack failed")
    return vals, idx


def unpack(vals: np.ndarray, H: int, key: int, scale: float = 1.0, idx=None, row0: int = 0):
    """Dense y with y[r, I_r[i]] = round(vals[r, i] * scale) and +0 elsewhere
    (Sec. 3.1 masking; App. F receiver-side rescale)."""
    vals = np.ascontiguousarray(vals)
    rows, K = vals.shape
    code = _dtype_code(vals)
    y = np.zeros((rows, H), dtype=vals.dtype)
    ip = None
    if idx is not None:
        idx = np.ascontiguousarray(idx, dtype=np.uint16)
        ip = idx.ctypes.data
    rc = _lib().orc_unpack(vals.ctypes.data, ip, code, rows, H, K, key, row0,
                           np.float32(scale), y.ctypes.data, H)
    if rc != 0:
        raise ValueError("unpack failed")
    return y


def bf16_from_double(v: float) -> int:
    return int(_lib().orc_bf16_from_double(v))


def bf16_to_double(h: int) -> float:
    return float(_lib().orc_bf16_to_double(h))


# --------------------------------------------------------------------------
# Bernoulli variant (App. F): each entry kept independently, rows of variable
# length laid out by row_ptr.
# --------------------------------------------------------------------------
def bern_threshold(keep: float) -> int:
    """T = round(keep * 65536) in [1, 65536]; inclusion probability T / 65536."""
    t = C.c_int(0)
    if _lib().orc_bern_threshold(keep, C.byref(t)) != 0:
        raise ValueError(f"invalid keep={keep}")
    return t.value


def bern_kept(key: int, row: int, j: int, keep: float) -> bool:
    return bool(_lib().orc_bern_kept(row_key(key, row), j, bern_threshold(keep)))


def bern_row_ptr(key: int, rows: int, H: int, keep: float, row0: int = 0) -> np.ndarray:
    """row_ptr [rows + 1] of rows row0 .. row0 + rows - 1, starting at 0."""
    rp = np.zeros(rows + 1, dtype=np.int64)
    _lib().orc_bern_row_ptr(key, rows, H, bern_threshold(keep), row0, rp.ctypes.data)
    return rp


def bern_mask_dense(key: int, rows: int, H: int, keep: float, row0: int = 0) -> np.ndarray:
    T = bern_threshold(keep)
    m = np.zeros((rows, H), dtype=np.uint8)
    lib = _lib()
    for r in range(rows):
        rk = row_key(key, row0 + r)
        for j in range(H):
            m[r, j] = lib.orc_bern_kept(rk, j, T)
    return m


def bern_pack(x: np.ndarray, keep: float, key: int, row0: int = 0, with_idx: bool = True):
    """(row_ptr, vals, idx): the kept entries of every row, ascending, in one
    flat array (App. F Bernoulli mask; only kept values cross the link)."""
    x = np.ascontiguousarray(x)
    rows, H = x.shape
    rp = bern_row_ptr(key, rows, H, keep, row0)
    nnz = int(rp[-1])
    vals = np.zeros(max(nnz, 1), dtype=x.dtype)[:nnz]
    idx = np.zeros(max(nnz, 1), dtype=np.uint16)[:nnz] if with_idx else None
    rc = _lib().orc_bern_pack(x.ctypes.data, x.dtype.itemsize, rows, H, H, bern_threshold(keep), key, row0,
                              rp.ctypes.data, vals.ctypes.data, idx.ctypes.data if idx is not None else None)
    if rc != 0:
        raise ValueError("bern_pack failed")
    return rp, vals, idx


def bern_unpack(vals: np.ndarray, row_ptr: np.ndarray, H: int, key: int, keep: float, scale: float = 1.0,
                idx=None, row0: int = 0):
    """Dense y: round(scale * value) at the kept entries, +0 elsewhere."""
    vals = np.ascontiguousarray(vals)
    rp = np.ascontiguousarray(row_ptr, dtype=np.int64)
    rows = rp.size - 1
    code = _dtype_code(vals)
    y = np.zeros((rows, H), dtype=vals.dtype)
    ip = None
    if idx is not None:
        idx = np.ascontiguousarray(idx, dtype=np.uint16)
        ip = idx.ctypes.data
    _lib().orc_bern_unpack(vals.ctypes.data, ip, code, rows, H, bern_threshold(keep), key, row0, rp.ctypes.data,
                           np.float32(scale), y.ctypes.data, H)
    return y
