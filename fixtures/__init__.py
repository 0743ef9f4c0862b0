"""Seeded synthetic inputs shared by the CPU oracle and the GPU library.

Only inputs live here (edge lists, features, weights, biases, random vertex
IDs).  None of the method's arithmetic does: aggregation, normalisation,
sampling and reordering are implemented separately by the oracle and by the
GPU library.  The heavy lifting is in ``fixgen.c`` (OpenMP C); this module is
a thin numpy wrapper around it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libfixgen.so")
_SRC = os.path.join(_HERE, "fixgen.c")

F32, BF16, F16 = 0, 1, 2
UNIFORM, NORMAL = 0, 1


def build(force: bool = True) -> str:
    """Compile fixgen.c into libfixgen.so (host code, gcc + OpenMP)."""
    if force or not os.path.exists(_SO):
        tmp = _SO + ".tmp"
        subprocess.check_call(["gcc", "-O3", "-fopenmp", "-fPIC", "-shared", "-Wall",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _SO)
    return _SO


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        i64, u64, i32, vp, dbl = (ctypes.c_int64, ctypes.c_uint64, ctypes.c_int,
                                  ctypes.c_void_p, ctypes.c_double)
        L.fx_hash.restype = u64
        L.fx_hash.argtypes = [u64, u64, i32, vp]
        L.fx_rmat.restype = i64
        L.fx_rmat.argtypes = [u64, i64, i64, dbl, dbl, dbl, vp, vp]
        L.fx_features.restype = None
        L.fx_features.argtypes = [u64, i32, i64, i64, i64, i32, vp]
        L.fx_fill_features.restype = i32
        L.fx_fill_features.argtypes = [vp, i64, i64, vp]
        L.fx_features_rows.restype = None
        L.fx_features_rows.argtypes = [u64, i32, i64, vp, i64, i32, vp]
        L.fx_weights.restype = None
        L.fx_weights.argtypes = [u64, i64, i64, i64, i64, i64, vp]
        L.fx_bias.restype = None
        L.fx_bias.argtypes = [u64, i64, i64, i64, vp]
        L.fx_attention.restype = None
        L.fx_attention.argtypes = [u64, i64, i64, vp]
        L.fx_round16.restype = None
        L.fx_round16.argtypes = [i64, vp, i32, vp]
        L.fx_random_ids.restype = i32
        L.fx_random_ids.argtypes = [u64, i64, vp]
        L.fx_relabel_edges.restype = None
        L.fx_relabel_edges.argtypes = [i64, vp, vp, vp]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def hash_u64(seed: int, tag: int, *args: int) -> int:
    a = np.array(args, dtype=np.uint64) if args else np.zeros(1, np.uint64)
    return int(lib().fx_hash(seed & (2**64 - 1), tag, len(args), _p(a)))


def rmat_edges(seed: int, n: int, e: int, a: float, b: float, c: float):
    """First ``e`` distinct RMAT pairs (u != v) in attempt order -> (src, dst) int32."""
    src = np.empty(e, np.int32)
    dst = np.empty(e, np.int32)
    r = lib().fx_rmat(seed, n, e, a, b, c, _p(src), _p(dst))
    if r < 0:
        raise RuntimeError(f"fx_rmat failed ({r}) for n={n} e={e}")
    return src, dst


def np_dtype(code: int):
    return np.float32 if code == F32 else np.uint16


def features(seed: int, dist: int, v0: int, v1: int, d: int, dtype: int = F32) -> np.ndarray:
    """Rows [v0, v1) x d of the seeded features; 16-bit types come back as uint16 bit patterns."""
    out = np.empty((v1 - v0, d), np_dtype(dtype))
    lib().fx_features(seed, dist, v0, v1, d, dtype, _p(out))
    return out


class FillCtx(ctypes.Structure):
    """Context of fx_fill_features (the chunk-loader fill callback)."""
    _fields_ = [("seed", ctypes.c_uint64), ("dist", ctypes.c_int32), ("out_dtype", ctypes.c_int32),
                ("d", ctypes.c_int64), ("threads", ctypes.c_int32)]


def feature_fill(seed: int, dist: int, d: int, dtype: int = F32, threads: int = 0):
    """(function address, context) of the native fill callback that writes the
    same rows as features(); keep the context alive while it is used."""
    ctx = FillCtx(seed & (2**64 - 1), dist, dtype, d, threads)
    fn = ctypes.cast(lib().fx_fill_features, ctypes.c_void_p).value
    return fn, ctx


def features_rows(seed: int, dist: int, ids: np.ndarray, d: int, dtype: int = F32) -> np.ndarray:
    ids = np.ascontiguousarray(ids, dtype=np.int64)
    out = np.empty((ids.size, d), np_dtype(dtype))
    lib().fx_features_rows(seed, dist, ids.size, _p(ids), d, dtype, _p(out))
    return out


def weights(seed: int, layer: int, rows: int, cols: int, fan_in: int, fan_out: int) -> np.ndarray:
    """Xavier-uniform matrix (rows = output width, cols = input width), fp32."""
    out = np.empty((rows, cols), np.float32)
    lib().fx_weights(seed, layer, rows, cols, fan_in, fan_out, _p(out))
    return out


def bias(seed: int, layer: int, d: int, fan_in: int) -> np.ndarray:
    out = np.empty(d, np.float32)
    lib().fx_bias(seed, layer, d, fan_in, _p(out))
    return out


def attention(seed: int, layer: int, d: int) -> np.ndarray:
    """GAT attention vectors [2][d] fp32: row 0 for the source, row 1 for the destination."""
    out = np.empty((2, d), np.float32)
    lib().fx_attention(seed, layer, d, _p(out))
    return out


def round16(x: np.ndarray, dtype: int) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().fx_round16(x.size, _p(x), dtype, _p(out))
    return out


def random_ids(seed: int, n: int) -> np.ndarray:
    out = np.empty(n, np.int32)
    if lib().fx_random_ids(seed, n, _p(out)) != 0:
        raise MemoryError("fx_random_ids")
    return out


def relabel_edges(new_of_old: np.ndarray, src: np.ndarray, dst: np.ndarray) -> None:
    lib().fx_relabel_edges(src.size, _p(new_of_old), _p(src), _p(dst))


def bits_to_float(x: np.ndarray, dtype: int) -> np.ndarray:
    """Widen stored feature bits to fp32 exactly (bf16: shift into the high half)."""
    if dtype == F32:
        return np.asarray(x, np.float32)
    if dtype == F16:
        return np.asarray(x, np.uint16).view(np.float16).astype(np.float32)
    return (np.asarray(x, np.uint16).astype(np.uint32) << 16).view(np.float32)
