"""ctypes wrapper over ``fathom_oracle.c`` (test infrastructure only).

Marshalling only: every number is computed by the C file, which follows the
paper step by step (see its header for the passage each function cites).
Arrays are numpy; one call handles one unit (one KV head of one sequence).
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

__all__ = [
    "build", "lib_path", "f32_to_f16_bits", "f32_to_f16_bits_array", "f16_bits_to_f64", "pack", "dequant",
    "importance", "alloc_waterfill", "depths_at", "bisect", "alloc_topr",
    "scores_f64", "scores_f32", "topk", "sparse_attn",
    "SCALE_OVERFLOW", "NONFINITE", "TOPK_SHORT",
]

SCALE_OVERFLOW = 1
NONFINITE = 2
TOPK_SHORT = 8

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fathom_oracle.c")
_LIB = os.path.join(_HERE, "_build", "liboracle.so")
_lib = None


def lib_path() -> str:
    return _LIB


def build() -> str:
    """Compile the oracle with gcc (-O2, no fused multiply-add contraction)."""
    os.makedirs(os.path.dirname(_LIB), exist_ok=True)
    tmp = _LIB + ".tmp"
    subprocess.check_call([
        "gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
        "-shared", "-Wall", "-o", tmp, _SRC, "-lm",
    ])
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = C.CDLL(_LIB)
        P = C.c_void_p
        i64, i32, u32 = C.c_int64, C.c_int, C.c_uint32
        lib.orc_f32_to_f16.restype = C.c_uint16
        lib.orc_f32_to_f16.argtypes = [C.c_float]
        lib.orc_f32_to_f16_n.restype = None
        lib.orc_f32_to_f16_n.argtypes = [P, i64, P]
        lib.orc_f16_to_f64.restype = C.c_double
        lib.orc_f16_to_f64.argtypes = [C.c_uint16]
        lib.orc_pack.restype = u32
        lib.orc_pack.argtypes = [P, i64, i32, i64, P, P]
        lib.orc_dequant.restype = C.c_double
        lib.orc_dequant.argtypes = [P, P, i64, i32, i32, i64]
        lib.orc_importance.restype = None
        lib.orc_importance.argtypes = [P, i32, i32, P, P]
        lib.orc_alloc_waterfill.restype = u32
        lib.orc_alloc_waterfill.argtypes = [P, i32, i32, P, i32, P, P]
        lib.orc_depths_at.restype = i32
        lib.orc_depths_at.argtypes = [P, i32, C.c_double, P]
        lib.orc_bisect.restype = C.c_double
        lib.orc_bisect.argtypes = [P, i32, i32, C.c_double, C.c_double, i32, P, P, P]
        lib.orc_alloc_topr.restype = u32
        lib.orc_alloc_topr.argtypes = [P, i32, i32, i32, P, P]
        lib.orc_scores_f64.restype = None
        lib.orc_scores_f64.argtypes = [P, P, i64, i64, i32, P, i32, P, P, P]
        lib.orc_scores_f32.restype = None
        lib.orc_scores_f32.argtypes = [P, P, i64, i64, i32, P, i32, P, P]
        lib.orc_topk.restype = u32
        lib.orc_topk.argtypes = [P, i64, i32, i64, i64, P, P]
        lib.orc_sparse_attn.restype = None
        lib.orc_sparse_attn.argtypes = [P, P, P, i64, i32, i32, P, i32, i32, i32, C.c_double, P]
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(C.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def f32_to_f16_bits(x: float) -> int:
    return int(_load().orc_f32_to_f16(float(np.float32(x))))


def f32_to_f16_bits_array(x: np.ndarray) -> np.ndarray:
    """orc_f32_to_f16 over an array of fp32 values (binary16 bit patterns)."""
    x = _c(x, np.float32).ravel()
    out = np.zeros(x.shape, np.uint16)
    _load().orc_f32_to_f16_n(_ptr(x), x.size, _ptr(out))
    return out


def f16_bits_to_f64(h: int) -> float:
    return float(_load().orc_f16_to_f64(int(h)))


def pack(K: np.ndarray, nb_cap: int | None = None):
    """Sec. 3.2: K [n][D] fp32 -> (planes [D][4][nb_cap] u64, scales [D][nb_cap] u16, status)."""
    K = _c(K, np.float32)
    n, D = K.shape
    nb = (n + 63) // 64
    nb_cap = nb if nb_cap is None else int(nb_cap)
    assert nb_cap >= nb
    planes = np.zeros((D, 4, nb_cap), np.uint64)
    scales = np.zeros((D, nb_cap), np.uint16)
    st = _load().orc_pack(_ptr(K), n, D, nb_cap, _ptr(planes), _ptr(scales))
    return planes, scales, int(st)


def dequant(planes, scales, j: int, t: int, i: int) -> float:
    planes = _c(planes, np.uint64)
    scales = _c(scales, np.uint16)
    return float(_load().orc_dequant(_ptr(planes), _ptr(scales), planes.shape[2], j, t, i))


def importance(q: np.ndarray, var: np.ndarray) -> np.ndarray:
    """Eq. (g) in the fp32 order fixed by the oracle; q [G][D] fp32, var [D] fp32."""
    q = _c(q, np.float32)
    var = _c(var, np.float32)
    G, D = q.shape
    g = np.zeros(D, np.float32)
    _load().orc_importance(_ptr(q), G, D, _ptr(var), _ptr(g))
    return g


def alloc_waterfill(q: np.ndarray, var: np.ndarray, B: int):
    """Eq. (wf) closed form -> (depths [D] u8, theta* float32, status)."""
    q = _c(q, np.float32)
    var = _c(var, np.float32)
    G, D = q.shape
    d = np.zeros(D, np.uint8)
    th = C.c_float(0.0)
    st = _load().orc_alloc_waterfill(_ptr(q), G, D, _ptr(var), int(B), _ptr(d), C.byref(th))
    return d, np.float32(th.value), int(st)


def depths_at(g: np.ndarray, theta: float):
    """Eq. (wf) at one theta (fp64 log4, round half up) -> (depths, sum)."""
    g = _c(g, np.float64)
    d = np.zeros(g.shape[0], np.uint8)
    s = _load().orc_depths_at(_ptr(g), g.shape[0], float(theta), _ptr(d))
    return d, int(s)


def bisect(g: np.ndarray, B: int, lo: float, hi: float, steps: int = 30):
    """App. A geometric bisection -> (final hi, depths at hi, trials, sums)."""
    g = _c(g, np.float64)
    tt = np.zeros(steps, np.float64)
    ts = np.zeros(steps, np.int32)
    d = np.zeros(g.shape[0], np.uint8)
    hi_f = _load().orc_bisect(_ptr(g), g.shape[0], int(B), float(lo), float(hi), int(steps),
                              _ptr(tt), _ptr(ts), _ptr(d))
    return float(hi_f), d, tt, ts


def alloc_topr(q: np.ndarray, r: int):
    """SparQ grouped top-r rule -> (depths [D] u8 in {0, 4}, theta, status)."""
    q = _c(q, np.float32)
    G, D = q.shape
    d = np.zeros(D, np.uint8)
    th = C.c_float(0.0)
    st = _load().orc_alloc_topr(_ptr(q), G, D, int(r), _ptr(d), C.byref(th))
    return d, np.float32(th.value), int(st)


def scores_f64(planes, scales, n: int, q, depths, with_abs: bool = False):
    """fp64 reference scores [G][n] (and sum_j |q khat| per score if asked)."""
    planes = _c(planes, np.uint64)
    scales = _c(scales, np.uint16)
    q = _c(q, np.float32)
    depths = _c(depths, np.uint8)
    D = planes.shape[0]
    G = q.shape[0]
    out = np.zeros((G, n), np.float64)
    ab = np.zeros((G, n), np.float64) if with_abs else None
    _load().orc_scores_f64(_ptr(planes), _ptr(scales), int(n), planes.shape[2], D, _ptr(q), G,
                           _ptr(depths), _ptr(out), _ptr(ab) if with_abs else None)
    return (out, ab) if with_abs else out


def scores_f32(planes, scales, n: int, q, depths):
    """fp32 score replica [G][n] in the documented channel-ascending FMA order."""
    planes = _c(planes, np.uint64)
    scales = _c(scales, np.uint16)
    q = _c(q, np.float32)
    depths = _c(depths, np.uint8)
    D = planes.shape[0]
    G = q.shape[0]
    out = np.zeros((G, n), np.float32)
    _load().orc_scores_f32(_ptr(planes), _ptr(scales), int(n), planes.shape[2], D, _ptr(q), G,
                           _ptr(depths), _ptr(out))
    return out


def topk(scores: np.ndarray, k: int, lo: int = 0, tail: int = 0):
    """Top-k of one row over [lo, n - tail) -> (idx int32 [k], val float32 [k], status)."""
    s = _c(scores, np.float32)
    idx = np.zeros(k, np.int32)
    val = np.zeros(k, np.float32)
    st = _load().orc_topk(_ptr(s), s.shape[0], int(k), int(lo), int(tail), _ptr(idx), _ptr(val))
    return idx, val, int(st)


def sparse_attn(q, K16, V16, idx, n_sink: int, n_local: int, sm_scale: float):
    """Exact attention over sink U local U idx per head -> out [G][D] fp64.

    q [G][D] fp32; K16, V16 [n][D] fp16 (or their uint16 bit patterns);
    idx [G][k] int32; sm_scale is taken as the fp32 value the kernel uses.
    """
    q = _c(q, np.float32)
    K16 = _c(np.asarray(K16).view(np.uint16), np.uint16)
    V16 = _c(np.asarray(V16).view(np.uint16), np.uint16)
    idx = _c(idx, np.int32)
    G, D = q.shape
    n = K16.shape[0]
    k = idx.shape[1] if idx.ndim == 2 else 0
    out = np.zeros((G, D), np.float64)
    _load().orc_sparse_attn(_ptr(q), _ptr(K16), _ptr(V16), n, G, D, _ptr(idx), k, int(n_sink),
                            int(n_local), float(np.float32(sm_scale)), _ptr(out))
    return out
