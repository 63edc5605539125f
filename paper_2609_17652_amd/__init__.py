"""Fathom per-query variable-depth key scan on MI355X (gfx950).

A thin ctypes binding over ``libfathom.so`` (declared in ``include/fathom.h``):
the functions below carry the C names and only marshal arguments -- tensors
in, device pointers and sizes out to the C ABI, the caller's current HIP
stream, status codes turned into exceptions.  Every step of the path runs in
the library's HIP kernels; PyTorch provides device memory and streams.  There
is no CPU fallback: if the library is not built, every call raises.
"""
from __future__ import annotations

import ctypes as C
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "_lib", "libfathom.so")

# status codes and device-status bits (include/fathom.h)
FATHOM_OK = 0
FATHOM_ERR_INVALID = -1
FATHOM_ERR_UNSUPPORTED = -2
FATHOM_ERR_RANGE = -3
FATHOM_ERR_HIP = -4
FATHOM_ERR_WORKSPACE = -5
FATHOM_F32 = 0
FATHOM_F16 = 1
FATHOM_WATERFILL = 0
FATHOM_UNIFORM_TOPR = 1
FATHOM_MAX_K = 8192
FATHOM_DEV_SCALE_OVERFLOW = 1
FATHOM_DEV_NONFINITE = 2
FATHOM_DEV_TOPK_FALLBACK = 4
FATHOM_DEV_TOPK_SHORT = 8
FATHOM_DEV_BAD_N = 16

EXPORTED = (
    "fathom_pack", "fathom_pack_append", "fathom_gather_store", "fathom_alloc_depths", "fathom_scan", "fathom_topk", "fathom_topk_workspace_size",
    "fathom_scan_topk", "fathom_scan_topk_ex", "fathom_scan_topk_workspace_size", "fathom_scan_topk_noalloc",
    "fathom_scan_topk_noalloc_capacity", "fathom_sparse_attn",
    "fathom_sparse_attn_workspace_size", "fathom_klt_calibrate", "fathom_klt_calibrate_workspace_size",
    "fathom_klt_rotate_keys", "fathom_klt_rotate_q", "fathom_status_string", "fathom_version",
)


class FathomError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {fathom_status_string(code)} ({code})")


_lib = None


def lib() -> C.CDLL:
    """The loaded C library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"libfathom.so is not built ({LIB_PATH}); run `python -m paper_2609_17652_amd.build` "
                "(or __graft_entry__.build()) first -- there is no fallback path")
        L = C.CDLL(LIB_PATH)
        P, i64, i32, st = C.c_void_p, C.c_int64, C.c_int, C.c_int
        sig = {
            "fathom_pack": [P, i32, i64, i64, P, i32, i32, i64, P, P, P, P],
            "fathom_pack_append": [P, i32, i64, i64, P, P, i64, i32, i32, i64, P, P, P, P],
            "fathom_gather_store": [P, P, P, i32, i32, i64, P, P, P],
            "fathom_alloc_depths": [P, i32, i32, i32, i32, P, i32, i32, P, P, P, P],
            "fathom_scan": [P, P, P, i32, i32, i64, P, i32, i32, P, P, i64, P, P],
            "fathom_topk": [P, i64, P, i32, i32, i32, i64, i64, P, P, P, C.c_size_t, P, P],
            "fathom_scan_topk": [P, P, P, i32, i32, i64, P, i32, i32, P, i32, i64, i64, P, P, P, C.c_size_t, P, P],
            "fathom_scan_topk_ex": [P, P, P, i32, i32, i64, P, i32, i32, P, i32, i64, i64, i32, P, P, P, C.c_size_t, P,
                                    P],
            "fathom_scan_topk_noalloc": [P, P, P, i32, i32, i64, P, i32, i32, P, i32, i64, i64, i32, P, P, P, P],
            "fathom_sparse_attn": [P, i32, P, P, i64, i64, P, i32, i32, i32, P, i32, i32, i32, C.c_float, P, P,
                                   C.c_size_t, P, P],
            "fathom_klt_calibrate": [P, i32, i64, i64, P, i64, i32, i32, P, P, P, P, C.c_size_t, P, P],
            "fathom_klt_rotate_keys": [P, i32, i64, i64, P, i64, i32, i32, P, P, P, i64, P, P],
            "fathom_klt_rotate_q": [P, i32, i32, i32, i32, P, P, P],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = st
        for name in ("fathom_topk_workspace_size", "fathom_scan_topk_workspace_size"):
            f = getattr(L, name)
            f.argtypes = [i32, i32, i64, i32]
            f.restype = C.c_size_t
        L.fathom_scan_topk_noalloc_capacity.argtypes = []
        L.fathom_scan_topk_noalloc_capacity.restype = C.c_size_t
        L.fathom_sparse_attn_workspace_size.argtypes = [i32, i32, i32, i32, i32]
        L.fathom_sparse_attn_workspace_size.restype = C.c_size_t
        L.fathom_klt_calibrate_workspace_size.argtypes = [i32]
        L.fathom_klt_calibrate_workspace_size.restype = C.c_size_t
        L.fathom_status_string.argtypes = [st]
        L.fathom_status_string.restype = C.c_char_p
        L.fathom_version.argtypes = []
        L.fathom_version.restype = C.c_char_p
        _lib = L
    return _lib


def fathom_status_string(code: int) -> str:
    return lib().fathom_status_string(int(code)).decode()


def fathom_version() -> str:
    return lib().fathom_version().decode()


def _p(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return FATHOM_F32
    if t.dtype == torch.float16:
        return FATHOM_F16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _check(code: int, where: str):
    if code != FATHOM_OK:
        raise FathomError(code, where)


def _dev(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("fathom calls take device tensors")


def new_status(device=None) -> torch.Tensor:
    """A zeroed device status word (int32 view of the uint32 the kernels OR into)."""
    return torch.zeros(1, dtype=torch.int32, device=device or "cuda")


def fathom_pack(K, n, nb_cap=None, planes=None, scales=None, dev_status=None, stream=None):
    """Sec. 3.2: K [U][n][D] (fp32/fp16, channel stride 1) -> (planes [U][D][4][nb_cap] u64 as int64,
    scales [U][D][nb_cap] fp16 bits as int16)."""
    _dev(K, n)
    U, ntok, D = K.shape
    if K.stride(2) != 1:
        raise ValueError("K channel stride must be 1")
    nb_cap = (ntok + 63) // 64 if nb_cap is None else int(nb_cap)
    if planes is None:
        planes = torch.empty((U, D, 4, nb_cap), dtype=torch.int64, device=K.device)
    if scales is None:
        scales = torch.empty((U, D, nb_cap), dtype=torch.int16, device=K.device)
    _check(lib().fathom_pack(_p(K), _dt(K), K.stride(1), K.stride(0), _p(n), U, D, nb_cap, _p(planes), _p(scales),
                             _p(dev_status), _stream(stream)), "fathom_pack")
    return planes, scales


def fathom_pack_append(K, n_old, n, max_new, planes, scales, dev_status=None, stream=None):
    """Sec. 3.2 on a growing cache: re-packs, per unit, blocks floor(n_old/64) .. ceil(n/64)-1 of
    (planes, scales) from K [U][>= n][D]; afterwards they equal fathom_pack of the first n tokens."""
    _dev(K, n_old, n, planes, scales)
    U, _, D = K.shape
    if K.stride(2) != 1:
        raise ValueError("K channel stride must be 1")
    nb_cap = planes.shape[-1]
    _check(lib().fathom_pack_append(_p(K), _dt(K), K.stride(1), K.stride(0), _p(n_old), _p(n), int(max_new), U, D,
                                    nb_cap, _p(planes), _p(scales), _p(dev_status), _stream(stream)),
           "fathom_pack_append")
    return planes, scales


def fathom_gather_store(host_planes, host_scales, depths, planes, scales, stream=None):
    """Sec. 3.6: copy the rows the depths read from a pinned host store into the device store."""
    if not (host_planes.is_pinned() and host_scales.is_pinned()):
        raise ValueError("the host store must be pinned host memory")
    _dev(depths, planes, scales)
    U, D, _, nb_cap = planes.shape
    if tuple(host_planes.shape) != tuple(planes.shape) or tuple(host_scales.shape) != tuple(scales.shape):
        raise ValueError("host and device stores must have the same shape")
    _check(lib().fathom_gather_store(_p(host_planes), _p(host_scales), _p(depths), U, D, nb_cap, _p(planes),
                                     _p(scales), _stream(stream)), "fathom_gather_store")
    return planes, scales


def fathom_alloc_depths(q, var, mode=FATHOM_WATERFILL, budget_or_r=48, depths=None, theta=None,
                        dev_status=None, stream=None):
    """Sec. 3.3: q [U][G][D] (fp32/fp16, contiguous), var [U][D] fp32 -> (depths [U][D] u8, theta [U] fp32)."""
    _dev(q, var)
    U, G, D = q.shape
    if not q.is_contiguous() or (var is not None and not var.is_contiguous()):
        raise ValueError("q and var must be contiguous")
    if depths is None:
        depths = torch.empty((U, D), dtype=torch.uint8, device=q.device)
    if theta is None:
        theta = torch.empty((U,), dtype=torch.float32, device=q.device)
    _check(lib().fathom_alloc_depths(_p(q), _dt(q), U, G, D, _p(var), int(mode), int(budget_or_r), _p(depths),
                                     _p(theta), _p(dev_status), _stream(stream)), "fathom_alloc_depths")
    return depths, theta


def fathom_scan(planes, scales, n, q, depths, scores=None, ld_s=None, dev_status=None, stream=None):
    """Sec. 3.2-3.3: approximate scores [U][G][ld_s] fp32 (ld_s defaults to 64 * nb_cap)."""
    _dev(planes, scales, n, q, depths)
    U, D, _, nb_cap = planes.shape
    G = q.shape[1]
    if scores is None:
        ld_s = 64 * nb_cap if ld_s is None else int(ld_s)
        scores = torch.empty((U, G, ld_s), dtype=torch.float32, device=q.device)
    else:
        ld_s = scores.shape[-1] if ld_s is None else int(ld_s)
    _check(lib().fathom_scan(_p(planes), _p(scales), _p(n), U, D, nb_cap, _p(q), _dt(q), G, _p(depths), _p(scores),
                             ld_s, _p(dev_status), _stream(stream)), "fathom_scan")
    return scores


def fathom_topk_workspace_size(U, G, max_n, k) -> int:
    return int(lib().fathom_topk_workspace_size(int(U), int(G), int(max_n), int(k)))


def fathom_scan_topk_workspace_size(U, G, max_n, k) -> int:
    return int(lib().fathom_scan_topk_workspace_size(int(U), int(G), int(max_n), int(k)))


def _ws(nbytes, ws, device):
    if ws is None:
        ws = torch.empty((max(int(nbytes), 1),), dtype=torch.uint8, device=device)
    return ws


def fathom_topk(scores, n, k, lo=0, tail=0, idx=None, val=None, ws=None, dev_status=None, stream=None):
    """Sec. 2: per-head top-k of scores [U][G][ld_s] over [lo, n - tail) -> (idx [U][G][k] i32, val fp32)."""
    _dev(scores, n)
    U, G, ld_s = scores.shape
    if idx is None:
        idx = torch.empty((U, G, k), dtype=torch.int32, device=scores.device)
    if val is None:
        val = torch.empty((U, G, k), dtype=torch.float32, device=scores.device)
    ws = _ws(fathom_topk_workspace_size(U, G, ld_s, k), ws, scores.device)
    _check(lib().fathom_topk(_p(scores), ld_s, _p(n), U, G, int(k), int(lo), int(tail), _p(idx), _p(val), _p(ws),
                             ws.numel() * ws.element_size(), _p(dev_status), _stream(stream)), "fathom_topk")
    return idx, val


def fathom_scan_topk(planes, scales, n, q, depths, k, lo=0, tail=0, idx=None, val=None, ws=None, dev_status=None,
                     stream=None, max_unit_bits=0):
    """fathom_scan + fathom_topk in one call (no score array output).  max_unit_bits: the caller's
    bound on every unit's depth bits (0: none); it selects work only, never the result."""
    _dev(planes, scales, n, q, depths)
    U, D, _, nb_cap = planes.shape
    G = q.shape[1]
    if idx is None:
        idx = torch.empty((U, G, k), dtype=torch.int32, device=q.device)
    if val is None:
        val = torch.empty((U, G, k), dtype=torch.float32, device=q.device)
    ws = _ws(fathom_scan_topk_workspace_size(U, G, 64 * nb_cap, k), ws, q.device)
    _check(lib().fathom_scan_topk_ex(_p(planes), _p(scales), _p(n), U, D, nb_cap, _p(q), _dt(q), G, _p(depths),
                                     int(k), int(lo), int(tail), int(max_unit_bits), _p(idx), _p(val), _p(ws),
                                     ws.numel() * ws.element_size(), _p(dev_status), _stream(stream)),
           "fathom_scan_topk")
    return idx, val


def fathom_scan_topk_noalloc_capacity() -> int:
    return int(lib().fathom_scan_topk_noalloc_capacity())


def fathom_scan_topk_noalloc(planes, scales, n, q, depths, k, lo, tail, idx, val, dev_status=None, stream=None,
                             max_unit_bits=0):
    """fathom_scan_topk with the library's own device workspace: nothing is allocated, here or in the call
    (idx and val are the caller's [U][G][k] outputs)."""
    _dev(planes, scales, n, q, depths, idx, val)
    U, D, _, nb_cap = planes.shape
    G = q.shape[1]
    _check(lib().fathom_scan_topk_noalloc(_p(planes), _p(scales), _p(n), U, D, nb_cap, _p(q), _dt(q), G, _p(depths),
                                          int(k), int(lo), int(tail), int(max_unit_bits), _p(idx), _p(val),
                                          _p(dev_status), _stream(stream)), "fathom_scan_topk_noalloc")
    return idx, val


def fathom_sparse_attn_workspace_size(U, G, k, n_sink=0, n_local=0) -> int:
    return int(lib().fathom_sparse_attn_workspace_size(int(U), int(G), int(k), int(n_sink), int(n_local)))


def fathom_sparse_attn(q, Krows, Vrows, n, idx, n_sink=0, n_local=0, sm_scale=None, out=None, dev_status=None,
                       stream=None, ws=None):
    """Sec. 2: exact attention over sink + local + idx rows; Krows/Vrows [U][n][D] fp16 -> out [U][G][D] fp32."""
    _dev(q, Krows, Vrows, n, idx)
    U, G, D = q.shape
    if Krows.dtype != torch.float16 or Vrows.dtype != torch.float16:
        raise TypeError("K/V rows must be fp16")
    if Krows.stride() != Vrows.stride() or Krows.stride(2) != 1 or not q.is_contiguous():
        raise ValueError("K and V rows need the same strides with channel stride 1; q contiguous")
    k = 0 if idx is None else idx.shape[-1]
    if sm_scale is None:
        sm_scale = 1.0 / (D ** 0.5)
    if out is None:
        out = torch.empty((U, G, D), dtype=torch.float32, device=q.device)
    wsb = fathom_sparse_attn_workspace_size(U, G, k, n_sink, n_local)
    ws = _ws(wsb, ws, q.device)
    _check(lib().fathom_sparse_attn(_p(q), _dt(q), _p(Krows), _p(Vrows), Krows.stride(1), Krows.stride(0), _p(n),
                                    U, G, D, _p(idx), k, int(n_sink), int(n_local), C.c_float(sm_scale), _p(out),
                                    _p(ws), ws.numel(), _p(dev_status), _stream(stream)), "fathom_sparse_attn")
    return out


# ---------------------------------------------------------------- KLT-rotated store (Sec. 3.5)
def fathom_klt_calibrate_workspace_size(U) -> int:
    return int(lib().fathom_klt_calibrate_workspace_size(int(U)))


def fathom_klt_calibrate(K, n, mu=None, V=None, lam=None, ws=None, dev_status=None, stream=None):
    """Sec. 3.5: per unit, the mean mu [U][D], eigenbasis V [U][D][D] (column c = eigenvector c) and
    eigenvalues lam [U][D] (descending) of the first n[u] keys of K [U][n_cap][D] (fp32 or fp16)."""
    _dev(K, n)
    U, ncap, D = K.shape
    if K.stride(2) != 1:
        raise ValueError("K channel stride must be 1")
    f32 = dict(dtype=torch.float32, device=K.device)
    mu = torch.empty((U, D), **f32) if mu is None else mu
    V = torch.empty((U, D, D), **f32) if V is None else V
    lam = torch.empty((U, D), **f32) if lam is None else lam
    ws = _ws(fathom_klt_calibrate_workspace_size(U), ws, K.device)
    _check(lib().fathom_klt_calibrate(_p(K), _dt(K), K.stride(1), K.stride(0), _p(n), ncap, U, D, _p(mu), _p(V),
                                      _p(lam), _p(ws), ws.numel(), _p(dev_status), _stream(stream)),
           "fathom_klt_calibrate")
    return mu, V, lam


def fathom_klt_rotate_keys(K, n, mu, V, out=None, dev_status=None, stream=None):
    """Sec. 3.5: (k - mu) V for the first n[u] keys of each unit -> fp32 [U][n_cap][D] (rows past n[u]
    are left as they were); pack it with fathom_pack."""
    _dev(K, n, mu, V)
    U, ncap, D = K.shape
    if K.stride(2) != 1 or not mu.is_contiguous() or not V.is_contiguous():
        raise ValueError("K channel stride 1; mu and V contiguous")
    if mu.dtype != torch.float32 or V.dtype != torch.float32:
        raise TypeError("mu and V must be fp32")
    if out is None:
        out = torch.empty((U, ncap, D), dtype=torch.float32, device=K.device)
    if out.dtype != torch.float32 or out.stride(2) != 1 or out.stride(1) != D:
        raise ValueError("out must be fp32 rows of D floats")
    _check(lib().fathom_klt_rotate_keys(_p(K), _dt(K), K.stride(1), K.stride(0), _p(n), ncap, U, D, _p(mu), _p(V),
                                        _p(out), out.stride(0), _p(dev_status), _stream(stream)),
           "fathom_klt_rotate_keys")
    return out


def fathom_klt_rotate_q(q, V, out=None, stream=None):
    """Sec. 3.5: q_h V per (unit, head) -> fp32 [U][G][D]."""
    _dev(q, V)
    U, G, D = q.shape
    if not q.is_contiguous() or not V.is_contiguous() or V.dtype != torch.float32:
        raise ValueError("q contiguous; V contiguous fp32")
    if out is None:
        out = torch.empty((U, G, D), dtype=torch.float32, device=q.device)
    _check(lib().fathom_klt_rotate_q(_p(q), _dt(q), U, G, D, _p(V), _p(out), _stream(stream)), "fathom_klt_rotate_q")
    return out
