"""Oracle for the MoE expert stage -- TEST INFRASTRUCTURE ONLY.

Plain, slow CPU implementation of what the GPU path computes, used by the tests,
the smoke check and the benchmark's CPU-baseline leg, and by nothing else. It
shares no code with the GPU library (`paper_2512_16473_amd`), and neither imports
the other. Numerics live in `moe_oracle.c` (built to `liboracle.so` by
`oracle/build.py`); the expert-cache policy lives in `oracle/lru.py`.

Functions follow the paper (Huang, Lin, Lee, ASP-DAC 2026):
  router      -- Section I MoE layer + Table II top-K (softmax, top-k, renormalise)
  expert      -- Table II expert size read as a SwiGLU FFN
  combine     -- Section I: layer output = gate-weighted sum of expert outputs
  moe_token   -- router + chosen experts + combine for one token
  lru         -- Section III-B LRU expert cache, per-layer set of M ways
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import lru  # noqa: F401  (re-exported)

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)
_i32p = ctypes.POINTER(ctypes.c_int32)
_u16p = ctypes.POINTER(ctypes.c_uint16)


def lib():
    """Load liboracle.so (build it with `python oracle/build.py`)."""
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "liboracle.so")
        if not os.path.exists(path):
            from . import build as _b
            _b.build()
        L = ctypes.CDLL(path)
        L.oracle_router.argtypes = [_f32p, _f32p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                    _i32p, _f32p, _f64p, _f64p]
        L.oracle_router.restype = ctypes.c_int
        L.oracle_router_forced.argtypes = [_f32p, _f32p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                           _i32p, _i32p, _f32p]
        L.oracle_router_forced.restype = ctypes.c_int
        L.oracle_router_logits.argtypes = [_f32p, _f32p, ctypes.c_int, ctypes.c_int, _f64p]
        L.oracle_router_logits.restype = None
        L.oracle_expert.argtypes = [_f32p, _u16p, ctypes.c_int, ctypes.c_int, _f32p]
        L.oracle_expert.restype = None
        L.oracle_combine.argtypes = [_f32p, _f32p, ctypes.c_int, ctypes.c_int, _f32p, _f32p]
        L.oracle_combine.restype = None
        L.oracle_moe_token.argtypes = [_f32p, _f32p, ctypes.POINTER(_u16p), _u16p, ctypes.c_int,
                                       ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       _i32p, _i32p, _f32p, _f32p, _f64p]
        L.oracle_moe_token.restype = ctypes.c_int
        L.oracle_set_threads.argtypes = [ctypes.c_int]
        L.oracle_set_threads.restype = None
        L.oracle_get_threads.argtypes = []
        L.oracle_get_threads.restype = ctypes.c_int
        _LIB = L
    return _LIB


def _p(a, t):
    return a.ctypes.data_as(t)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _u16(a):
    return np.ascontiguousarray(a, dtype=np.uint16)


def set_threads(n: int) -> None:
    lib().oracle_set_threads(int(n))


def get_threads() -> int:
    return int(lib().oracle_get_threads())


def router_logits(x, wr):
    x, wr = _f32(x), _f32(wr)
    n, d = wr.shape
    out = np.empty(n, dtype=np.float64)
    lib().oracle_router_logits(_p(x, _f32p), _p(wr, _f32p), d, n, _p(out, _f64p))
    return out


def router(x, wr, k):
    """Returns (idx int32 [k], w fp32 [k], gap float, logits fp64 [n])."""
    x, wr = _f32(x), _f32(wr)
    n, d = wr.shape
    idx = np.empty(k, dtype=np.int32)
    w = np.empty(k, dtype=np.float32)
    logits = np.empty(n, dtype=np.float64)
    gap = ctypes.c_double(0.0)
    rc = lib().oracle_router(_p(x, _f32p), _p(wr, _f32p), d, n, k, _p(idx, _i32p), _p(w, _f32p),
                             _p(logits, _f64p), ctypes.byref(gap))
    if rc:
        raise ValueError(f"oracle_router: bad sizes n={n} k={k} d={d}")
    return idx, w, float(gap.value), logits


def router_forced(x, wr, k, expert_set):
    x, wr = _f32(x), _f32(wr)
    n, d = wr.shape
    s = np.ascontiguousarray(expert_set, dtype=np.int32)
    idx = np.empty(k, dtype=np.int32)
    w = np.empty(k, dtype=np.float32)
    rc = lib().oracle_router_forced(_p(x, _f32p), _p(wr, _f32p), d, n, k, _p(s, _i32p),
                                    _p(idx, _i32p), _p(w, _f32p))
    if rc:
        raise ValueError("oracle_router_forced: invalid expert set")
    return idx, w


def expert(x, slab, d, f):
    """SwiGLU expert output y fp32 [d] for one bf16 slab (uint16 [3*d*f])."""
    x, slab = _f32(x), _u16(slab)
    assert x.size == d and slab.size == 3 * d * f
    y = np.empty(d, dtype=np.float32)
    lib().oracle_expert(_p(x, _f32p), _p(slab, _u16p), d, f, _p(y, _f32p))
    return y


def combine(ys, w, y_shared=None):
    ys, w = _f32(ys), _f32(w)
    k, d = ys.shape
    out = np.empty(d, dtype=np.float32)
    ysh = None if y_shared is None else _f32(y_shared)
    lib().oracle_combine(_p(ys, _f32p), _p(w, _f32p), k, d,
                         None if ysh is None else _p(ysh, _f32p), _p(out, _f32p))
    return out


def moe_token(x, wr, slabs, k, f, shared_slab=None, f_shared=0, forced_set=None):
    """One token through one MoE layer.

    slabs: sequence of n uint16 slabs (one per expert). Returns (idx, w, out, gap).
    """
    x, wr = _f32(x), _f32(wr)
    n, d = wr.shape
    keep = [_u16(s) for s in slabs]
    assert len(keep) == n
    arr = (_u16p * n)(*[_p(s, _u16p) for s in keep])
    sh = None if shared_slab is None else _u16(shared_slab)
    idx = np.empty(k, dtype=np.int32)
    w = np.empty(k, dtype=np.float32)
    out = np.empty(d, dtype=np.float32)
    gap = ctypes.c_double(0.0)
    fs = None if forced_set is None else np.ascontiguousarray(forced_set, dtype=np.int32)
    rc = lib().oracle_moe_token(_p(x, _f32p), _p(wr, _f32p), arr,
                                None if sh is None else _p(sh, _u16p), d, f, int(f_shared), n, k,
                                None if fs is None else _p(fs, _i32p),
                                _p(idx, _i32p), _p(w, _f32p), _p(out, _f32p), ctypes.byref(gap))
    if rc:
        raise ValueError(f"oracle_moe_token failed rc={rc}")
    return idx, w, out, float(gap.value)
