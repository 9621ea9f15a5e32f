"""MI355X (gfx950) MoE expert stage for single-request decode.

Thin Python binding over libmoe.so (include/moe.h): every step of the path runs in
the library's HIP kernels and host C++ runtime; this module only marshals
arguments. Device buffers are torch tensors on the GPU (torch provides device
memory and streams); host buffers are numpy arrays or pinned torch tensors.

The library must be built (python paper_2512_16473_amd/build.py); importing this
package fails loudly otherwise. There is no fallback implementation.
"""
from __future__ import annotations

import ctypes

import numpy as np

from . import _abi
from ._abi import LayerDesc, PrefillDesc, RuntimeStats
from ._abi import MAX_D, MAX_EXPERTS, MAX_TOKENS, MAX_TOPK  # noqa: F401  (ABI bounds)

_lib = _abi.load()

__all__ = [
    "MoeError", "lib", "slab_bytes", "router_topk", "Cache", "ffn_workspace_bytes", "expert_ffn_hits",
    "combine", "PinnedBuffer", "HostPool", "Runtime", "prefill_workspace_bytes", "prefill_forward", "read_stream",
    "ffn_tokens_workspace_bytes", "expert_ffn_tokens", "ffn_noalloc_max_bytes", "expert_ffn_hits_noalloc",
]


class MoeError(RuntimeError):
    def __init__(self, fn, code):
        msg = _lib.moe_last_error().decode(errors="replace")
        super().__init__(f"{fn} failed ({code}): {msg}")
        self.code = code


def lib():
    return _lib


def _check(fn, rc):
    if rc != _abi.MOE_OK:
        raise MoeError(fn, rc)


def _ptr(t):
    """Device/host address of a torch tensor (or None)."""
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _np_ptr(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def slab_bytes(d: int, f: int) -> int:
    return int(_lib.moe_slab_bytes(d, f))


# --------------------------------------------------------------------------- router
def router_topk(x, w_router, k, idx_out=None, w_out=None, stream=None):
    """x: cuda fp32 [T, d]; w_router: cuda fp32 [n, d]. Returns (idx int32 [T,k], w fp32 [T,k])."""
    import torch
    T, d = x.shape
    n = w_router.shape[0]
    if idx_out is None:
        idx_out = torch.empty((T, k), dtype=torch.int32, device=x.device)
    if w_out is None:
        w_out = torch.empty((T, k), dtype=torch.float32, device=x.device)
    _check("moe_router_topk", _lib.moe_router_topk(_ptr(x), _ptr(w_router), T, d, n, k, _ptr(idx_out),
                                                   _ptr(w_out), _stream(stream)))
    return idx_out, w_out


# --------------------------------------------------------------------------- cache
POLICIES = {"lru": 0, "fifo": 1, "static": 2}


class Cache:
    """Host slot table of the per-layer expert cache (policy "lru", "fifo" or
    "static"; `static_content` [n_layers][ways] for "static")."""

    def __init__(self, n_layers, n_experts, ways, top_k, policy="lru", static_content=None):
        h = ctypes.c_void_p()
        if policy == "static":
            content = np.ascontiguousarray(static_content, dtype=np.int32).reshape(n_layers, ways)
            cptr = _np_ptr(content, ctypes.c_int32)
        else:
            content, cptr = None, None
        _check("moe_cache_create_policy", _lib.moe_cache_create_policy(n_layers, n_experts, ways, top_k,
                                                                       POLICIES[policy], cptr, ctypes.byref(h)))
        self.handle = h
        self.n_layers, self.n, self.ways, self.k, self.policy = n_layers, n_experts, ways, top_k, policy

    def close(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.moe_cache_destroy(self.handle)
            self.handle = None

    __del__ = close

    def reset(self):
        _check("moe_cache_reset", _lib.moe_cache_reset(self.handle))

    def lookup(self, layer, experts):
        e = np.ascontiguousarray(experts, dtype=np.int32)
        slots = np.empty(e.size, np.int32)
        hits = np.empty(e.size, np.uint8)
        _check("moe_cache_lookup", _lib.moe_cache_lookup(self.handle, layer, _np_ptr(e, ctypes.c_int32), e.size,
                                                         _np_ptr(slots, ctypes.c_int32),
                                                         _np_ptr(hits, ctypes.c_uint8)))
        return slots, hits.astype(bool)

    def update(self, layer, experts):
        e = np.ascontiguousarray(experts, dtype=np.int32)
        fill = np.empty(e.size, np.int32)
        ev = np.empty(e.size, np.int32)
        _check("moe_cache_update", _lib.moe_cache_update(self.handle, layer, _np_ptr(e, ctypes.c_int32), e.size,
                                                         _np_ptr(fill, ctypes.c_int32), _np_ptr(ev, ctypes.c_int32)))
        return fill, ev

    def update_masked(self, layer, experts, insert):
        e = np.ascontiguousarray(experts, dtype=np.int32)
        ins = np.ascontiguousarray(insert, dtype=np.uint8)
        fill = np.empty(e.size, np.int32)
        ev = np.empty(e.size, np.int32)
        _check("moe_cache_update_masked",
               _lib.moe_cache_update_masked(self.handle, layer, _np_ptr(e, ctypes.c_int32), e.size,
                                            _np_ptr(ins, ctypes.c_uint8), _np_ptr(fill, ctypes.c_int32),
                                            _np_ptr(ev, ctypes.c_int32)))
        return fill, ev

    def slotmap(self, layer):
        m = np.empty(self.n, np.int32)
        _check("moe_cache_slotmap", _lib.moe_cache_slotmap(self.handle, layer, _np_ptr(m, ctypes.c_int32)))
        return m

    def save(self) -> bytes:
        """The cache state (slots, recency stamps, set clocks) as bytes."""
        nb = int(_lib.moe_cache_state_bytes(self.handle))
        buf = ctypes.create_string_buffer(nb)
        _check("moe_cache_save", _lib.moe_cache_save(self.handle, buf, nb))
        return buf.raw

    def restore(self, state: bytes):
        """Load a state saved from a cache of the same geometry, policy and content."""
        buf = ctypes.create_string_buffer(bytes(state), len(state))
        _check("moe_cache_restore", _lib.moe_cache_restore(self.handle, buf, len(state)))


def cache_geometry(budget_bytes, expert_bytes, ways, n_layers):
    """(slots S, covered layers min(N, n_layers)) for a memory budget (Section III-B)."""
    S, N = ctypes.c_int(), ctypes.c_int()
    _check("moe_cache_geometry", _lib.moe_cache_geometry(int(budget_bytes), int(expert_bytes), ways, n_layers,
                                                         ctypes.byref(S), ctypes.byref(N)))
    return S.value, N.value


# --------------------------------------------------------------------------- hit FFN / combine
def ffn_workspace_bytes(max_jobs, d, f_max) -> int:
    return int(_lib.moe_ffn_workspace_bytes(max_jobs, d, f_max))


def expert_ffn_hits(x, slot_pool, n_slots, hit_slots, hit_w, d, f, y, workspace, stream=None):
    """y = sum_j hit_w[j] FFN(slot hit_slots[j]) (x); all cuda tensors."""
    n_hits = int(hit_slots.numel())
    _check("moe_expert_ffn_hits", _lib.moe_expert_ffn_hits(
        _ptr(x), _ptr(slot_pool), n_slots, _ptr(hit_slots), _ptr(hit_w), n_hits, d, f, _ptr(y),
        _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream)))
    return y


def ffn_noalloc_max_bytes() -> int:
    return int(_lib.moe_ffn_noalloc_max_bytes())


def expert_ffn_hits_noalloc(x, slot_pool, n_slots, hit_slots, hit_w, d, f, y, stream=None):
    """expert_ffn_hits with the library's static device scratch instead of a workspace
    (allocates nothing; calls that overlap on one device race)."""
    n_hits = int(hit_slots.numel())
    _check("moe_expert_ffn_hits_noalloc", _lib.moe_expert_ffn_hits_noalloc(
        _ptr(x), _ptr(slot_pool), n_slots, _ptr(hit_slots), _ptr(hit_w), n_hits, d, f, _ptr(y), _stream(stream)))
    return y


def ffn_tokens_workspace_bytes(T, k, d, f) -> int:
    return int(_lib.moe_ffn_tokens_workspace_bytes(T, k, d, f))


def expert_ffn_tokens(x, slot_pool, n_slots, slots, w, d, f, y, workspace, stream=None):
    """y[t] = sum_j w[t][j] FFN(slot slots[t][j]) (x[t]) for T small-batch tokens, each
    selected slab read once; x, y cuda fp32 [T, d], slots int32 / w fp32 cuda [T, k]."""
    T, k = int(slots.shape[0]), int(slots.shape[1])
    _check("moe_expert_ffn_tokens", _lib.moe_expert_ffn_tokens(
        _ptr(x), _ptr(slot_pool), n_slots, _ptr(slots), _ptr(w), T, k, d, f, _ptr(y),
        _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream)))
    return y


def combine(out, y_gpu=None, y_host=None, y_shared=None, stream=None):
    d = out.numel()
    _check("moe_combine", _lib.moe_combine(_ptr(y_gpu), _ptr(y_host), _ptr(y_shared), d, _ptr(out),
                                           _stream(stream)))
    return out


# --------------------------------------------------------------------------- host path
class PinnedBuffer:
    """Page-locked host buffer from moe_host_alloc, exposed as a numpy uint8 array."""

    def __init__(self, nbytes: int):
        p = ctypes.c_void_p()
        _check("moe_host_alloc", _lib.moe_host_alloc(int(nbytes), ctypes.byref(p)))
        self.ptr = p.value
        self.nbytes = int(nbytes)
        self.array = np.ctypeslib.as_array((ctypes.c_uint8 * self.nbytes).from_address(self.ptr))

    def close(self):
        if getattr(self, "ptr", None) and _lib is not None:
            self.array = None
            _lib.moe_host_free(ctypes.c_void_p(self.ptr))
            self.ptr = None

    __del__ = close


class HostPool:
    """Host thread pool running missed experts (n_threads <= 0: OMP_NUM_THREADS / all cores)."""

    def __init__(self, n_threads=0):
        h = ctypes.c_void_p()
        _check("moe_host_pool_create", _lib.moe_host_pool_create(n_threads, ctypes.byref(h)))
        self.handle = h

    @property
    def threads(self):
        return int(_lib.moe_host_pool_threads(self.handle))

    @property
    def dot(self):
        """Form of the row dot products: "fp32" (widened weights) or "bf16" (pair-dot)."""
        v = int(_lib.moe_host_pool_get_dot(self.handle))
        return {1: "fp32", 2: "bf16"}[v]

    def set_dot(self, kind):
        """kind: "auto", "fp32" or "bf16" (MoeError if the CPU lacks AVX512_BF16)."""
        _check("moe_host_pool_set_dot", _lib.moe_host_pool_set_dot(self.handle, _abi.HOST_DOT[kind]))

    def close(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.moe_host_pool_destroy(self.handle)
            self.handle = None

    __del__ = close

    def expert_ffn(self, x, slabs, w, d, f, y=None):
        """x fp32 [d] numpy; slabs: list of host arrays/tensors (bf16 bit patterns); w fp32 [ne]."""
        x = np.ascontiguousarray(x, dtype=np.float32)
        w = np.ascontiguousarray(w, dtype=np.float32)
        ptrs = (ctypes.c_void_p * max(1, len(slabs)))(*[_host_addr(s) for s in slabs])
        if y is None:
            y = np.empty(d, np.float32)
        _check("moe_host_expert_ffn", _lib.moe_host_expert_ffn(self.handle, _np_ptr(x, ctypes.c_float), ptrs,
                                                               _np_ptr(w, ctypes.c_float), len(slabs), d, f,
                                                               _np_ptr(y, ctypes.c_float)))
        return y


def _host_addr(a):
    if hasattr(a, "data_ptr"):
        return a.data_ptr()
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


# --------------------------------------------------------------------------- runtime
class Runtime:
    """Per-layer decode runtime (steps 1-3 of the method) over caller-owned buffers.

    w_router: cuda fp32 [L, n, d]; slot_pool: cuda uint8 (covered*ways slabs, where
    covered = cache.n_layers <= L; None when no layer is covered);
    shared_pool: cuda uint8 (L slabs of d x f_shared) or None;
    host_slabs: sequence of L*n host addresses (ints) of pinned bf16 slabs.
    """

    def __init__(self, d, f, n, k, ways, n_layers, w_router, slot_pool, host_slabs, cache: Cache,
                 pool: HostPool, f_shared=0, shared_pool=None):
        self._keep = (w_router, slot_pool, shared_pool, cache, pool)
        arr = (ctypes.c_void_p * len(host_slabs))(*[int(a) for a in host_slabs])
        desc = LayerDesc(d, f, n, k, ways, n_layers, f_shared, w_router.data_ptr(),
                         slot_pool.data_ptr() if slot_pool is not None else None,
                         shared_pool.data_ptr() if shared_pool is not None else None,
                         ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p)), cache.handle, pool.handle)
        h = ctypes.c_void_p()
        _check("moe_runtime_create", _lib.moe_runtime_create(ctypes.byref(desc), ctypes.byref(h)))
        self.handle = h
        self.d, self.f, self.n, self.k, self.ways, self.L = d, f, n, k, ways, n_layers

    def close(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.moe_runtime_destroy(self.handle)
            self.handle = None

    __del__ = close

    def layer_forward(self, layer, x, out, streams):
        idx = np.empty(self.k, np.int32)
        w = np.empty(self.k, np.float32)
        hit = np.empty(self.k, np.uint8)
        sc, sa, sw = streams
        _check("moe_layer_forward", _lib.moe_layer_forward(
            self.handle, layer, _ptr(x), _ptr(out), _np_ptr(idx, ctypes.c_int32), _np_ptr(w, ctypes.c_float),
            _np_ptr(hit, ctypes.c_uint8), _stream(sc), _stream(sa), _stream(sw)))
        return idx, w, hit.astype(bool)

    def decode_step(self, x, out, streams, idx=None, w=None, hit=None):
        """x, out: cuda fp32 [L, d]. idx/w/hit: optional numpy [L, k] outputs."""
        sc, sa, sw = streams
        _check("moe_decode_step", _lib.moe_decode_step(
            self.handle, _ptr(x), _ptr(out),
            None if idx is None else _np_ptr(idx, ctypes.c_int32),
            None if w is None else _np_ptr(w, ctypes.c_float),
            None if hit is None else _np_ptr(hit, ctypes.c_uint8),
            _stream(sc), _stream(sa), _stream(sw)))

    def sync(self):
        _check("moe_runtime_sync", _lib.moe_runtime_sync(self.handle))

    def device_slotmap(self, layer):
        m = np.empty(self.n, np.int32)
        _check("moe_runtime_device_slotmap", _lib.moe_runtime_device_slotmap(self.handle, layer,
                                                                             _np_ptr(m, ctypes.c_int32)))
        return m

    def set_timing(self, on: bool):
        _check("moe_runtime_set_timing", _lib.moe_runtime_set_timing(self.handle, 1 if on else 0))

    def set_nonblocking(self, enable=True):
        _check("moe_runtime_set_nonblocking", _lib.moe_runtime_set_nonblocking(self.handle, int(bool(enable))))

    def set_fill_limit(self, max_slabs_in_flight):
        _check("moe_runtime_set_fill_limit", _lib.moe_runtime_set_fill_limit(self.handle, int(max_slabs_in_flight)))

    def stats(self) -> dict:
        s = RuntimeStats()
        _check("moe_runtime_get_stats", _lib.moe_runtime_get_stats(self.handle, ctypes.byref(s)))
        return {name: getattr(s, name) for name, _ in RuntimeStats._fields_}

    def reset_stats(self):
        _check("moe_runtime_reset_stats", _lib.moe_runtime_reset_stats(self.handle))


# --------------------------------------------------------------------------- prefill
def prefill_workspace_bytes(d, f, n, k, T) -> int:
    P = PrefillDesc(d, f, n, k, None, None)
    return int(_lib.moe_prefill_workspace_bytes(ctypes.byref(P), T))


def prefill_forward(X, w_router, expert_pool, d, f, n, k, OUT, workspace, idx=None, w=None, stream=None):
    """OUT[t] = routed SwiGLU expert output of X[t] (all experts resident in expert_pool)."""
    T = X.shape[0]
    P = PrefillDesc(d, f, n, k, w_router.data_ptr(), expert_pool.data_ptr())
    _check("moe_prefill_forward", _lib.moe_prefill_forward(
        ctypes.byref(P), _ptr(X), T, _ptr(OUT), _ptr(idx), _ptr(w), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))
    return OUT


# --------------------------------------------------------------------------- yardstick
def read_stream(buf, nbytes, sink, grid=0, stream=None):
    """Plain nontemporal read of nbytes of the device tensor buf (the HBM read ceiling
    used as a yardstick for the weight-streaming kernels); sink is a device tensor of at
    least 4 bytes. Launched on `stream`; the caller times it."""
    if nbytes > buf.numel() * buf.element_size():
        raise ValueError(f"read_stream: {nbytes} bytes exceed the buffer")
    _check("moe_read_stream", _lib.moe_read_stream(_ptr(buf), nbytes, _ptr(sink), grid, _stream(stream)))
