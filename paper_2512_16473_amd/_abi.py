"""ctypes declarations of the C ABI in include/moe.h (argument marshalling only)."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmoe.so")

c_int, c_size_t, c_void_p, c_float, c_double = (ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p,
                                                ctypes.c_float, ctypes.c_double)
c_i32p = ctypes.POINTER(ctypes.c_int32)
c_u8p = ctypes.POINTER(ctypes.c_uint8)
c_f32p = ctypes.POINTER(ctypes.c_float)
c_char_p = ctypes.c_char_p

MOE_OK, MOE_EINVAL, MOE_EHIP, MOE_ESTATE, MOE_ENOMEM = 0, -1, -2, -3, -4
MAX_EXPERTS, MAX_TOPK, MAX_D, MAX_TOKENS = 256, 16, 8192, 8
HOST_DOT = {"auto": 0, "fp32": 1, "bf16": 2}


class LayerDesc(ctypes.Structure):
    _fields_ = [
        ("d", c_int), ("f", c_int), ("n", c_int), ("k", c_int), ("ways", c_int),
        ("n_layers", c_int), ("f_shared", c_int),
        ("w_router", c_void_p), ("slot_pool", c_void_p), ("shared_pool", c_void_p),
        ("host_slabs", ctypes.POINTER(c_void_p)),
        ("cache", c_void_p), ("pool", c_void_p),
    ]


class RuntimeStats(ctypes.Structure):
    _fields_ = [
        ("layer_calls", ctypes.c_int64), ("expert_hits", ctypes.c_int64),
        ("expert_misses", ctypes.c_int64), ("fills", ctypes.c_int64),
        ("host_ffn_ms", c_double), ("route_wait_ms", c_double),
        ("gate_up_launches", ctypes.c_int64), ("gate_up_ms", c_double), ("gate_up_bytes", c_double),
        ("down_launches", ctypes.c_int64), ("down_ms", c_double), ("down_bytes", c_double),
        ("fills_skipped", ctypes.c_int64), ("inflight_misses", ctypes.c_int64),
    ]


class PrefillDesc(ctypes.Structure):
    _fields_ = [("d", c_int), ("f", c_int), ("n", c_int), ("k", c_int),
                ("w_router", c_void_p), ("expert_pool", c_void_p)]


# (name, restype, argtypes) for every function the header declares.
SIGNATURES = [
    ("moe_last_error", c_char_p, []),
    ("moe_version", c_int, []),
    ("moe_slab_bytes", c_size_t, [c_int, c_int]),
    ("moe_router_topk", c_int, [c_void_p, c_void_p, c_int, c_int, c_int, c_int, c_void_p, c_void_p, c_void_p]),
    ("moe_cache_create", c_int, [c_int, c_int, c_int, c_int, ctypes.POINTER(c_void_p)]),
    ("moe_cache_create_policy", c_int, [c_int, c_int, c_int, c_int, c_int, c_i32p, ctypes.POINTER(c_void_p)]),
    ("moe_cache_geometry", c_int, [c_size_t, c_size_t, c_int, c_int, ctypes.POINTER(c_int), ctypes.POINTER(c_int)]),
    ("moe_cache_destroy", None, [c_void_p]),
    ("moe_cache_reset", c_int, [c_void_p]),
    ("moe_cache_lookup", c_int, [c_void_p, c_int, c_i32p, c_int, c_i32p, c_u8p]),
    ("moe_cache_update", c_int, [c_void_p, c_int, c_i32p, c_int, c_i32p, c_i32p]),
    ("moe_cache_update_masked", c_int, [c_void_p, c_int, c_i32p, c_int, c_u8p, c_i32p, c_i32p]),
    ("moe_cache_slotmap", c_int, [c_void_p, c_int, c_i32p]),
    ("moe_cache_state_bytes", c_size_t, [c_void_p]),
    ("moe_cache_save", c_int, [c_void_p, c_void_p, c_size_t]),
    ("moe_cache_restore", c_int, [c_void_p, c_void_p, c_size_t]),
    ("moe_ffn_workspace_bytes", c_size_t, [c_int, c_int, c_int]),
    ("moe_expert_ffn_hits", c_int, [c_void_p, c_void_p, c_int, c_void_p, c_void_p, c_int, c_int, c_int,
                                    c_void_p, c_void_p, c_size_t, c_void_p]),
    ("moe_ffn_noalloc_max_bytes", c_size_t, []),
    ("moe_expert_ffn_hits_noalloc", c_int, [c_void_p, c_void_p, c_int, c_void_p, c_void_p, c_int, c_int, c_int,
                                            c_void_p, c_void_p]),
    ("moe_combine", c_int, [c_void_p, c_void_p, c_void_p, c_int, c_void_p, c_void_p]),
    ("moe_ffn_tokens_workspace_bytes", c_size_t, [c_int, c_int, c_int, c_int]),
    ("moe_expert_ffn_tokens", c_int, [c_void_p, c_void_p, c_int, c_void_p, c_void_p, c_int, c_int, c_int, c_int,
                                      c_void_p, c_void_p, c_size_t, c_void_p]),
    ("moe_host_alloc", c_int, [c_size_t, ctypes.POINTER(c_void_p)]),
    ("moe_host_free", c_int, [c_void_p]),
    ("moe_host_pool_create", c_int, [c_int, ctypes.POINTER(c_void_p)]),
    ("moe_host_pool_destroy", None, [c_void_p]),
    ("moe_host_pool_threads", c_int, [c_void_p]),
    ("moe_host_pool_set_dot", c_int, [c_void_p, c_int]),
    ("moe_host_pool_get_dot", c_int, [c_void_p]),
    ("moe_host_expert_ffn", c_int, [c_void_p, c_f32p, ctypes.POINTER(c_void_p), c_f32p, c_int, c_int, c_int,
                                    c_f32p]),
    ("moe_runtime_create", c_int, [ctypes.POINTER(LayerDesc), ctypes.POINTER(c_void_p)]),
    ("moe_runtime_destroy", None, [c_void_p]),
    ("moe_layer_forward", c_int, [c_void_p, c_int, c_void_p, c_void_p, c_i32p, c_f32p, c_u8p,
                                  c_void_p, c_void_p, c_void_p]),
    ("moe_decode_step", c_int, [c_void_p, c_void_p, c_void_p, c_i32p, c_f32p, c_u8p,
                                c_void_p, c_void_p, c_void_p]),
    ("moe_runtime_sync", c_int, [c_void_p]),
    ("moe_runtime_device_slotmap", c_int, [c_void_p, c_int, c_i32p]),
    ("moe_runtime_set_fill_limit", c_int, [c_void_p, c_int]),
    ("moe_runtime_set_nonblocking", c_int, [c_void_p, c_int]),
    ("moe_runtime_set_timing", c_int, [c_void_p, c_int]),
    ("moe_runtime_get_stats", c_int, [c_void_p, ctypes.POINTER(RuntimeStats)]),
    ("moe_runtime_reset_stats", c_int, [c_void_p]),
    ("moe_prefill_workspace_bytes", c_size_t, [ctypes.POINTER(PrefillDesc), c_int]),
    ("moe_prefill_forward", c_int, [ctypes.POINTER(PrefillDesc), c_void_p, c_int, c_void_p, c_void_p, c_void_p,
                                    c_void_p, c_size_t, c_void_p]),
    ("moe_read_stream", c_int, [c_void_p, c_size_t, c_void_p, c_int, c_void_p]),
]


def load(path: str = LIB_PATH):
    # torch ships its own HIP runtime (same soname as the system one). Loading torch
    # first makes libmoe.so bind to that runtime, so the process has one HIP runtime
    # and torch's streams and device memory are valid handles for the library.
    import torch  # noqa: F401
    if not os.path.exists(path):
        raise ImportError(
            f"{path} is missing: build the HIP library first "
            "(python paper_2512_16473_amd/build.py or __graft_entry__.build())")
    lib = ctypes.CDLL(path)
    for name, res, args in SIGNATURES:
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib
