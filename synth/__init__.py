"""Seeded synthetic inputs for the MoE expert-stage workloads.

This module only draws numbers: router weights, expert weight slabs, hidden-state
streams and the shapes of the five workloads. It holds none of the method's
arithmetic (no routing, no expert FFN, no cache policy), so both the CPU oracle
and the GPU path can take their inputs from it without sharing any computation.

Paper models (Table II): Mixtral-8x7B has 32 layers of 8 experts with top-2
routing; Phi-3.5-MoE has 32 layers of 16 experts with top-2 routing. Expert sizes
(340 MB / 152 MB) imply three d x f matrices of 2-byte weights per expert, i.e. a
SwiGLU expert. The trained weights are not available; the weights here are
Gaussian with the stated standard deviations.

Hidden states follow an AR(1) process per layer,
x_0 ~ N(0, I), x_t = rho * x_{t-1} + sigma * eps_t, with rho = 0.9 and
sigma = 0.436 (so the marginal stays close to N(0, 1) and consecutive tokens are
correlated, a stand-in for the consecutive-tokens expert-reuse pattern of
Section II-B).

Expert slab layout (one contiguous bf16 block per expert, row-major [out, in]):
    W1 [f, d] | W3 [f, d] | W2 [d, f]
bf16 values are carried as uint16 bit patterns in numpy.
"""
from __future__ import annotations

import dataclasses
import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "seed_for", "bf16_bits", "bf16_to_f32",
    "router_weights", "expert_slab", "ar1_states", "iid_states",
    "expert_slab_torch", "router_weights_torch", "slab_elems", "slab_bytes",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    d: int              # d_model
    f: int              # d_ffn of a routed expert
    n: int              # routed experts per layer
    k: int              # experts selected per token
    L: int              # MoE layers
    T: int              # decode steps (or prompt tokens for prefill)
    ways: int           # cache slots per layer (M); == n means every expert resident
    f_shared: int = 0   # d_ffn of the always-active shared expert (0 = none)
    w_std: float | None = 0.02   # None: std = 1/sqrt(fan_in) per matrix
    prefill: bool = False
    desc: str = ""


WORKLOADS = {
    "tiny": Workload(
        "tiny", d=256, f=512, n=4, k=2, L=1, T=64, ways=2, w_std=None,
        desc="tiny MoE layer d256 f512 4e top-2, 64 AR(1) decode steps, 2-slot LRU cache"),
    "mixtral": Workload(
        "mixtral", d=4096, f=14336, n=8, k=2, L=32, T=256, ways=4,
        desc="Mixtral-8x7B-shaped decode d4096 f14336 8e top-2 32 layers, 4 of 8 experts cached per layer, LRU"),
    "phi": Workload(
        "phi", d=4096, f=6400, n=16, k=2, L=32, T=256, ways=6,
        desc="Phi-3.5-MoE-shaped decode d4096 f6400 16e top-2 32 layers, 6 of 16 experts cached per layer, LRU"),
    "prefill": Workload(
        "prefill", d=4096, f=14336, n=8, k=2, L=32, T=512, ways=8, prefill=True,
        desc="Mixtral-8x7B-shaped prefill, one 512-token prompt, all 8 experts resident"),
    "fine": Workload(
        "fine", d=3584, f=2560, n=64, k=8, L=28, T=256, ways=24, f_shared=20480,
        desc="fine-grained MoE decode d3584 f2560 64e top-8 + shared expert f20480, 28 layers, 24 of 64 cached"),
}

# Tensor kinds used when deriving per-tensor seeds.
_KIND = {"router": 1, "expert": 2, "shared": 3, "states": 4, "prompt": 5, "static-content": 6, "subsets": 7}
_WL_ID = {name: i + 1 for i, name in enumerate(WORKLOADS)}


def seed_for(seed: int, workload: str, kind: str, layer: int = 0, expert: int = 0) -> int:
    """A 63-bit seed for one tensor, derived from (seed, workload, kind, layer, expert)."""
    ss = np.random.SeedSequence([int(seed), _WL_ID.get(workload, 0), _KIND[kind],
                                 int(layer), int(expert)])
    return int(ss.generate_state(1, np.uint64)[0] & np.uint64((1 << 63) - 1))


def slab_elems(d: int, f: int) -> int:
    return 3 * d * f


def slab_bytes(d: int, f: int) -> int:
    return 2 * slab_elems(d, f)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> fp32 (exact widening)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _std_pair(wl_std, d, f):
    if wl_std is None:
        return 1.0 / np.sqrt(d), 1.0 / np.sqrt(f)   # W1/W3 fan-in d, W2 fan-in f
    return float(wl_std), float(wl_std)


def router_weights(seed: int, n: int, d: int) -> np.ndarray:
    """fp32 [n, d] router weights ~ N(0, 1/d)."""
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((n, d), dtype=np.float32) * np.float32(1.0 / np.sqrt(d))).astype(np.float32)


def expert_slab(seed: int, d: int, f: int, w_std: float | None = 0.02) -> np.ndarray:
    """One expert's bf16 slab (uint16 [3*d*f]): W1 [f,d] | W3 [f,d] | W2 [d,f]."""
    rng = np.random.default_rng(seed)
    s_in, s_out = _std_pair(w_std, d, f)
    w1 = rng.standard_normal(f * d, dtype=np.float32) * np.float32(s_in)
    w3 = rng.standard_normal(f * d, dtype=np.float32) * np.float32(s_in)
    w2 = rng.standard_normal(d * f, dtype=np.float32) * np.float32(s_out)
    return bf16_bits(np.concatenate([w1, w3, w2]))


def ar1_states(seed: int, T: int, d: int, rho: float = 0.9, sigma: float = 0.436) -> np.ndarray:
    """fp32 [T, d] hidden states: x_0 ~ N(0,I), x_t = rho x_{t-1} + sigma eps_t."""
    rng = np.random.default_rng(seed)
    eps = rng.standard_normal((T, d))
    x = np.empty((T, d), dtype=np.float64)
    x[0] = eps[0]
    for t in range(1, T):
        x[t] = rho * x[t - 1] + sigma * eps[t]
    return x.astype(np.float32)


def iid_states(seed: int, T: int, d: int) -> np.ndarray:
    """fp32 [T, d] i.i.d. N(0,1) hidden states (prefill prompt)."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal((T, d), dtype=np.float32)


# ---- torch generators for the large shapes (drawn directly on the device) ----

def expert_slab_torch(seed: int, d: int, f: int, w_std: float | None = 0.02, device="cuda", out=None):
    """One expert's slab as a torch bf16 tensor [3*d*f] drawn on `device`.

    Values come from torch's generator for that device; the CPU oracle receives
    a host copy of the very same tensor, so the two sides see identical weights.
    """
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    s_in, s_out = _std_pair(w_std, d, f)
    if out is None:
        out = torch.empty(3 * d * f, dtype=torch.bfloat16, device=device)
    fd = f * d
    tmp = torch.empty(fd, dtype=torch.float32, device=device)
    for part, s in ((0, s_in), (1, s_in), (2, s_out)):
        tmp.normal_(0.0, s, generator=g)
        out[part * fd:(part + 1) * fd].copy_(tmp)
    return out


def router_weights_torch(seed: int, n: int, d: int, device="cuda"):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    w = torch.empty((n, d), dtype=torch.float32, device=device)
    w.normal_(0.0, 1.0 / float(np.sqrt(d)), generator=g)
    return w
