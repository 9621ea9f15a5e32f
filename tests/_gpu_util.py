"""Shared helpers of the GPU parity tests: seeded inputs on the device and in
pinned host memory, and the comparisons against the oracle."""
from __future__ import annotations

import sys

import numpy as np

import oracle
import synth

TOL = 2e-2          # max |gpu - oracle| <= TOL * RMS(oracle) per output vector
TRIPWIRE = 1e-3     # fp32 accumulation lands near 1e-6; a layout bug lands near 1
NEAR_TIE = 1e-6     # relative logit margin under which either expert set is accepted


def say(*a):
    print("[gpu-test]", *a, file=sys.stderr, flush=True)


def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    return torch


def rel_err(got, ref):
    ref = np.asarray(ref, dtype=np.float64)
    got = np.asarray(got, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref ** 2)))
    err = float(np.max(np.abs(got - ref))) if ref.size else 0.0
    return err / rms if rms > 0 else err


def assert_close(got, ref, what=""):
    r = rel_err(got, ref)
    assert r <= TOL, f"{what}: max|err|/RMS = {r:.3e} > {TOL}"
    assert r <= TRIPWIRE, f"{what}: max|err|/RMS = {r:.3e} above the fp32-accumulation tripwire {TRIPWIRE}"
    return r


def make_slabs_host(torch, L, n, d, f, w_std, seed, wl_name, kind="expert"):
    """L*n expert slabs drawn on the GPU, copied into one pinned host buffer.

    Returns (PinnedBuffer, stride, list of L*n numpy uint16 views).
    """
    import paper_2512_16473_amd as moe
    stride = moe.slab_bytes(d, f)
    buf = moe.PinnedBuffer(L * n * stride)
    host = torch.from_numpy(buf.array)
    tmp = torch.empty(3 * d * f, dtype=torch.bfloat16, device="cuda")
    views = []
    for l in range(L):
        for e in range(n):
            s = synth.seed_for(seed, wl_name, kind, l, e)
            synth.expert_slab_torch(s, d, f, w_std, device="cuda", out=tmp)
            off = (l * n + e) * stride
            host[off: off + 3 * d * f * 2].copy_(tmp.view(torch.uint8))
            views.append(buf.array[off: off + 3 * d * f * 2].view(np.uint16))
    torch.cuda.synchronize()
    return buf, stride, views


def router_parity(gpu_idx, gpu_w, x, wr, k):
    """Routing check with the near-tie protocol. Returns the oracle (idx, w) for the
    expert set the GPU chose (identical to the oracle's own when no near-tie)."""
    idx, w, gap, logits = oracle.router(x, wr, k)
    if list(gpu_idx) != list(idx):
        scale = max(1.0, float(np.max(np.abs(logits))))
        assert set(gpu_idx) != set(idx) and gap < NEAR_TIE * scale, \
            f"routing differs without a near-tie: gpu={list(gpu_idx)} oracle={list(idx)} gap={gap}"
        idx, w = oracle.router_forced(x, wr, k, gpu_idx)
        assert list(idx) == list(gpu_idx)
    ulp = np.spacing(np.maximum(np.abs(w), np.float32(1e-30)))
    assert np.all(np.abs(np.asarray(gpu_w, np.float64) - w) <= 4 * ulp), (gpu_w, w)
    return idx, w
