"""Prefill path (all experts resident, T tokens, grouped MFMA GEMMs) vs the oracle.

The oracle evaluates each token through the same layer definition as decode (router,
chosen SwiGLU experts, combine). The GPU rounds the hidden states and the SwiGLU
activations to bf16 for the matrix cores (fp32 accumulation), so its error is that of
bf16 activations: ~1e-3 x RMS per element, within the 2e-2 x RMS bound.
"""
import os

import numpy as np
import pytest

import oracle
import synth
from _gpu_util import TOL, rel_err, router_parity, say, torch_cuda

pytestmark = pytest.mark.gpu


def _run(torch, X, wr, pool, d, f, n, k):
    import paper_2512_16473_amd as moe
    T = X.shape[0]
    ws = torch.empty(max(256, moe.prefill_workspace_bytes(d, f, n, k, T)), dtype=torch.uint8, device="cuda")
    Xd = torch.from_numpy(X).cuda()
    out = torch.full((T, d), float("nan"), device="cuda")
    idx = torch.full((T, k), -1, dtype=torch.int32, device="cuda")
    w = torch.zeros((T, k), device="cuda")
    moe.prefill_forward(Xd, torch.from_numpy(wr).cuda(), pool, d, f, n, k, out, ws, idx=idx, w=w)
    torch.cuda.synchronize()
    return out.cpu().numpy(), idx.cpu().numpy(), w.cpu().numpy()


def _bf16_activation_ref(x, slabs, idx, w, d, f):
    """Test-side reference: x and h rounded to bf16 (RNE), everything else fp64."""
    xb = synth.bf16_to_f32(synth.bf16_bits(x)).astype(np.float64)
    y = np.zeros(d)
    for e, we in zip(idx, w):
        W = synth.bf16_to_f32(slabs[e]).astype(np.float64)
        w1, w3, w2 = W[: f * d].reshape(f, d), W[f * d: 2 * f * d].reshape(f, d), W[2 * f * d:].reshape(d, f)
        g, u = w1 @ xb, w3 @ xb
        h = (g / (1.0 + np.exp(-g)) * u).astype(np.float32)
        hb = synth.bf16_to_f32(synth.bf16_bits(h)).astype(np.float64)
        y += float(we) * (w2 @ hb)
    return y


def _pool_np(torch, slabs, d, f):
    import paper_2512_16473_amd as moe
    stride = moe.slab_bytes(d, f)
    pool = torch.zeros(len(slabs) * stride, dtype=torch.uint8)
    for i, s in enumerate(slabs):
        pool[i * stride: i * stride + s.nbytes] = torch.from_numpy(s.view(np.uint8))
    return pool.cuda()


# (256, 512, 4, 2, 700): 1400 pairs (two chunks of the grouping sort) and ~350 tokens per
# expert (two 192-token tiles); (384, 640, ...): d not a multiple of 256 (128-row down tiles)
# and f not a multiple of 256 (two K splits). With one expert per XCD and 32 gate/up work
# groups resident per XCD, the gate/up tiles of the last partial round are split over K:
# (512, 1024, 8, 2, 300) 8 tiles per XCD in 4 parts each; (256, 512, 4, 2, 700) two M tiles
# per expert, 4 parts; (256, 5120, 8, 2, 256) a full round of 32 tiles, then 8 tiles in 4
# parts; (256, 1024, 16, 2, 520) two experts per XCD, 16 tiles in 2 parts.
@pytest.mark.parametrize("d,f,n,k,T", [(256, 512, 4, 2, 64), (256, 512, 4, 2, 37), (512, 1024, 8, 2, 300),
                                       (384, 640, 16, 4, 130), (256, 256, 8, 1, 1), (256, 512, 64, 8, 48),
                                       (256, 512, 4, 2, 700), (256, 5120, 8, 2, 256), (256, 1024, 16, 2, 520)])
def test_prefill_small(d, f, n, k, T):
    torch = torch_cuda()
    say("prefill", d, f, n, k, T)
    wr = synth.router_weights(synth.seed_for(3, "prefill", "router", d, n), n, d)
    slabs = [synth.expert_slab(synth.seed_for(3, "prefill", "expert", d, e), d, f, None) for e in range(n)]
    X = synth.iid_states(synth.seed_for(3, "prefill", "prompt", d, T), T, d)
    pool = _pool_np(torch, slabs, d, f)
    out, idx, w = _run(torch, X, wr, pool, d, f, n, k)
    worst = worst_b = 0.0
    for t in range(T):
        oidx, ow = router_parity(idx[t], w[t], X[t], wr, k)
        _, _, ref, _ = oracle.moe_token(X[t], wr, slabs, k, f, forced_set=oidx)
        r = rel_err(out[t], ref)
        assert r <= TOL, (t, r)
        worst = max(worst, r)
        # The same layer with the two bf16 roundings the matrix cores need (x and h),
        # fp64 otherwise: what is left is accumulation order only.
        rb = rel_err(out[t], _bf16_activation_ref(X[t], slabs, oidx, ow, d, f))
        assert rb <= 2e-3, (t, rb)
        worst_b = max(worst_b, rb)
    say("  worst max|err|/RMS vs oracle", worst, "vs bf16-activation reference", worst_b)


@pytest.mark.parametrize("shape", ["mixtral", "phi", "fine"])
def test_prefill_full_shape(shape):
    """Configs: one 512-token prompt through a full-size layer with every expert resident,
    in the launch configuration the benchmark times, every token's routing and output
    compared with the oracle.
    * mixtral (the benchmark's prefill line): one M tile per expert, one expert per XCD,
      the gate/up tail split in 2 K parts;
    * phi (d 4096, f 6400, 16 experts top-2): two experts per XCD, 100 gate/up tiles per
      XCD, the last 4 split in 8 K parts;
    * fine (d 3584, f 2560, 64 experts top-8, routed experts only): d not a multiple of
      256 (128-row down tiles) and 64 (token, expert) pairs per expert on average."""
    torch = torch_cuda()
    import paper_2512_16473_amd as moe
    if shape == "mixtral":
        wl = synth.WORKLOADS["prefill"]
        tag = "prefill"
    else:
        wl = synth.WORKLOADS[shape]
        tag = "prefill-" + shape
    d, f, n, k, T = wl.d, wl.f, wl.n, wl.k, 512
    say("prefill", shape, d, f, n, k, T)
    stride = moe.slab_bytes(d, f)
    pool = torch.empty(n * stride, dtype=torch.uint8, device="cuda")
    host = []
    for e in range(n):
        t = pool[e * stride: e * stride + 3 * d * f * 2].view(torch.bfloat16)
        synth.expert_slab_torch(synth.seed_for(0, tag, "expert", 0, e), d, f, wl.w_std, out=t)
        host.append(t.view(torch.uint8).cpu().numpy().view(np.uint16))
    wr = synth.router_weights(synth.seed_for(0, tag, "router", 0), n, d)
    X = synth.iid_states(synth.seed_for(0, tag, "prompt"), T, d)
    out, idx, w = _run(torch, X, wr, pool, d, f, n, k)
    oracle.set_threads(min(16, os.cpu_count() or 1))
    sets = []
    for t in range(T):
        oidx, ow = router_parity(idx[t], w[t], X[t], wr, k)
        sets.append(oidx)
    counts = np.bincount(idx.ravel(), minlength=n)
    say("  tokens per expert", counts.tolist())
    worst = 0.0
    for t in range(T):
        _, _, ref, _ = oracle.moe_token(X[t], wr, host, k, f, forced_set=sets[t])
        r = rel_err(out[t], ref)
        assert r <= TOL, (t, r)
        worst = max(worst, r)
        if t % 128 == 127:
            say("  tokens compared", t + 1, "worst max|err|/RMS so far", worst)
    say("  worst max|err|/RMS", worst)


def test_prefill_empty_and_invalid():
    torch = torch_cuda()
    import paper_2512_16473_amd as moe
    d, f, n, k = 256, 512, 4, 2
    pool = torch.zeros(n * moe.slab_bytes(d, f), dtype=torch.uint8, device="cuda")
    wr = torch.zeros((n, d), device="cuda")
    X = torch.zeros((0, d), device="cuda")
    out = torch.zeros((1, d), device="cuda")
    ws = torch.empty(256, dtype=torch.uint8, device="cuda")
    moe.prefill_forward(X, wr, pool, d, f, n, k, out, ws)        # T = 0: no-op
    with pytest.raises(moe.MoeError):
        moe.prefill_forward(torch.zeros((4, 200), device="cuda"), torch.zeros((n, 200), device="cuda"), pool,
                            200, f, n, k, out, ws)                # d not a multiple of 128
