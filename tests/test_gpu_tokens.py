"""GPU multi-token decode FFN (a small batch of tokens, every selected expert resident)
vs the oracle: y[t] = sum_j w[t][j] * expert(slot[t][j])(x[t]) (SwiGLU expert, Section I
weighted combine), each selected slab read once for all the tokens that chose it."""
import os

import numpy as np
import pytest

import oracle
import synth
from _gpu_util import assert_close, say, torch_cuda

pytestmark = pytest.mark.gpu


def _pool(torch, slabs_np, d, f):
    import paper_2512_16473_amd as moe
    stride = moe.slab_bytes(d, f)
    pool = torch.zeros(len(slabs_np) * stride, dtype=torch.uint8)
    for i, s in enumerate(slabs_np):
        pool[i * stride: i * stride + s.nbytes] = torch.from_numpy(s.view(np.uint8))
    return pool.cuda()


def _run(torch, X, pool, nslots, slots, w, d, f):
    import paper_2512_16473_amd as moe
    T, k = slots.shape
    ws = torch.empty(moe.ffn_tokens_workspace_bytes(T, k, d, f), dtype=torch.uint8, device="cuda")
    y = torch.full((T, d), float("nan"), dtype=torch.float32, device="cuda")
    moe.expert_ffn_tokens(torch.from_numpy(X).cuda(), pool, nslots, torch.from_numpy(slots).cuda(),
                          torch.from_numpy(w).cuda(), d, f, y, ws)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def _expect(X, slabs, slots, w, d, f, nslots):
    out = []
    for t in range(X.shape[0]):
        ys, ws = [], []
        for j in range(slots.shape[1]):
            s = int(slots[t, j])
            if 0 <= s < nslots:
                ys.append(oracle.expert(X[t], slabs[s], d, f))
                ws.append(w[t, j])
        out.append(oracle.combine(np.stack(ys), np.array(ws, np.float32)) if ys else np.zeros(d, np.float32))
    return out


def _selection(rng, T, k, nslots):
    return np.stack([rng.choice(nslots, k, replace=False) for _ in range(T)]).astype(np.int32)


@pytest.mark.parametrize("d,f,nslots,T,k", [
    (256, 512, 4, 3, 2),        # tiny shapes, overlapping selections
    (264, 520, 5, 5, 2),        # ragged d and f
    (1024, 4104, 4, 4, 2),      # two down segments, ragged tail
    (512, 1024, 8, 8, 4),       # eight tokens, four ranks
    (4096, 1792, 6, 8, 2),      # Mixtral-wide rows, T*d at the staging limit (128 KiB of x)
    (3584, 2560, 12, 6, 8),     # fine-grained expert shape, top-8
    (8192, 1032, 3, 4, 3),      # d = MOE_MAX_D
])
def test_tokens_parity(d, f, nslots, T, k):
    torch = torch_cuda()
    oracle.set_threads(min(16, os.cpu_count() or 1))
    say("ffn_tokens", d, f, nslots, T, k)
    rng = np.random.default_rng(d * 31 + f + T)
    slabs = [synth.expert_slab(900 + 17 * i + d, d, f, None) for i in range(nslots)]
    pool = _pool(torch, slabs, d, f)
    X = rng.standard_normal((T, d)).astype(np.float32)
    slots = _selection(rng, T, k, nslots)
    w = rng.random((T, k)).astype(np.float32)
    y = _run(torch, X, pool, nslots, slots, w, d, f)
    for t, e in enumerate(_expect(X, slabs, slots, w, d, f, nslots)):
        assert_close(y[t], e, f"tokens d={d} f={f} t={t} slots={list(slots[t])}")


def test_tokens_invalid_slots_and_single_token():
    """Slots outside [0, n_slots) are skipped (a token with none gets zeros), and one token
    gives what the one-token hit path gives."""
    torch = torch_cuda()
    import paper_2512_16473_amd as moe
    say("ffn_tokens invalid slots / T = 1")
    d, f, nslots = 256, 512, 4
    slabs = [synth.expert_slab(40 + i, d, f, None) for i in range(nslots)]
    pool = _pool(torch, slabs, d, f)
    rng = np.random.default_rng(5)
    X = rng.standard_normal((3, d)).astype(np.float32)
    slots = np.array([[1, -1], [nslots, -5], [3, 1]], np.int32)
    w = rng.random((3, 2)).astype(np.float32)
    y = _run(torch, X, pool, nslots, slots, w, d, f)
    assert np.all(y[1] == 0.0)
    for t in (0, 2):
        assert_close(y[t], _expect(X[t:t + 1], slabs, slots[t:t + 1], w[t:t + 1], d, f, nslots)[0], f"t={t}")
    # T = 1 against the one-token path (the same expert FFN, the same fixed-order sums)
    s1 = np.array([[2, 0]], np.int32)
    w1 = np.array([[0.7, 0.3]], np.float32)
    y1 = _run(torch, X[:1], pool, nslots, s1, w1, d, f)
    ws = torch.empty(moe.ffn_workspace_bytes(2, d, f), dtype=torch.uint8, device="cuda")
    yh = torch.empty(d, dtype=torch.float32, device="cuda")
    moe.expert_ffn_hits(torch.from_numpy(X[0]).cuda(), pool, nslots, torch.from_numpy(s1[0]).cuda(),
                        torch.from_numpy(w1[0]).cuda(), d, f, yh, ws)
    torch.cuda.synchronize()
    assert_close(y1[0], yh.cpu().numpy(), "T=1 vs hit path")


@pytest.mark.parametrize("T,k,nslots,pattern", [
    (2, 4, 3, "dup"),        # a job with 6 pairs for T = 2: h staged in three groups of T
    (8, 16, 2, "one"),       # 128 pairs of one slot: results past the 64th pair, eight groups
])
def test_tokens_repeated_slots(T, k, nslots, pattern):
    """A slot listed several times (also by one token) contributes once per listing, each
    with its own weight: the job then has more (token, rank) pairs than tokens."""
    torch = torch_cuda()
    say("ffn_tokens repeated slots", T, k, nslots, pattern)
    d, f = 256, 520
    slabs = [synth.expert_slab(70 + i, d, f, None) for i in range(nslots)]
    pool = _pool(torch, slabs, d, f)
    rng = np.random.default_rng(T * 100 + k)
    X = rng.standard_normal((T, d)).astype(np.float32)
    if pattern == "dup":
        slots = np.array([[1, 1, 1, 1], [1, 1, 2, 2]], np.int32)
    else:
        slots = np.zeros((T, k), np.int32)
    w = rng.random((T, k)).astype(np.float32)
    y = _run(torch, X, pool, nslots, slots, w, d, f)
    for t, e in enumerate(_expect(X, slabs, slots, w, d, f, nslots)):
        assert_close(y[t], e, f"repeated slots t={t} slots={list(slots[t])}")


def test_tokens_mixtral_shape_sampled():
    """Full Mixtral expert shape (d 4096, f 14336), 4 tokens top-2 over 4 resident slabs."""
    torch = torch_cuda()
    oracle.set_threads(min(16, os.cpu_count() or 1))
    say("ffn_tokens mixtral shape")
    wl = synth.WORKLOADS["mixtral"]
    d, f, nslots, T, k = wl.d, wl.f, 4, 4, 2
    slabs = [synth.expert_slab(synth.seed_for(0, "mixtral", "expert", 0, e), d, f, wl.w_std) for e in range(nslots)]
    pool = _pool(torch, slabs, d, f)
    X = synth.ar1_states(synth.seed_for(0, "mixtral", "states", 0), T, d)
    slots = np.array([[0, 1], [1, 2], [0, 1], [3, 0]], np.int32)
    w = np.array([[0.6, 0.4], [0.55, 0.45], [0.7, 0.3], [0.5, 0.5]], np.float32)
    y = _run(torch, X, pool, nslots, slots, w, d, f)
    for t, e in enumerate(_expect(X, slabs, slots, w, d, f, nslots)):
        assert_close(y[t], e, f"mixtral t={t}")
