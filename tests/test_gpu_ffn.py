"""GPU cache-hit expert FFN and combine vs the oracle (SwiGLU expert, Table II size
reading; Section I weighted combine)."""
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


def _ffn(torch, x, pool, n_slots, slots, w, d, f, k_ws=None):
    import paper_2512_16473_amd as moe
    ws = torch.empty(moe.ffn_workspace_bytes(len(slots) if k_ws is None else k_ws, d, f), dtype=torch.uint8,
                     device="cuda")
    y = torch.full((d,), float("nan"), dtype=torch.float32, device="cuda")
    moe.expert_ffn_hits(torch.from_numpy(x).cuda(), pool, n_slots,
                        torch.tensor(slots, dtype=torch.int32, device="cuda"),
                        torch.tensor(w, dtype=torch.float32, device="cuda"), d, f, y, ws)
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("d,f,nslots,slots", [
    (256, 512, 4, [2, 0]),            # tiny layer: two hits
    (256, 512, 4, [3]),               # one hit
    (264, 520, 3, [1, 2, 0]),         # ragged: d and f not multiples of 512 / the segment
    (1024, 4104, 2, [1, 0]),          # several down segments with a ragged tail
    (512, 1024, 8, [7, 0, 3, 5, 1, 2, 6, 4]),   # eight jobs
    (4096, 256, 2, [0, 1]),           # short reduction, wide rows
    (8192, 1032, 16, list(range(15, -1, -1))),   # the ABI maxima: d = MOE_MAX_D, 16 jobs
])
def test_hits_parity(d, f, nslots, slots):
    torch = torch_cuda()
    say("ffn_hits", d, f, nslots, slots)
    slabs = [synth.expert_slab(700 + 13 * i + d, d, f, None) for i in range(nslots)]
    pool = _pool(torch, slabs, d, f)
    rng = np.random.default_rng(d + f)
    x = rng.standard_normal(d).astype(np.float32)
    w = rng.random(len(slots)).astype(np.float32)
    y = _ffn(torch, x, pool, nslots, slots, w, d, f)
    ys = np.stack([oracle.expert(x, slabs[s], d, f) for s in slots])
    assert_close(y, oracle.combine(ys, w), f"ffn d={d} f={f} slots={slots}")


def test_hits_skip_invalid_slots_and_empty():
    torch = torch_cuda()
    say("ffn_hits skip")
    d, f = 256, 512
    slabs = [synth.expert_slab(900 + i, d, f, None) for i in range(3)]
    pool = _pool(torch, slabs, d, f)
    x = np.random.default_rng(3).standard_normal(d).astype(np.float32)
    y = _ffn(torch, x, pool, 3, [-1, 2, 3, 99], [0.4, 0.3, 0.2, 0.1], d, f)   # only slot 2 is valid
    assert_close(y, np.float32(0.3) * oracle.expert(x, slabs[2], d, f), "skip")
    y0 = _ffn(torch, x, pool, 3, [], [], d, f, k_ws=1)
    assert np.all(y0 == 0)


@pytest.mark.parametrize("name", ["mixtral", "phi", "fine"])
def test_hits_parity_full_shape(name):
    """Full per-expert shapes of the decode workloads, in the launch configuration
    the benchmark uses; every output compared."""
    torch = torch_cuda()
    import paper_2512_16473_amd as moe
    wl = synth.WORKLOADS[name]
    d, f, k = wl.d, wl.f, wl.k
    say("ffn_hits full", name, d, f, k)
    stride = moe.slab_bytes(d, f)
    nslots = k + 1
    pool = torch.empty(nslots * stride, dtype=torch.uint8, device="cuda")
    host = []
    for s in range(nslots):
        t = pool[s * stride: s * stride + 3 * d * f * 2].view(torch.bfloat16)
        synth.expert_slab_torch(synth.seed_for(5, name, "expert", 0, s), d, f, wl.w_std, out=t)
        host.append(t.view(torch.uint8).cpu().numpy().view(np.uint16))
    x = synth.ar1_states(synth.seed_for(5, name, "states"), 1, d)[0]
    slots = list(range(nslots - 1, 0, -1))[:k]
    w = np.random.default_rng(1).random(k).astype(np.float32)
    w /= w.sum()
    y = _ffn(torch, x, pool, nslots, slots, w, d, f)
    oracle.set_threads(min(16, os.cpu_count() or 1))
    ys = np.stack([oracle.expert(x, host[s], d, f) for s in slots])
    r = assert_close(y, oracle.combine(ys, w), name)
    say("  max|err|/RMS", r)


def test_combine():
    """moe_combine against the oracle's combine (Section I: the layer output is the
    gate-weighted sum of the selected experts' outputs, a shared expert at weight 1).
    The GPU hit part and the host miss part each arrive already weighted; their sum
    plus the shared expert must equal the oracle's combine over all selected experts."""
    torch = torch_cuda()
    import paper_2512_16473_amd as moe
    say("combine")
    d, f, n, k = 264, 520, 6, 4
    slabs = [synth.expert_slab(1200 + e, d, f, None) for e in range(n)]
    shared = synth.expert_slab(1299, d, 2 * f, None)
    rng = np.random.default_rng(11)
    x = rng.standard_normal(d).astype(np.float32)
    sel = [4, 1, 5, 0]
    w = rng.random(k).astype(np.float32)
    w /= w.sum()
    ys = np.stack([oracle.expert(x, slabs[e], d, f) for e in sel])
    y_sh = oracle.expert(x, shared, d, 2 * f)
    hits, misses = [0, 2], [1, 3]                  # ranks that ran on the GPU / on the host
    y_gpu = oracle.combine(ys[hits], w[hits])
    y_host = oracle.combine(ys[misses], w[misses])
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    out = torch.full((d,), float("nan"), device="cuda")
    moe.combine(out, dev(y_gpu), dev(y_host), dev(y_sh))
    torch.cuda.synchronize()
    r = assert_close(out.cpu().numpy(), oracle.combine(ys, w, y_shared=y_sh), "combine, hits + misses + shared")
    # every hit (no host part, no shared expert) and every miss (no GPU part)
    moe.combine(out, dev(oracle.combine(ys, w)), None, None)
    torch.cuda.synchronize()
    assert_close(out.cpu().numpy(), oracle.combine(ys, w), "combine, all hits")
    moe.combine(out, None, dev(oracle.combine(ys, w)), dev(y_sh))
    torch.cuda.synchronize()
    assert_close(out.cpu().numpy(), oracle.combine(ys, w, y_shared=y_sh), "combine, all misses + shared")
    moe.combine(out)
    assert torch.count_nonzero(out) == 0            # nothing selected: zero output
    say("  max|err|/RMS", r)
