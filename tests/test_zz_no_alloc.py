"""The allocation-free hit FFN (moe_expert_ffn_hits_noalloc, its scratch in a static
device array) against the entry point with a caller workspace (moe_expert_ffn_hits):
same kernels, so the outputs must agree bit for bit, and both within tolerance of the
oracle. Two calls in a row, the second with a smaller input, so the second runs over
the first's leftovers in the shared scratch."""
import os

import numpy as np
import pytest

import oracle
import synth
from _gpu_util import assert_close, say, torch_cuda

pytestmark = pytest.mark.gpu


def _case(torch, d, f, nslots, slots, seed, full=False):
    import paper_2512_16473_amd as moe
    stride = moe.slab_bytes(d, f)
    pool = torch.zeros(nslots * stride, dtype=torch.uint8, device="cuda")
    host = []
    for s in range(nslots):
        t = pool[s * stride: s * stride + 3 * d * f * 2].view(torch.bfloat16)
        synth.expert_slab_torch(synth.seed_for(seed, "noalloc", "expert", d, s), d, f, 0.02 if full else None, out=t)
        host.append(t.view(torch.uint8).cpu().numpy().view(np.uint16))
    rng = np.random.default_rng(seed + d)
    x = rng.standard_normal(d).astype(np.float32)
    w = rng.random(len(slots)).astype(np.float32)
    w /= w.sum()
    return pool, host, x, w


def _both(torch, pool, nslots, slots, x, w, d, f):
    import paper_2512_16473_amd as moe
    xd = torch.from_numpy(x).cuda()
    sd = torch.tensor(slots, dtype=torch.int32, device="cuda")
    wd = torch.from_numpy(w).cuda()
    ws = torch.empty(moe.ffn_workspace_bytes(len(slots), d, f), dtype=torch.uint8, device="cuda")
    y_ws = torch.full((d,), float("nan"), device="cuda")
    y_na = torch.full((d,), float("nan"), device="cuda")
    moe.expert_ffn_hits(xd, pool, nslots, sd, wd, d, f, y_ws, ws)
    moe.expert_ffn_hits_noalloc(xd, pool, nslots, sd, wd, d, f, y_na)
    torch.cuda.synchronize()
    return y_ws.cpu().numpy(), y_na.cpu().numpy()


def test_noalloc_matches_workspace_entry_point():
    torch = torch_cuda()
    oracle.set_threads(min(16, os.cpu_count() or 1))
    # first call: the Mixtral-8x7B expert shape, two hits out of three slots
    d, f, slots = 4096, 14336, [2, 0]
    say("noalloc call 1", d, f, slots)
    pool, host, x, w = _case(torch, d, f, 3, slots, 1, full=True)
    y_ws, y_na = _both(torch, pool, 3, slots, x, w, d, f)
    assert np.array_equal(y_ws, y_na)
    ref = oracle.combine(np.stack([oracle.expert(x, host[s], d, f) for s in slots]), w)
    r1 = assert_close(y_na, ref, "noalloc mixtral shape")
    # second call, smaller: ragged d and f, three hits, one slot out of range (skipped)
    d, f, slots = 264, 520, [1, 5, 0, 2]
    say("noalloc call 2", d, f, slots)
    pool, host, x, w = _case(torch, d, f, 3, slots, 2)
    y_ws, y_na = _both(torch, pool, 3, slots, x, w, d, f)
    assert np.array_equal(y_ws, y_na)
    keep = [j for j, s in enumerate(slots) if s < 3]
    ref = oracle.combine(np.stack([oracle.expert(x, host[slots[j]], d, f) for j in keep]), w[keep])
    r2 = assert_close(y_na, ref, "noalloc ragged")
    # third: nothing to compute gives zeros
    y0_ws, y0_na = _both(torch, pool, 3, [], x, np.zeros(0, np.float32), d, f)
    assert np.all(y0_na == 0) and np.array_equal(y0_ws, y0_na)
    say("  max|err|/RMS", r1, r2)


def test_noalloc_rejects_oversize():
    torch = torch_cuda()
    import paper_2512_16473_amd as moe
    x = torch.zeros(8192, device="cuda")
    with pytest.raises(moe.MoeError):
        moe.expert_ffn_hits_noalloc(x, x, 1, torch.zeros(2, dtype=torch.int32, device="cuda"),
                                    torch.zeros(2, device="cuda"), 8192, 65536, x)
