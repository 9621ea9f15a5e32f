"""GPU router gating vs the oracle (Section I MoE layer; Table II top-K)."""
import numpy as np
import pytest

import oracle
import synth
from _gpu_util import router_parity, say, torch_cuda

pytestmark = pytest.mark.gpu


def _run(torch, X, wr, k):
    import paper_2512_16473_amd as moe
    xd = torch.from_numpy(X).cuda()
    wd = torch.from_numpy(wr).cuda()
    idx, w = moe.router_topk(xd, wd, k)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), w.cpu().numpy()


@pytest.mark.parametrize("d,n,k,T", [(256, 4, 2, 64), (4096, 8, 2, 256), (4096, 16, 2, 64),
                                     (3584, 64, 8, 64), (264, 8, 1, 33), (4096, 8, 8, 16), (8192, 256, 16, 4)])
def test_router_parity_ar1(d, n, k, T):
    torch = torch_cuda()
    say("router", d, n, k, T)
    wr = synth.router_weights(synth.seed_for(1, "mixtral", "router", d, n), n, d)
    X = synth.ar1_states(synth.seed_for(1, "mixtral", "states", d, k), T, d)
    gi, gw = _run(torch, X, wr, k)
    for t in range(T):
        router_parity(gi[t], gw[t], X[t], wr, k)


def test_router_exact_ties():
    torch = torch_cuda()
    say("router ties")
    d, n = 64, 8
    X = np.random.default_rng(0).standard_normal((4, d)).astype(np.float32)
    # zero router: every logit is 0, the k lowest ids win with equal weights
    gi, gw = _run(torch, X, np.zeros((n, d), np.float32), 3)
    assert np.all(gi == np.array([0, 1, 2])) and np.all(gw == np.float32(1 / 3))
    # duplicated rows tie exactly; the lower id ranks first
    wr = np.random.default_rng(1).standard_normal((n, d)).astype(np.float32)
    for t in range(4):
        l = wr.astype(np.float64) @ X[t]
        top = int(np.argmax(l))
        other = (top + 3) % n
        wr2 = wr.copy()
        wr2[other] = wr2[top]
        gi, gw = _run(torch, X[t:t + 1], wr2, 2)
        idx, w, _, _ = oracle.router(X[t], wr2, 2)
        assert list(gi[0]) == list(idx) == sorted([top, other])
        assert gw[0][0] == gw[0][1] == np.float32(0.5)


def test_router_empty_batch_is_noop():
    torch = torch_cuda()
    import paper_2512_16473_amd as moe
    idx = torch.full((1, 2), -7, dtype=torch.int32, device="cuda")
    w = torch.zeros((1, 2), dtype=torch.float32, device="cuda")
    x = torch.zeros((0, 64), dtype=torch.float32, device="cuda")
    wr = torch.zeros((8, 64), dtype=torch.float32, device="cuda")
    moe.router_topk(x, wr, 2, idx_out=idx, w_out=w)
    torch.cuda.synchronize()
    assert int(idx[0, 0]) == -7
