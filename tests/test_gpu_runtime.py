"""The whole per-layer decode path (router, cache check/update, hit FFN on the GPU,
misses on the host, post-fetch, combine) vs the oracle: routing bit-exact (near-tie
protocol), hit/miss trace and slot table bit-exact against the oracle LRU replayed on
the chosen expert sets, outputs within 2e-2 x RMS."""
import os

import numpy as np
import pytest

import oracle
from oracle import lru as olru
import synth
from _gpu_util import assert_close, make_slabs_host, router_parity, say, torch_cuda

pytestmark = pytest.mark.gpu


class World:
    """A decode world on the GPU: router weights, slot pool, pinned host experts,
    shared experts, AR(1) hidden states, library runtime."""

    def __init__(self, name, L=None, T=None, ways=None, threads=4, seed=0, policy="lru", covered=None, wl=None):
        torch = torch_cuda()
        import paper_2512_16473_amd as moe
        wl = wl or synth.WORKLOADS[name]
        self.wl = wl
        self.L = L or wl.L
        self.T = T or wl.T
        self.ways = ways or wl.ways
        d, f, n, k = wl.d, wl.f, wl.n, wl.k
        self.d, self.f, self.n, self.k = d, f, n, k
        self.wr = np.stack([synth.router_weights(synth.seed_for(seed, name, "router", l), n, d)
                            for l in range(self.L)])
        self.X = np.stack([synth.ar1_states(synth.seed_for(seed, name, "states", l), self.T, d)
                           for l in range(self.L)])                       # [L, T, d]
        self.host, stride, self.views = make_slabs_host(torch, self.L, n, d, f, wl.w_std, seed, name)
        self.host_addrs = [self.host.ptr + i * stride for i in range(self.L * n)]
        self.policy = policy
        self.covered = self.L if covered is None else covered
        # the static policy's content: a seeded uniform draw of `ways` experts per layer
        rng = np.random.default_rng(synth.seed_for(seed, name, "static-content"))
        self.content = [sorted(rng.choice(n, self.ways, replace=False).tolist()) for _ in range(self.covered)]
        self.pool = (torch.zeros(self.covered * self.ways * stride, dtype=torch.uint8, device="cuda")
                     if self.covered else None)
        self.shared = None
        self.shared_views = None
        if wl.f_shared:
            sh_host, sstride, self.shared_views = make_slabs_host(torch, self.L, 1, d, wl.f_shared, wl.w_std, seed,
                                                                  name, kind="shared")
            self.shared = torch.from_numpy(sh_host.array).cuda()
            self._sh_host = sh_host
        self.cache = moe.Cache(self.covered, n, self.ways, k, policy=policy,
                               static_content=self.content if policy == "static" else None)
        self.hpool = moe.HostPool(threads)
        self.rt = moe.Runtime(d, f, n, k, self.ways, self.L, torch.from_numpy(self.wr).cuda(), self.pool,
                              self.host_addrs, self.cache, self.hpool, f_shared=wl.f_shared,
                              shared_pool=self.shared)
        self.streams = (torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream())
        self.xd = torch.from_numpy(np.ascontiguousarray(self.X.transpose(1, 0, 2))).cuda()   # [T, L, d]
        self.out = torch.empty((self.T, self.L, d), dtype=torch.float32, device="cuda")

    def run(self, steps):
        idx = np.empty((steps, self.L, self.k), np.int32)
        w = np.empty((steps, self.L, self.k), np.float32)
        hit = np.empty((steps, self.L, self.k), np.uint8)
        for t in range(steps):
            self.rt.decode_step(self.xd[t], self.out[t], self.streams, idx[t], w[t], hit[t])
        import torch
        torch.cuda.synchronize()
        self.rt.sync()
        return idx, w, hit.astype(bool), self.out[:steps].cpu().numpy()

    def oracle_out(self, layer, t, expert_set):
        slabs = self.views[layer * self.n:(layer + 1) * self.n]
        sh = None if self.shared_views is None else self.shared_views[layer]
        _, _, out, _ = oracle.moe_token(self.X[layer, t], self.wr[layer], slabs, self.k, self.f,
                                        shared_slab=sh, f_shared=self.wl.f_shared, forced_set=expert_set)
        return out


def _check_trace(world, idx, w, hit, out, steps, layers, check_out):
    """Replays the GPU's chosen sets through the oracle's cache (same policy; layers
    past the covered ones never hit and hold nothing)."""
    ref = olru.LRUCache(world.covered, world.ways, policy=world.policy,
                        static_content=world.content if world.policy == "static" else None)
    worst = 0.0
    for t in range(steps):
        for l in range(world.L):
            if l in layers:
                oidx, ow = router_parity(idx[t, l], w[t, l], world.X[l, t], world.wr[l], world.k)
            if l < world.covered:
                slots, hits, fills, ev = ref.access(l, list(idx[t, l]))
            else:
                hits = [False] * world.k
            assert list(hit[t, l]) == hits, (t, l, list(hit[t, l]), hits)
            if l in layers and check_out(t, l):
                o = world.oracle_out(l, t, oidx)
                worst = max(worst, assert_close(out[t, l], o, f"t={t} layer={l}"))
    for l in range(world.L):
        expect = ref.slotmap(l, world.n) if l < world.covered else [-1] * world.n
        assert list(world.rt.device_slotmap(l)) == expect
        if l < world.covered:
            assert list(world.cache.slotmap(l)) == expect
    return worst


def test_runtime_tiny_full_trace():
    say("runtime tiny full trace")
    world = World("tiny")
    steps = world.T
    idx, w, hit, out = world.run(steps)
    worst = _check_trace(world, idx, w, hit, out, steps, set(range(world.L)), lambda t, l: True)
    st = world.rt.stats()
    assert st["expert_hits"] + st["expert_misses"] == steps * world.L * world.k
    assert st["fills"] == st["expert_misses"]
    assert 0 < st["expert_hits"] and 0 < st["expert_misses"]
    say("  worst max|err|/RMS", worst, "hit rate", st["expert_hits"] / (steps * world.k))


def test_runtime_tiny_all_resident_and_host_only_agree():
    """Caching decides only where an expert runs, never its result (Section I: the
    method keeps the model's accuracy): M = n (all hits after warm-up) vs M = k."""
    say("runtime tiny M=n vs M=k")
    a = World("tiny", ways=4, T=24)
    b = World("tiny", ways=2, T=24)
    ia, wa, ha, oa = a.run(24)
    ib, wb, hb, ob = b.run(24)
    assert np.array_equal(ia, ib)
    assert ha[4:].sum() > hb[4:].sum()
    for t in range(24):
        assert_close(oa[t, 0], ob[t, 0], f"t={t}")


@pytest.mark.parametrize("name,L,T,layers", [("mixtral", 2, 10, {0, 1}), ("phi", 1, 12, {0}),
                                             ("fine", 1, 8, {0})])
def test_runtime_full_shapes(name, L, T, layers):
    """Full per-layer shapes; fewer layers and steps than the benchmark (host memory
    and oracle time), same kernels and launch configuration; every step's output of
    every listed layer compared."""
    oracle.set_threads(min(16, os.cpu_count() or 1))
    say("runtime", name, "L", L, "T", T)
    world = World(name, L=L, T=T, threads=8)
    idx, w, hit, out = world.run(T)
    worst = _check_trace(world, idx, w, hit, out, T, layers, lambda t, l: True)
    say("  worst max|err|/RMS", worst)


@pytest.mark.parametrize("d,n,k,ways", [(3072, 16, 4, 8), (2048, 40, 3, 6), (8192, 8, 2, 4), (768, 256, 16, 16)])
def test_runtime_router_shapes(d, n, k, ways):
    """The single-token decode routers at their edges, through the whole path: a router
    matrix read by one work group (at most 64 (expert, 1024-float segment) items, segment
    count dividing 8: d = 8192 with 8 segments) and by many work groups with the arrival
    counter (3 segments; 80 items; 256 experts top-16), over many layer calls so the
    counter's reset is exercised. Routing, trace and every output against the oracle."""
    oracle.set_threads(min(16, os.cpu_count() or 1))
    say("runtime router shape", d, n, k, ways)
    wl = synth.Workload("tiny", d=d, f=256, n=n, k=k, L=2, T=12, ways=ways, w_std=None)
    world = World("tiny", wl=wl)
    idx, w, hit, out = world.run(wl.T)
    worst = _check_trace(world, idx, w, hit, out, wl.T, {0, 1}, lambda t, l: True)
    say("  worst max|err|/RMS", worst)


@pytest.mark.parametrize("policy", ["fifo", "static"])
def test_runtime_tiny_policies(policy):
    """Section IV-D's other policies through the whole path: FIFO (post-fetch as LRU,
    no refresh on hits) and static (fixed content loaded at creation, misses never
    fetched). Trace bit-exact against the oracle's policy, outputs within tolerance."""
    say("runtime tiny policy", policy)
    world = World("tiny", policy=policy)
    steps = world.T
    idx, w, hit, out = world.run(steps)
    worst = _check_trace(world, idx, w, hit, out, steps, set(range(world.L)), lambda t, l: True)
    st = world.rt.stats()
    assert st["expert_hits"] + st["expert_misses"] == steps * world.L * world.k
    assert st["fills"] == (0 if policy == "static" else st["expert_misses"])
    say("  worst max|err|/RMS", worst, "hit rate", st["expert_hits"] / (steps * world.k))


@pytest.mark.parametrize("covered", [0, 1, 2])
def test_runtime_uncovered_layers(covered):
    """Section III-B: a memory budget covers layers 0..N-1 only; the other layers run
    every selected expert on the host and fetch nothing. Three tiny-shaped layers."""
    say("runtime tiny, 3 layers, covered", covered)
    world = World("tiny", L=3, T=20, covered=covered)
    idx, w, hit, out = world.run(20)
    worst = _check_trace(world, idx, w, hit, out, 20, {0, 1, 2}, lambda t, l: True)
    st = world.rt.stats()
    assert not hit[:, covered:].any()
    assert st["fills"] == st["expert_misses"] - 20 * (3 - covered) * world.k
    say("  worst max|err|/RMS", worst)


def test_runtime_mixtral_static_policy():
    """Mixtral-shaped layer with a static 4-of-8 content: the four resident slabs are
    loaded at creation and every other expert always runs on the host."""
    oracle.set_threads(min(16, os.cpu_count() or 1))
    say("runtime mixtral static")
    world = World("mixtral", L=1, T=6, threads=8, policy="static")
    idx, w, hit, out = world.run(6)
    worst = _check_trace(world, idx, w, hit, out, 6, {0}, lambda t, l: True)
    assert world.rt.stats()["fills"] == 0
    say("  worst max|err|/RMS", worst)


@pytest.mark.parametrize("name,L,T,limit", [("tiny", 1, 64, 1), ("tiny", 3, 24, 2), ("mixtral", 2, 8, 1)])
def test_runtime_bounded_postfetch(name, L, T, limit):
    """Bounded post-fetch (at most `limit` slabs in flight): a miss beyond the budget runs
    on the host and is not inserted. Which misses were inserted depends on copy timing,
    so it is read back from the cache table after every layer call; replaying the GPU's
    sets with those insertions through the oracle's masked LRU must reproduce every hit,
    slot and the device mirror bit for bit, and the outputs stay within tolerance."""
    oracle.set_threads(min(16, os.cpu_count() or 1))
    say("runtime bounded post-fetch", name, L, T, limit)
    world = World(name, L=L, T=T, threads=8)
    world.rt.set_fill_limit(limit)
    import torch
    ref = olru.LRUCache(world.L, world.ways)
    sc = world.streams
    worst = 0.0
    skipped = 0
    for t in range(T):
        for l in range(world.L):
            idx, w, hit = world.rt.layer_forward(l, world.xd[t, l], world.out[t, l], sc)
            after = world.cache.slotmap(l)
            inserted = [bool(after[e] >= 0) for e in idx]          # hits stay, inserted misses appear
            slots, hits, fills, ev = ref.access(l, list(idx), inserted)
            assert list(hit) == hits, (t, l)
            assert list(after) == ref.slotmap(l, world.n), (t, l)
            skipped += sum(1 for h, i in zip(hits, inserted) if not h and not i)
            torch.cuda.synchronize()
            oidx, ow = router_parity(idx, w, world.X[l, t], world.wr[l], world.k)
            o = world.oracle_out(l, t, oidx)
            worst = max(worst, assert_close(world.out[t, l].cpu().numpy(), o, f"t={t} layer={l}"))
    torch.cuda.synchronize()
    world.rt.sync()
    for l in range(world.L):
        assert list(world.rt.device_slotmap(l)) == ref.slotmap(l, world.n)
    st = world.rt.stats()
    assert st["fills_skipped"] == skipped
    assert st["fills"] + st["fills_skipped"] == st["expert_misses"]
    say("  worst max|err|/RMS", worst, "fills", st["fills"], "skipped", skipped)


@pytest.mark.parametrize("name,L,T,limit", [("tiny", 3, 24, 0), ("mixtral", 2, 8, 0), ("mixtral", 2, 8, 2)])
def test_runtime_nonblocking(name, L, T, limit):
    """Non-blocking post-fetch: a layer call never waits for its set's copies; an expert
    whose copy has not landed runs on the host. The cache table must still follow the
    oracle bit for bit (read back before and after every call, replayed with the
    insertions it shows), the GPU may only run table hits, every output must match the
    oracle (no expert counted twice or lost), and after a sync the device mirror equals
    the table."""
    oracle.set_threads(min(16, os.cpu_count() or 1))
    say("runtime non-blocking", name, L, T, limit)
    world = World(name, L=L, T=T, threads=8)
    world.rt.set_nonblocking(True)
    world.rt.set_fill_limit(limit)
    import torch
    ref = olru.LRUCache(world.L, world.ways)
    worst = 0.0
    inflight = 0
    for t in range(T):
        for l in range(world.L):
            before = world.cache.slotmap(l)
            idx, w, gpu = world.rt.layer_forward(l, world.xd[t, l], world.out[t, l], world.streams)
            after = world.cache.slotmap(l)
            table_hits = [bool(before[e] >= 0) for e in idx]
            inserted = [bool(after[e] >= 0) for e in idx]
            slots, hits, fills, ev = ref.access(l, list(idx), inserted)
            assert hits == table_hits, (t, l)
            assert list(after) == ref.slotmap(l, world.n), (t, l)
            assert all(h or not g for g, h in zip(gpu, table_hits)), (t, l)   # GPU runs table hits only
            inflight += sum(1 for g, h in zip(gpu, table_hits) if h and not g)
            torch.cuda.synchronize()
            oidx, ow = router_parity(idx, w, world.X[l, t], world.wr[l], world.k)
            o = world.oracle_out(l, t, oidx)
            worst = max(worst, assert_close(world.out[t, l].cpu().numpy(), o, f"t={t} layer={l}"))
    world.rt.sync()
    for l in range(world.L):
        assert list(world.rt.device_slotmap(l)) == ref.slotmap(l, world.n)
    st = world.rt.stats()
    assert st["inflight_misses"] == inflight
    say("  worst max|err|/RMS", worst, "in-flight misses", inflight, "fills", st["fills"])


@pytest.mark.parametrize("nonblocking", [False, True])
def test_runtime_delayed_copies(nonblocking):
    """Post-fetch copies held back on purpose: before every token a bounded spin kernel
    (about 10 ms) is queued on the copy stream, so each token's post-fetches land late.
    Parity mode must then make the compute stream wait for them (trace and outputs equal
    to the oracle, as without the delay); non-blocking mode must run the experts whose
    copies are still in flight on the host (some of them do, every output still
    matches the oracle)."""
    torch = torch_cuda()
    oracle.set_threads(min(16, os.cpu_count() or 1))
    say("runtime delayed copies, non-blocking" if nonblocking else "runtime delayed copies, parity")
    world = World("tiny", L=3, T=24, threads=4)
    world.rt.set_nonblocking(nonblocking)
    ref = olru.LRUCache(world.L, world.ways)
    worst, inflight = 0.0, 0
    for t in range(world.T):
        with torch.cuda.stream(world.streams[2]):
            torch.cuda._sleep(20_000_000)
        for l in range(world.L):
            before = world.cache.slotmap(l)
            idx, w, gpu = world.rt.layer_forward(l, world.xd[t, l], world.out[t, l], world.streams)
            after = world.cache.slotmap(l)
            table_hits = [bool(before[e] >= 0) for e in idx]
            slots, hits, fills, ev = ref.access(l, list(idx), [bool(after[e] >= 0) for e in idx])
            assert hits == table_hits, (t, l)
            assert list(after) == ref.slotmap(l, world.n), (t, l)
            if nonblocking:
                assert all(h or not g for g, h in zip(gpu, table_hits)), (t, l)
                inflight += sum(1 for g, h in zip(gpu, table_hits) if h and not g)
            else:
                assert list(gpu) == table_hits, (t, l)       # parity: every table hit runs on the GPU
            world.streams[0].synchronize()    # the output only: the copy stream keeps running
            oidx, ow = router_parity(idx, w, world.X[l, t], world.wr[l], world.k)
            worst = max(worst, assert_close(world.out[t, l].cpu().numpy(), world.oracle_out(l, t, oidx),
                                            f"t={t} layer={l}"))
    world.rt.sync()
    for l in range(world.L):
        assert list(world.rt.device_slotmap(l)) == ref.slotmap(l, world.n)
    st = world.rt.stats()
    assert st["inflight_misses"] == inflight
    if nonblocking:
        assert inflight > 0
    say("  worst max|err|/RMS", worst, "in-flight misses", inflight, "fills", st["fills"])


def test_runtime_resume_from_checkpoint():
    """Stop a decode half way, save the cache state, drop the runtime and clear the
    device slot pool (as a new process would start), restore the state into a new cache
    and runtime: the runtime refills the held slots from the host, and the continued
    trace and outputs equal the oracle's uninterrupted run."""
    torch = torch_cuda()
    import paper_2512_16473_amd as moe
    say("runtime resume from a cache checkpoint")
    world = World("tiny", L=3, T=24, threads=4)
    half = world.T // 2
    idx = np.empty((world.T, world.L, world.k), np.int32)
    w = np.empty((world.T, world.L, world.k), np.float32)
    hit = np.empty((world.T, world.L, world.k), np.uint8)
    for t in range(half):
        world.rt.decode_step(world.xd[t], world.out[t], world.streams, idx[t], w[t], hit[t])
    torch.cuda.synchronize()
    world.rt.sync()
    state = world.cache.save()
    world.rt.close()
    world.cache.close()
    world.pool.zero_()
    torch.cuda.synchronize()
    cache = moe.Cache(world.L, world.n, world.ways, world.k)
    cache.restore(state)
    rt = moe.Runtime(world.d, world.f, world.n, world.k, world.ways, world.L, torch.from_numpy(world.wr).cuda(),
                     world.pool, world.host_addrs, cache, world.hpool)
    world.cache, world.rt = cache, rt
    for t in range(half, world.T):
        rt.decode_step(world.xd[t], world.out[t], world.streams, idx[t], w[t], hit[t])
    torch.cuda.synchronize()
    rt.sync()
    out = world.out.cpu().numpy()
    worst = _check_trace(world, idx, w, hit.astype(bool), out, world.T, set(range(world.L)), lambda t, l: True)
    say("  worst max|err|/RMS", worst)
