"""C-ABI library checks that need no GPU: symbols, argument validation, and the
host-side parts of the path (LRU slot table, host expert path) against the oracle."""
import ctypes
import itertools
import json
import random
import re
import os

import numpy as np
import pytest

import oracle
from oracle import lru as olru
import synth

import paper_2512_16473_amd as moe  # noqa: E402
from paper_2512_16473_amd import _abi  # noqa: E402

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "moe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z0-9_]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = _declared_functions()
    assert len(names) >= 25
    lib = ctypes.CDLL(_abi.LIB_PATH)
    for name in names:
        assert hasattr(lib, name), name
    assert {s[0] for s in _abi.SIGNATURES} == set(names)


def test_version_and_sizes():
    lib = moe.lib()
    assert lib.moe_version() >= 100
    assert moe.slab_bytes(4096, 14336) == 352_321_536
    assert moe.slab_bytes(256, 512) % 256 == 0 and moe.slab_bytes(256, 512) >= 3 * 256 * 512 * 2
    assert moe.slab_bytes(0, 8) == 0


def test_argument_errors_do_not_touch_the_device():
    lib = moe.lib()
    # k > n, n too large, d not a multiple of 8: rejected before any HIP call
    assert lib.moe_router_topk(None, None, 1, 64, 4, 5, None, None, None) == _abi.MOE_EINVAL
    assert b"k=5" in lib.moe_last_error()
    assert lib.moe_router_topk(None, None, 1, 64, 300, 2, None, None, None) == _abi.MOE_EINVAL
    assert lib.moe_router_topk(None, None, 1, 60, 8, 2, None, None, None) == _abi.MOE_EINVAL
    assert lib.moe_router_topk(None, None, 0, 64, 8, 2, None, None, None) == _abi.MOE_OK   # T == 0: no-op
    assert lib.moe_expert_ffn_hits(None, None, 4, None, None, 2, 64, 64, None, None, 0, None) == _abi.MOE_EINVAL
    assert lib.moe_expert_ffn_hits(None, None, 4, None, None, 17, 64, 64, None, None, 0, None) == _abi.MOE_EINVAL
    assert lib.moe_combine(None, None, None, 16, None, None) == _abi.MOE_EINVAL
    assert lib.moe_runtime_create(None, None) == _abi.MOE_EINVAL
    # multi-token FFN: T, k, the staging limit and pointers checked before any HIP call
    assert lib.moe_expert_ffn_tokens(None, None, 4, None, None, 0, 2, 256, 512, None, None, 0, None) == \
        _abi.MOE_EINVAL
    assert lib.moe_expert_ffn_tokens(None, None, 4, None, None, 9, 2, 256, 512, None, None, 0, None) == \
        _abi.MOE_EINVAL
    assert lib.moe_expert_ffn_tokens(None, None, 4, None, None, 8, 2, 8192, 512, None, None, 0, None) == \
        _abi.MOE_EINVAL                                                    # 8 x 8192 floats > 128 KiB
    assert b"staging" in lib.moe_last_error()
    assert lib.moe_expert_ffn_tokens(None, None, 4, None, None, 2, 17, 256, 512, None, None, 0, None) == \
        _abi.MOE_EINVAL
    assert lib.moe_expert_ffn_tokens(None, None, 4, None, None, 2, 2, 256, 512, None, None, 0, None) == \
        _abi.MOE_EINVAL                                                    # null pointers
    assert lib.moe_ffn_tokens_workspace_bytes(0, 2, 256, 512) == 0
    assert lib.moe_ffn_tokens_workspace_bytes(2, 2, 256, 512) >= 4 * 512 * 4 + 4 * 256 * 4
    # allocation-free hit FFN: the scratch limit and the arguments checked before any HIP call
    assert lib.moe_ffn_noalloc_max_bytes() == 8 << 20
    a = ctypes.c_void_p(1 << 20)       # an aligned stand-in address: never dereferenced here
    assert lib.moe_expert_ffn_hits_noalloc(a, a, 4, a, a, 2, 8192, 65536, a, None) == _abi.MOE_EINVAL
    assert b"scratch" in lib.moe_last_error()
    assert moe.ffn_workspace_bytes(2, 8192, 65536) > lib.moe_ffn_noalloc_max_bytes()
    assert moe.ffn_workspace_bytes(2, 4096, 14336) <= lib.moe_ffn_noalloc_max_bytes()
    assert lib.moe_expert_ffn_hits_noalloc(None, a, 4, a, a, 2, 64, 64, a, None) == _abi.MOE_EINVAL
    assert lib.moe_expert_ffn_hits_noalloc(a, a, 4, a, a, 17, 64, 64, a, None) == _abi.MOE_EINVAL
    assert lib.moe_expert_ffn_hits_noalloc(a, a, 4, a, a, 2, 60, 64, a, None) == _abi.MOE_EINVAL
    # read-stream yardstick: size, grid and pointers checked before any HIP call
    assert lib.moe_read_stream(None, 24, None, 0, None) == _abi.MOE_EINVAL
    assert b"multiple of 16" in lib.moe_last_error()
    assert lib.moe_read_stream(None, 32, None, -1, None) == _abi.MOE_EINVAL
    assert lib.moe_read_stream(None, 32, None, 0, None) == _abi.MOE_EINVAL
    assert lib.moe_read_stream(None, 0, None, 0, None) == _abi.MOE_OK   # nothing to read: no-op


def test_cache_create_validation():
    with pytest.raises(moe.MoeError):
        moe.Cache(2, 8, 1, 2)          # ways < top_k
    with pytest.raises(moe.MoeError):
        moe.Cache(2, 8, 9, 2)          # ways > n
    with pytest.raises(moe.MoeError):
        moe.Cache(-1, 8, 4, 2)
    empty = moe.Cache(0, 8, 4, 2)      # no covered layer: a runtime runs every layer on the host
    with pytest.raises(moe.MoeError):
        empty.update(0, [1, 2])
    c = moe.Cache(2, 8, 4, 2)
    with pytest.raises(moe.MoeError):
        c.update(0, [1, 1])            # duplicate ids
    with pytest.raises(moe.MoeError):
        c.update(2, [1, 2])            # layer out of range
    with pytest.raises(moe.MoeError):
        c.update(0, [1, 8])            # id out of range
    with pytest.raises(moe.MoeError):
        c.update(0, [1, 2, 3])         # more than top_k
    assert np.all(c.slotmap(0) == -1)  # failed calls changed nothing


def _lib_trace(seq, n, ways, k):
    c = moe.Cache(1, n, ways, k)
    out = []
    for sel in seq:
        slots, hits = c.lookup(0, sel)
        fill, ev = c.update(0, sel)
        out.append((list(slots), list(hits), list(fill), list(ev)))
    return out, c


@pytest.mark.parametrize("k,ways,length", [(1, 1, 6), (1, 2, 6), (1, 3, 6), (1, 4, 6),
                                           (2, 2, 6), (2, 3, 6), (2, 4, 6)])
def test_library_lru_exhaustive_vs_oracle(k, ways, length):
    n = 4
    subs = [list(c) for c in itertools.combinations(range(n), k)]
    rng = random.Random(ways * 7 + k)
    c = moe.Cache(1, n, ways, k)
    for seq in itertools.product(subs, repeat=length):
        seq = [rng.sample(s, len(s)) for s in seq]
        c.reset()
        ref = olru.LRUSet(ways)
        for sel in seq:
            slots, hits = c.lookup(0, sel)
            fill, ev = c.update(0, sel)
            r_slots, r_hits, r_fill, r_ev = ref.access(sel)
            assert list(slots) == r_slots and list(hits) == r_hits
            assert list(fill) == r_fill and list(ev) == r_ev


@pytest.mark.parametrize("n,k,ways", [(8, 2, 4), (16, 2, 6), (64, 8, 24)])
def test_library_lru_long_traces_vs_oracle(n, k, ways):
    rng = random.Random(n + ways)
    L = 3
    c = moe.Cache(L, n, ways, k)
    ref = olru.LRUCache(L, ways)
    # correlated selections (a mix of reuse and fresh draws), several layers interleaved
    prev = [rng.sample(range(n), k) for _ in range(L)]
    for t in range(600):
        for layer in range(L):
            keep = [e for e in prev[layer] if rng.random() < 0.6]
            fresh = [e for e in rng.sample(range(n), n) if e not in keep][: k - len(keep)]
            sel = keep + fresh
            rng.shuffle(sel)
            prev[layer] = sel
            slots, hits = c.lookup(layer, sel)
            fill, ev = c.update(layer, sel)
            r = ref.access(layer, sel)
            assert (list(slots), list(hits), list(fill), list(ev)) == r
            assert list(c.slotmap(layer)) == ref.slotmap(layer, n)


@pytest.mark.parametrize("policy", ["lru", "fifo", "static"])
@pytest.mark.parametrize("n,k,ways", [(8, 2, 4), (16, 2, 6), (64, 8, 24), (4, 1, 2)])
def test_library_policies_vs_oracle(policy, n, k, ways):
    """Section IV-D's policies: the library's slots, hits, fills and evictions equal the
    oracle's on correlated multi-layer traces, and reset restores the initial state."""
    rng = random.Random(sum(map(ord, policy)) * 1000 + n * 100 + k * 10 + ways)
    L = 3
    content = [rng.sample(range(n), ways) for _ in range(L)] if policy == "static" else None
    c = moe.Cache(L, n, ways, k, policy=policy, static_content=content)
    for rep in range(2):
        ref = olru.LRUCache(L, ways, policy=policy, static_content=content)
        prev = [rng.sample(range(n), k) for _ in range(L)]
        for t in range(300):
            for layer in range(L):
                keep = [e for e in prev[layer] if rng.random() < 0.6]
                fresh = [e for e in rng.sample(range(n), n) if e not in keep][: k - len(keep)]
                sel = keep + fresh
                rng.shuffle(sel)
                prev[layer] = sel
                slots, hits = c.lookup(layer, sel)
                fill, ev = c.update(layer, sel)
                assert (list(slots), list(hits), list(fill), list(ev)) == ref.access(layer, sel)
                assert list(c.slotmap(layer)) == ref.slotmap(layer, n)
        c.reset()


@pytest.mark.parametrize("policy", ["lru", "fifo"])
def test_library_masked_insertion_vs_oracle(policy):
    """Bounded post-fetch: misses that may not be inserted (random masks) give the same
    slots, hits, fills and evictions as the oracle's masked access."""
    rng = random.Random(sum(map(ord, policy)))
    n, k, ways, L = 8, 2, 4, 2
    c = moe.Cache(L, n, ways, k, policy=policy)
    ref = olru.LRUCache(L, ways, policy=policy)
    for t in range(500):
        for layer in range(L):
            sel = rng.sample(range(n), k)
            ins = [rng.random() < 0.4 for _ in sel]
            slots, hits = c.lookup(layer, sel)
            fill, ev = c.update_masked(layer, sel, ins)
            assert (list(slots), list(hits), list(fill), list(ev)) == ref.access(layer, sel, ins)
            assert list(c.slotmap(layer)) == ref.slotmap(layer, n)


@pytest.mark.parametrize("policy", ["lru", "fifo", "static"])
def test_cache_checkpoint_resume(policy):
    """A cache saved mid-trace and restored into a new cache of the same geometry goes on
    exactly like the original and like the oracle's uninterrupted cache (plain and masked
    insertion), and restoring returns the table it was saved from."""
    rng = random.Random(17 + sum(map(ord, policy)))
    n, k, ways, L = 8, 2, 4, 3
    content = [rng.sample(range(n), ways) for _ in range(L)] if policy == "static" else None
    a = moe.Cache(L, n, ways, k, policy=policy, static_content=content)
    ref = olru.LRUCache(L, ways, policy=policy, static_content=content)

    def step(caches, layer, sel, ins):
        r = ref.access(layer, sel, ins)
        for c in caches:
            slots, hits = c.lookup(layer, sel)
            fill, ev = c.update_masked(layer, sel, ins)
            assert (list(slots), list(hits), list(fill), list(ev)) == r
            assert list(c.slotmap(layer)) == ref.slotmap(layer, n)

    for t in range(40):
        for layer in range(L):
            sel = rng.sample(range(n), k)
            step([a], layer, sel, [rng.random() < 0.8 for _ in sel])
    state = a.save()
    assert len(state) == 28 + L * ways * 12 + L * 8
    b = moe.Cache(L, n, ways, k, policy=policy, static_content=content)
    b.restore(state)
    assert b.save() == state
    for layer in range(L):
        assert list(b.slotmap(layer)) == list(a.slotmap(layer))
    for t in range(40):
        for layer in range(L):
            sel = rng.sample(range(n), k)
            step([a, b], layer, sel, [rng.random() < 0.8 for _ in sel])


def test_cache_restore_rejects_bad_states():
    """A state of another geometry or policy, a truncated or foreign buffer, and
    inconsistent contents are refused with EINVAL and leave the cache as it was."""
    import struct
    n, k, ways, L = 8, 2, 4, 2
    src = moe.Cache(L, n, ways, k)
    for sel in ([0, 1], [2, 3], [4, 1], [5, 6]):
        src.update(0, sel)
    good = bytearray(src.save())
    dst = moe.Cache(L, n, ways, k)
    dst.update(1, [7, 6])
    before = dst.save()
    head, sx0, su0, ck0 = 28, 28, 28 + L * ways * 4, 28 + L * ways * 12

    def patched(off, fmt, value):
        b = bytearray(good)
        struct.pack_into(fmt, b, off, value)
        return bytes(b)

    bad = {
        "truncated": bytes(good[:-1]),
        "foreign": b"x" * len(good),
        "other policy": patched(24, "<i", 1),
        "expert out of range": patched(sx0, "<i", n),
        "expert twice": patched(sx0 + 4, "<i", struct.unpack_from("<i", good, sx0)[0]),
        "stamp after clock": patched(su0, "<Q", struct.unpack_from("<Q", good, ck0)[0] + 1),
        "stamp 0 on a resident slot": patched(su0, "<Q", 0),
        "two slots one stamp": patched(su0 + 8, "<Q", struct.unpack_from("<Q", good, su0)[0]),
    }
    for what, state in bad.items():
        with pytest.raises(moe.MoeError):
            dst.restore(state)
        assert dst.save() == before, what
    with pytest.raises(moe.MoeError):
        moe.Cache(L, n, ways + 1, k).restore(bytes(good))          # another geometry
    with pytest.raises(moe.MoeError):
        moe.Cache(L, n, ways, k, policy="static",
                  static_content=[[0, 1, 2, 3]] * L).restore(bytes(good))
    st = moe.Cache(1, n, 2, 2, policy="static", static_content=[[3, 5]]).save()
    with pytest.raises(moe.MoeError):    # a static set whose content differs
        moe.Cache(1, n, 2, 2, policy="static", static_content=[[5, 3]]).restore(st)
    lib = _abi.load()
    assert lib.moe_cache_state_bytes(None) == 0
    assert lib.moe_cache_save(None, None, 0) == _abi.MOE_EINVAL
    buf = ctypes.create_string_buffer(len(good) - 1)
    assert lib.moe_cache_save(src.handle, buf, len(good) - 1) == _abi.MOE_EINVAL


def test_static_policy_validation():
    with pytest.raises(moe.MoeError):
        moe.Cache(1, 8, 2, 2, policy="static", static_content=[[1, 1]])      # duplicate
    with pytest.raises(moe.MoeError):
        moe.Cache(1, 8, 2, 2, policy="static", static_content=[[1, 8]])      # out of range
    lib = _abi.load()
    h = ctypes.c_void_p()
    assert lib.moe_cache_create_policy(1, 8, 2, 2, 2, None, ctypes.byref(h)) == _abi.MOE_EINVAL  # no content
    assert lib.moe_cache_create_policy(1, 8, 2, 2, 7, None, ctypes.byref(h)) == _abi.MOE_EINVAL  # no such policy
    # a static set may have fewer ways than top_k: misses are never inserted
    c = moe.Cache(1, 8, 1, 2, policy="static", static_content=[[5]])
    fill, ev = c.update(0, [5, 2])
    assert list(fill) == [-1, -1] and list(ev) == [-1, -1]
    assert list(c.lookup(0, [2, 5])[1]) == [False, True]


def test_cache_geometry_vs_oracle(golden_dir):
    """Section III-B sizing through the library equals the oracle's (and the paper's
    worked example: 56 slots, 4 ways -> 14 indexes, layers 0-13)."""
    ex = json.load(open(os.path.join(golden_dir, "paper_cache_sizing.json")))["example"]
    assert moe.cache_geometry(ex["slots"], 1, ex["ways"], 32) == (ex["slots"], ex["indexes"])
    for budget, eb, ways, L in [(24 * 10**9, 352_321_536, 4, 32), (10**12, 352_321_536, 4, 32),
                                (3 * 10**8, 352_321_536, 4, 32), (80 * 10**9, 157_286_400, 6, 32)]:
        S, N, covered = olru.cache_geometry(budget, eb, ways, L)
        assert moe.cache_geometry(budget, eb, ways, L) == (S, len(covered))


def _pool_case(d, f, ne, seed):
    slabs = [synth.expert_slab(seed + j, d, f, None) for j in range(ne)]
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(d).astype(np.float32)
    w = rng.random(ne).astype(np.float32)
    w /= w.sum()
    return x, slabs, w


def _cpu_flags():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("flags"):
                    return set(line.split(":", 1)[1].split())
    except OSError:
        pass
    return set()


_HOST_DOTS = ["fp32"] + (["bf16"] if "avx512_bf16" in _cpu_flags() else [])


@pytest.mark.parametrize("dot", _HOST_DOTS)
@pytest.mark.parametrize("d,f,ne", [(256, 512, 2), (64, 40, 3), (512, 1024, 1), (128, 96, 8), (4096, 136, 2)])
def test_host_expert_path_vs_oracle(d, f, ne, dot):
    """Both forms of the host dot product (fp32 widening; AVX512_BF16 pair-dot with
    hi + lo activation parts) against the oracle, at fp32-accumulation error; f = 40,
    96, 136 leave 8, 0 and 8 elements past a 32-wide step (the masked tail)."""
    x, slabs, w = _pool_case(d, f, ne, 40 + d + ne)
    pool = moe.HostPool(4)
    pool.set_dot(dot)
    assert pool.dot == dot
    y = pool.expert_ffn(x, slabs, w, d, f)
    ys = np.stack([oracle.expert(x, s, d, f) for s in slabs])
    ref = oracle.combine(ys, w)
    rms = float(np.sqrt(np.mean(ref.astype(np.float64) ** 2)))
    err = float(np.max(np.abs(y - ref)))
    assert err <= 1e-4 * rms, (err, rms)


@pytest.mark.parametrize("dot", _HOST_DOTS)
def test_host_expert_path_thread_independent_and_empty(dot):
    d, f = 256, 512
    x, slabs, w = _pool_case(d, f, 2, 5)
    p1, p5 = moe.HostPool(1), moe.HostPool(5)
    p1.set_dot(dot)
    p5.set_dot(dot)
    y1 = p1.expert_ffn(x, slabs, w, d, f)
    y5 = p5.expert_ffn(x, slabs, w, d, f)
    assert np.array_equal(y1, y5)
    y0 = moe.HostPool(3).expert_ffn(x, [], np.zeros(0, np.float32), d, f, y=np.full(d, 7.0, np.float32))
    assert np.all(y0 == 0)
    with pytest.raises(moe.MoeError):
        moe.HostPool(2).expert_ffn(x, slabs, w, 250, f)


def test_host_pool_dot_kinds_and_shared_use():
    """The dot-form switch (unknown kinds refused; bf16 refused without AVX512_BF16),
    and one pool used from several threads at once: calls are serialised, so every
    result equals the one-call result."""
    import threading
    p = moe.HostPool(3)
    assert p.dot == "fp32"
    p.set_dot("auto")
    assert p.dot == "fp32"
    with pytest.raises(KeyError):
        p.set_dot("fp8")
    assert _abi_lib().moe_host_pool_set_dot(p.handle, 7) == -1
    if "bf16" not in _HOST_DOTS:
        with pytest.raises(moe.MoeError):
            p.set_dot("bf16")
    d, f = 128, 96
    cases = [_pool_case(d, f, 2, 70 + i) for i in range(6)]
    want = [p.expert_ffn(x, s, w, d, f) for x, s, w in cases]
    got = [None] * len(cases)

    def work(i):
        for _ in range(20):
            x, s, w = cases[i]
            got[i] = p.expert_ffn(x, s, w, d, f)

    th = [threading.Thread(target=work, args=(i,)) for i in range(len(cases))]
    for t in th:
        t.start()
    for t in th:
        t.join()
    for a, b in zip(got, want):
        assert np.array_equal(a, b)


def _abi_lib():
    from paper_2512_16473_amd import _lib
    return _lib
