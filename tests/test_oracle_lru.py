"""Pins for the oracle's expert cache (Section III-A/B LRU; Section IV-D closed form).

The procedural LRU is checked against an independent definitional model on every
access sequence of small caches, against textbook single-reference LRU for k = 1,
against structural invariants, and statistically against the paper's closed-form
hit probabilities for i.i.d. selections.
"""
import itertools
import json
import math
import os
import random

import pytest

from oracle import lru


def _subsets(n, k):
    return [list(c) for c in itertools.combinations(range(n), k)]


def _run(seq, ways):
    s = lru.LRUSet(ways)
    return [s.access(sel) for sel in seq], s


@pytest.mark.parametrize("k,ways,length", [(1, 1, 6), (1, 2, 6), (1, 3, 6), (1, 4, 6),
                                           (2, 2, 6), (2, 3, 6), (2, 4, 6)])
def test_exhaustive_vs_definitional(k, ways, length):
    n = 4
    subs = _subsets(n, k)
    rng = random.Random(k * 100 + ways)
    for seq in itertools.product(subs, repeat=length):
        # rank order inside a token does not matter for the cache; permute it
        seq = [rng.sample(s, len(s)) for s in seq]
        res, st = _run(seq, ways)
        hits = [r[1] for r in res]
        assert hits == lru.definitional_hits(seq, ways)
        if k == 1:
            assert [h[0] for h in hits] == lru.textbook_lru_hits([s[0] for s in seq], ways)


def _check_invariants(seq, ways, n):
    s = lru.LRUSet(ways)
    seen = set()
    prev_content = set()
    for sel in seq:
        slots, hits, fills, evicted = s.access(sel)
        for j, e in enumerate(sel):
            assert hits[j] == (e in prev_content)
            assert (slots[j] >= 0) == hits[j] and (fills[j] >= 0) != hits[j]
            assert 0 <= (slots[j] if hits[j] else fills[j]) < ways
            if not hits[j]:
                assert evicted[j] not in sel                     # never evict a current expert
                if evicted[j] >= 0:
                    assert evicted[j] in prev_content
        content = s.content()
        occupied = [e for e in s.expert if e >= 0]
        assert len(occupied) == len(set(occupied)) <= ways    # no duplicates, capacity
        assert set(sel) <= content                            # every selected expert is cached
        if ways == n:
            for j, e in enumerate(sel):
                assert hits[j] == (e in seen)                 # only first-use misses
        seen |= set(sel)
        prev_content = content


@pytest.mark.parametrize("n,k,ways", [(8, 2, 4), (16, 2, 6), (64, 8, 24), (8, 2, 8), (4, 2, 2), (64, 8, 8)])
def test_invariants_random(n, k, ways):
    rng = random.Random(n * 1000 + k * 10 + ways)
    seq = [rng.sample(range(n), k) for _ in range(400)]
    _check_invariants(seq, ways, n)


@pytest.mark.parametrize("n,k", [(8, 2), (6, 3)])
def test_inclusion_property(n, k):
    """hits with M ways are a subset of hits with M+1 ways, access by access."""
    rng = random.Random(n + k)
    seq = [rng.sample(range(n), k) for _ in range(300)]
    prev = None
    for ways in range(k, n + 1):
        res, _ = _run(seq, ways)
        hits = [h for r in res for h in r[1]]
        if prev is not None:
            assert all((not a) or b for a, b in zip(prev, hits))
        prev = hits


def test_slot_assignment_trace():
    """A hand-traced 2-way sequence: slots, fills and evictions."""
    s = lru.LRUSet(2)
    assert s.access([3, 1]) == ([-1, -1], [False, False], [1, 0], [-1, -1])  # ascending ids: 1->slot0, 3->slot1
    assert s.access([1, 2]) == ([0, -1], [True, False], [-1, 1], [-1, 3])    # 3 is LRU and not current
    assert s.access([2, 0]) == ([1, -1], [True, False], [-1, 0], [-1, 1])
    assert s.access([0, 2]) == ([0, 1], [True, True], [-1, -1], [-1, -1])


def _make_set(policy, n, M, rng):
    if policy == "static":
        return lru.StaticSet(M, rng.sample(range(n), M))
    return {"lru": lru.LRUSet, "fifo": lru.FIFOSet}[policy](M)


@pytest.mark.parametrize("policy", ["lru", "fifo", "static"])
def test_random_policy_closed_form(golden_dir, policy):
    """Section IV-D: a static random set of M experts hits with the closed-form
    probabilities. With i.i.d. uniform expert pairs the content of an LRU or FIFO
    cache is independent of the next draw too, so their long-run hit rates must
    converge to the same formulas."""
    data = json.load(open(os.path.join(golden_dir, "paper_random_policy.json")))
    for c in data["cases"]:
        n, M = c["n"], c["M"]
        p_any = 1 - ((n - M) / n) * ((n - M - 1) / (n - 1))
        p_both = (M / n) * ((M - 1) / (n - 1))
        rng = random.Random(n * 31 + M)
        s = _make_set(policy, n, M, rng)
        N = 20000
        any_hits = both_hits = 0
        for t in range(N + 50):
            _, hits, _, _ = s.access(rng.sample(range(n), 2))
            if t >= 50:
                any_hits += any(hits)
                both_hits += all(hits)
        for got, p in ((any_hits / N, p_any), (both_hits / N, p_both)):
            sigma = math.sqrt(p * (1 - p) / N)
            assert abs(got - p) <= 4 * sigma + 1e-12, (c["name"], got, p)


def test_cache_sizing_example(golden_dir):
    ex = json.load(open(os.path.join(golden_dir, "paper_cache_sizing.json")))["example"]
    per_expert = 1  # slots counted directly in the worked example
    S, N, covered = lru.cache_geometry(ex["slots"] * per_expert, per_expert, ex["ways"], 32)
    assert (S, N) == (ex["slots"], ex["indexes"])
    assert (covered[0], covered[-1]) == tuple(ex["covered_layers"])
    # from memory sizes: (24 - 5) GB / 340 MB gives about 56 slots
    S2, _, _ = lru.cache_geometry((ex["gpu_GB"] - ex["non_expert_GB"]) * 10**9, ex["per_expert_MB"] * 10**6, 4, 32)
    assert abs(S2 - ex["slots"]) <= 2
    assert 8 * 32 == ex["total_experts"]


def test_rejects_bad_access():
    s = lru.LRUSet(2)
    with pytest.raises(ValueError):
        s.access([1, 1])
    with pytest.raises(ValueError):
        s.access([0, 1, 2])


# ---- FIFO and static (Section IV-D's comparison policies) ---------------------------

@pytest.mark.parametrize("ways", [1, 2, 3, 4])
def test_fifo_k1_exhaustive_vs_textbook(ways):
    """k = 1: the procedural FIFO set equals a plain bounded queue on every
    sequence of length 6 over 4 experts."""
    for seq in itertools.product(range(4), repeat=6):
        s = lru.FIFOSet(ways)
        hits = [s.access([e])[1][0] for e in seq]
        assert hits == lru.textbook_fifo_hits(list(seq), ways), seq


def test_fifo_differs_from_lru_by_hand():
    """M = 2, k = 1, accesses 1 2 1 3 1: LRU keeps 1 (refreshed by its hit) and evicts
    2; FIFO evicts 1, the earliest inserted, so the last access misses."""
    seq = [1, 2, 1, 3, 1]
    lru_s, fifo_s = lru.LRUSet(2), lru.FIFOSet(2)
    assert [lru_s.access([e])[1][0] for e in seq] == [False, False, True, False, True]
    assert [fifo_s.access([e])[1][0] for e in seq] == [False, False, True, False, False]


@pytest.mark.parametrize("n,k,ways", [(8, 2, 4), (16, 2, 6), (64, 8, 24), (4, 2, 2)])
def test_fifo_invariants(n, k, ways):
    """Capacity, no duplicates, every selected expert cached after its token, a
    current expert never evicted, and a hit never changes any slot or stamp."""
    rng = random.Random(7 * n + k + ways)
    s = lru.FIFOSet(ways)
    prev_content = set()
    for _ in range(400):
        sel = rng.sample(range(n), k)
        before = (list(s.expert), list(s.stamp))
        slots, hits, fills, evicted = s.access(sel)
        for j, e in enumerate(sel):
            assert hits[j] == (e in prev_content)
            if not hits[j]:
                assert evicted[j] not in sel
        if all(hits):
            assert (list(s.expert), list(s.stamp)) == before
        occupied = [e for e in s.expert if e >= 0]
        assert len(occupied) == len(set(occupied)) <= ways
        assert set(sel) <= s.content()
        prev_content = s.content()


def test_fifo_evicts_in_insertion_order():
    """With every slot full and no current-token conflicts, the victims come out in
    the order the experts went in, whatever the hits in between."""
    s = lru.FIFOSet(3)
    for e in (5, 6, 7):
        s.access([e])
    s.access([5])          # a hit: FIFO does not refresh
    s.access([6])
    _, _, _, ev = s.access([8])
    assert ev == [5]
    _, _, _, ev = s.access([9])
    assert ev == [6]


def test_static_set_never_changes():
    rng = random.Random(3)
    content = [4, 1, 6, 2]
    s = lru.StaticSet(4, content)
    for _ in range(200):
        sel = rng.sample(range(8), 2)
        slots, hits, fills, evicted = s.access(sel)
        assert hits == [e in content for e in sel]
        assert slots == [content.index(e) if e in content else -1 for e in sel]
        assert fills == [-1, -1] and evicted == [-1, -1]
        assert s.expert == content
    with pytest.raises(ValueError):
        lru.StaticSet(2, [1, 1])


# ---- bounded post-fetch: misses that are not inserted -------------------------------

@pytest.mark.parametrize("k,ways", [(1, 2), (2, 2), (2, 3)])
def test_masked_insertion_vs_definitional(k, ways):
    """A miss whose post-fetch is not issued is not inserted. Against the content
    definition (top-M keys among the old content and the inserted misses) on every
    length-5 sequence over 4 experts, with random insertion masks."""
    subs = _subsets(4, k)
    rng = random.Random(11 * k + ways)
    for seq in itertools.product(subs, repeat=5):
        seq = [rng.sample(s_, len(s_)) for s_ in seq]
        masks = [[rng.random() < 0.5 for _ in s_] for s_ in seq]
        s = lru.LRUSet(ways)
        hits = [s.access(sel, ins)[1] for sel, ins in zip(seq, masks)]
        assert hits == lru.definitional_hits_masked(seq, masks, ways)


def test_masked_insertion_extremes():
    rng = random.Random(5)
    seq = [rng.sample(range(8), 2) for _ in range(200)]
    a, b = lru.LRUSet(4), lru.LRUSet(4)
    for sel in seq:                                   # all allowed == plain LRU
        assert a.access(sel, [True, True]) == b.access(sel)
    c = lru.LRUSet(4)
    c.access([1, 2])
    for sel in seq:                                   # nothing allowed: content frozen
        _, hits, fills, ev = c.access(sel, [False, False])
        assert hits == [e in (1, 2) for e in sel] and fills == [-1, -1] and ev == [-1, -1]
        assert c.content() == {1, 2}
