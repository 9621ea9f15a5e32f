"""Expert-cache policy oracle -- TEST INFRASTRUCTURE ONLY.

Section III-A/B of the paper: GPU memory holds an N-index, M-way set-associative
expert cache whose index is the layer number; each set keeps up to M experts of
its layer and evicts with LRU. On each access (one token at one layer) the cache
is checked for the selected experts (step 1), hits run on the GPU and misses on
the CPU (step 2), and every missed expert is then copied into the cache so
later tokens hit it (step 3).

Points the paper leaves open, and the reading taken here:
  * hits are decided for all selected experts against the state before the token;
  * the set is then updated in ascending expert-id order, one clock tick per
    expert: a hit refreshes its slot's stamp; a miss takes the lowest-index empty
    slot, else the least recently stamped slot whose expert is not selected by the
    current token (a current-token expert is never a victim);
  * the cache starts empty and every miss is inserted (so k <= M is required).

`LRUSet` is that procedure. `definitional_hits` is an independent statement of the
same policy (content = the M experts with the most recent use keys) and
`textbook_lru_hits` is classic single-reference LRU (stack distance < M) for k = 1.

Section IV-D compares LRU with two other policies, modelled here the same way:
  * `FIFOSet`: first in, first out -- identical to `LRUSet` except that a hit does
    not refresh its slot, so the victim is the earliest-inserted slot whose expert
    is not selected by the current token;
  * `StaticSet` (the paper's "random" policy): a fixed set of M experts chosen once
    (the caller draws it, e.g. uniformly at random, and passes it in); misses are
    never inserted, so the content never changes.
`textbook_fifo_hits` is classic single-reference FIFO for k = 1.
"""
from __future__ import annotations

from typing import Iterable, List, Sequence, Tuple


class LRUSet:
    """One set (one layer) of the expert cache with M ways."""

    def __init__(self, ways: int):
        if ways < 1:
            raise ValueError("ways must be >= 1")
        self.ways = ways
        self.expert = [-1] * ways     # expert held by each slot, -1 = empty
        self.stamp = [0] * ways       # last-use clock of each slot
        self.clock = 0

    def content(self) -> set:
        return {e for e in self.expert if e >= 0}

    def lookup(self, selected: Sequence[int]) -> Tuple[List[int], List[bool]]:
        """Step 1, pure: slot of each selected expert (-1 on miss) and the hit mask."""
        slots = [self.expert.index(e) if e in self.expert else -1 for e in selected]
        return slots, [s >= 0 for s in slots]

    def access(self, selected: Sequence[int], insert=None):
        """Check, then update for one token. `selected` is in rank order.

        insert (optional, aligned with `selected`): False for a missed expert that must
        not be inserted (its post-fetch was not issued); such a miss takes no slot and
        evicts nothing, though it still takes its clock tick.

        Returns (slots, hits, fills, evicted), each aligned with `selected`:
        slots[j]   slot holding expert j before the update (-1 on miss)
        hits[j]    whether expert j was cached before the token
        fills[j]   slot expert j was inserted into (-1 on hit or when not inserted)
        evicted[j] expert removed to make room for j (-1 if none)
        """
        sel = list(selected)
        allow = dict(zip(sel, [True] * len(sel) if insert is None else [bool(v) for v in insert]))
        if len(set(sel)) != len(sel):
            raise ValueError("selected experts must be distinct")
        if len(sel) > self.ways:
            raise ValueError("more selected experts than ways")
        slots, hits = self.lookup(sel)
        hit_of = dict(zip(sel, hits))
        current = set(sel)
        fill_of, evict_of = {}, {}
        for e in sorted(sel):
            self.clock += 1
            if hit_of[e]:
                self.stamp[self.expert.index(e)] = self.clock
                continue
            if not allow[e]:
                continue
            empty = [s for s in range(self.ways) if self.expert[s] < 0]
            if empty:
                victim = empty[0]
            else:
                candidates = [s for s in range(self.ways) if self.expert[s] not in current]
                victim = min(candidates, key=lambda s: self.stamp[s])
            fill_of[e] = victim
            evict_of[e] = self.expert[victim]
            self.expert[victim] = e
            self.stamp[victim] = self.clock
        fills = [fill_of.get(e, -1) for e in sel]
        evicted = [evict_of.get(e, -1) for e in sel]
        return slots, hits, fills, evicted


class FIFOSet(LRUSet):
    """One set with first-in-first-out replacement: a hit leaves the stamps alone,
    so a slot's stamp is the clock of its insertion."""

    def access(self, selected: Sequence[int], insert=None):
        sel = list(selected)
        if len(set(sel)) != len(sel):
            raise ValueError("selected experts must be distinct")
        if len(sel) > self.ways:
            raise ValueError("more selected experts than ways")
        allow = dict(zip(sel, [True] * len(sel) if insert is None else [bool(v) for v in insert]))
        slots, hits = self.lookup(sel)
        hit_of = dict(zip(sel, hits))
        current = set(sel)
        fill_of, evict_of = {}, {}
        for e in sorted(sel):
            self.clock += 1
            if hit_of[e]:
                continue                      # no refresh: insertion order decides
            if not allow[e]:
                continue
            empty = [s for s in range(self.ways) if self.expert[s] < 0]
            if empty:
                victim = empty[0]
            else:
                candidates = [s for s in range(self.ways) if self.expert[s] not in current]
                victim = min(candidates, key=lambda s: self.stamp[s])
            fill_of[e] = victim
            evict_of[e] = self.expert[victim]
            self.expert[victim] = e
            self.stamp[victim] = self.clock
        fills = [fill_of.get(e, -1) for e in sel]
        evicted = [evict_of.get(e, -1) for e in sel]
        return slots, hits, fills, evicted


class StaticSet(LRUSet):
    """One set whose content is fixed: slot s holds content[s] forever."""

    def __init__(self, ways: int, content: Sequence[int]):
        super().__init__(ways)
        content = list(content)
        if len(content) != ways or len(set(content)) != ways or min(content) < 0:
            raise ValueError("static content must be `ways` distinct expert ids")
        self.expert = content

    def access(self, selected: Sequence[int], insert=None):
        sel = list(selected)
        if len(set(sel)) != len(sel):
            raise ValueError("selected experts must be distinct")
        slots, hits = self.lookup(sel)
        return slots, hits, [-1] * len(sel), [-1] * len(sel)


POLICIES = {"lru": LRUSet, "fifo": FIFOSet}


class LRUCache:
    """The N-index (one index per layer), M-way cache.

    policy "lru" (the paper's), "fifo", or "static" with `static_content[layer]`
    giving each covered layer's M experts. Only layers 0..n_layers-1 own a set.
    """

    def __init__(self, n_layers: int, ways: int, policy: str = "lru", static_content=None):
        if policy == "static":
            self.sets = [StaticSet(ways, static_content[l]) for l in range(n_layers)]
        else:
            self.sets = [POLICIES[policy](ways) for _ in range(n_layers)]

    def access(self, layer: int, selected: Sequence[int], insert=None):
        return self.sets[layer].access(selected, insert)

    def slotmap(self, layer: int, n_experts: int) -> List[int]:
        """Expert -> slot table of one layer (-1 when not cached)."""
        m = [-1] * n_experts
        for s, e in enumerate(self.sets[layer].expert):
            if e >= 0:
                m[e] = s
        return m


def definitional_hits(trace: Iterable[Sequence[int]], ways: int) -> List[List[bool]]:
    """Hit masks from the content definition, with no slots or stamps.

    Each expert carries the key (last token that used it, its position in
    ascending-id order within that token). After token t the cache holds the
    min(M, #distinct) experts with the largest keys; expert e hits at token t iff it
    is in the content after token t-1.
    """
    key = {}
    content: set = set()
    out = []
    for t, sel in enumerate(trace):
        out.append([e in content for e in sel])
        for pos, e in enumerate(sorted(sel)):
            key[e] = (t, pos)
        ranked = sorted(key, key=lambda e: key[e], reverse=True)
        content = set(ranked[:ways])
    return out


def definitional_hits_masked(trace: Iterable[Sequence[int]], inserts: Iterable[Sequence[bool]],
                             ways: int) -> List[List[bool]]:
    """`definitional_hits` when some misses are not inserted: the content after token t
    is the min(M, size) experts with the largest keys among the content after token
    t-1 plus the misses of token t that were inserted; hits and inserted misses take
    the key (t, position in ascending-id order)."""
    key = {}
    content: set = set()
    out = []
    for t, (sel, ins) in enumerate(zip(trace, inserts)):
        hits = [e in content for e in sel]
        out.append(hits)
        allow = dict(zip(sel, ins))
        for pos, e in enumerate(sorted(sel)):
            if e in content or allow[e]:
                key[e] = (t, pos)
        pool = content | {e for e in sel if allow[e]}
        content = set(sorted(pool, key=lambda e: key[e], reverse=True)[:ways])
    return out


def textbook_lru_hits(trace: Iterable[int], ways: int) -> List[bool]:
    """Classic LRU for one reference per step: a hit iff fewer than M distinct
    other items were referenced since the item's previous reference."""
    hist: List[int] = []
    out = []
    for e in trace:
        if e in hist:
            last = len(hist) - 1 - hist[::-1].index(e)
            out.append(len(set(hist[last + 1:])) < ways)
        else:
            out.append(False)
        hist.append(e)
    return out


def textbook_fifo_hits(trace: Iterable[int], ways: int) -> List[bool]:
    """Classic FIFO for one reference per step: a queue of at most M items; a miss
    appends the item and drops the oldest when the queue is over M; a hit changes
    nothing."""
    queue: List[int] = []
    out = []
    for e in trace:
        if e in queue:
            out.append(True)
            continue
        out.append(False)
        queue.append(e)
        if len(queue) > ways:
            queue.pop(0)
    return out


def cache_geometry(avail_bytes: int, expert_bytes: int, ways: int, n_layers: int):
    """Section III-B sizing: S = floor(avail / per-expert size), N = floor(S / M).

    Returns (S, N, covered) where covered = the layers 0..min(N, n_layers)-1 that own
    a cache set; layers from N on run every expert on the host.
    """
    if expert_bytes <= 0 or ways <= 0:
        raise ValueError("expert_bytes and ways must be positive")
    S = int(avail_bytes) // int(expert_bytes)
    N = S // int(ways)
    return S, N, list(range(min(N, n_layers)))
