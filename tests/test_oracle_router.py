"""Pins for the oracle's router gating (Section I MoE layer, Table II top-K).

The router formula is not printed in the paper; the reading is softmax over all
logits, top-k with ties to the lower id, renormalised. These tests pin the oracle to
hand-derived closed forms, to an independent brute-force characterisation of the
top-k set (the k-subset with the largest logit sum), and to invariants.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle


def _sigmoid(z):
    return 1.0 / (1.0 + math.exp(-z))


def _closed(expr, x):
    xs = [float(v) for v in x]
    m = max(xs)
    e = [math.exp(v - m) for v in xs]
    sm = [v / sum(e) for v in e]
    env = {"sigmoid": _sigmoid, "softmax": lambda _x: sm, "x": xs}
    return eval(expr, {"__builtins__": {}}, env)


def test_hand_cases(golden_dir):
    data = json.load(open(os.path.join(golden_dir, "router_hand_cases.json")))
    for c in data["cases"]:
        x = np.array(c["x"], dtype=np.float32)
        wr = np.eye(4, dtype=np.float32) if c["wr"] == "identity" else np.zeros((4, 4), np.float32)
        idx, w, gap, logits = oracle.router(x, wr, c["k"])
        assert list(idx) == c["idx"], c["name"]
        for got, expr in zip(w, c["w_closed_form"]):
            exp_v = _closed(expr, x)
            assert abs(float(got) - exp_v) <= 2 * np.spacing(np.float32(exp_v)), (c["name"], got, exp_v)


def _brute_topk(l, k):
    """The top-k set is the k-subset with the largest logit sum; among subsets with
    equal sums (ties) the lexicographically smallest sorted id tuple."""
    best = None
    for comb in itertools.combinations(range(len(l)), k):
        s = sum(l[i] for i in comb)
        if best is None or s > best[0]:
            best = (s, comb)
    return set(best[1])


@pytest.mark.parametrize("n,k", [(4, 1), (4, 2), (6, 2), (6, 3), (8, 2), (16, 2), (8, 8)])
def test_topk_set_brute_force(n, k):
    rng = np.random.default_rng(100 + n * 10 + k)
    d = 32
    for _ in range(40):
        wr = rng.standard_normal((n, d)).astype(np.float32)
        x = rng.standard_normal(d).astype(np.float32)
        idx, w, gap, logits = oracle.router(x, wr, k)
        l64 = wr.astype(np.float64) @ x.astype(np.float64)
        assert np.allclose(logits, l64, rtol=1e-12, atol=1e-12)
        assert set(idx.tolist()) == _brute_topk(l64, k)
        # ordered by logit descending
        assert all(l64[idx[i]] >= l64[idx[i + 1]] for i in range(k - 1))
        # gate weights: renormalised softmax restricted to the set, in closed form
        ref = np.exp(l64[idx] - l64[idx[0]])
        ref = ref / ref.sum()
        assert np.allclose(w, ref, rtol=4e-7, atol=1e-9)
        # margin between the last chosen and the best unchosen logit
        if k < n:
            rest = np.delete(l64, idx)
            assert math.isclose(gap, l64[idx[-1]] - rest.max(), rel_tol=1e-12, abs_tol=1e-12)
        else:
            assert math.isinf(gap)


def test_invariants():
    rng = np.random.default_rng(7)
    for n, k in [(8, 2), (16, 2), (64, 8), (4, 4), (8, 1)]:
        d = 64
        for _ in range(25):
            wr = (rng.standard_normal((n, d)) / math.sqrt(d)).astype(np.float32)
            x = rng.standard_normal(d).astype(np.float32)
            idx, w, gap, logits = oracle.router(x, wr, k)
            assert len(set(idx.tolist())) == k
            assert abs(float(np.sum(w, dtype=np.float64)) - 1.0) <= 4 * np.finfo(np.float32).eps
            assert all(w[i] >= w[i + 1] for i in range(k - 1))
            if k == 1:
                assert w[0] == 1.0
            if k == 2:
                assert math.isclose(float(w[0]), _sigmoid(logits[idx[0]] - logits[idx[1]]), rel_tol=3e-7)
            if k == n:
                p = np.exp(logits - logits.max())
                p /= p.sum()
                assert np.allclose(w, p[idx], rtol=4e-7, atol=1e-9)


def test_duplicate_rows_tie_to_lower_id():
    # experts 1 and 5 have identical router rows: they tie exactly; with k = 1 and
    # both at the top, the lower id wins.
    rng = np.random.default_rng(3)
    d, n = 16, 6
    wr = rng.standard_normal((n, d)).astype(np.float32)
    x = rng.standard_normal(d).astype(np.float32)
    l = wr.astype(np.float64) @ x
    top = int(np.argmax(l))
    wr[5] = wr[top]
    lo = min(top, 5)
    idx, w, gap, _ = oracle.router(x, wr, 1)
    assert idx[0] == lo and gap == 0.0
    idx2, w2, _, _ = oracle.router(x, wr, 2)
    assert sorted(idx2.tolist()) == sorted({top, 5}) and idx2[0] == lo
    assert w2[0] == w2[1] == 0.5


def test_forced_set_matches_router_on_its_own_set():
    rng = np.random.default_rng(11)
    d, n, k = 32, 8, 2
    wr = rng.standard_normal((n, d)).astype(np.float32)
    x = rng.standard_normal(d).astype(np.float32)
    idx, w, _, _ = oracle.router(x, wr, k)
    idx2, w2 = oracle.router_forced(x, wr, k, idx[::-1].copy())
    assert list(idx2) == list(idx) and np.array_equal(w, w2)
    with pytest.raises(ValueError):
        oracle.router_forced(x, wr, k, [3, 3])


def test_bad_sizes():
    x = np.zeros(4, np.float32)
    with pytest.raises(ValueError):
        oracle.router(x, np.zeros((4, 4), np.float32), 5)
