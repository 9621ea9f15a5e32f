"""Pins for the oracle's SwiGLU expert and combine (Section I; Table II size reading).

Pinned against SwiGLU special cases, scalar cases derived by hand, an fp64 numpy
brute force on small shapes, the decomposition of a layer into per-expert outputs,
and thread-count independence.
"""
import math

import numpy as np
import pytest

import oracle
import synth


def _silu(z):
    return z / (1.0 + math.exp(-z))


def _np_expert(x, slab, d, f):
    """Test-side definition: y = W2 (SiLU(W1 x) * W3 x), fp64 throughout."""
    w = synth.bf16_to_f32(slab).astype(np.float64)
    w1 = w[: f * d].reshape(f, d)
    w3 = w[f * d: 2 * f * d].reshape(f, d)
    w2 = w[2 * f * d:].reshape(d, f)
    x = x.astype(np.float64)
    g, u = w1 @ x, w3 @ x
    h = g / (1.0 + np.exp(-g)) * u
    return w2 @ h


def _slab_from(w1, w3, w2):
    return synth.bf16_bits(np.concatenate([np.ravel(w1), np.ravel(w3), np.ravel(w2)]).astype(np.float32))


def test_scalar_by_hand():
    # d = f = 1: y = w2 * SiLU(w1 x) * (w3 x); all values exact in bf16
    for w1, w3, w2, x in [(1.0, 1.0, 1.0, 1.0), (0.5, 2.0, -1.5, 3.0), (-2.0, 0.25, 4.0, 1.0)]:
        slab = _slab_from([w1], [w3], [w2])
        y = oracle.expert(np.array([x], np.float32), slab, 1, 1)
        ref = w2 * _silu(w1 * x) * (w3 * x)
        assert abs(float(y[0]) - ref) <= 2 * np.spacing(np.float32(abs(ref)))
    # SiLU(1) = sigma(1) = 0.7310585786...
    y = oracle.expert(np.array([1.0], np.float32), _slab_from([1.0], [1.0], [1.0]), 1, 1)
    assert abs(float(y[0]) - 0.7310585786300049) < 1e-7


def test_special_cases():
    rng = np.random.default_rng(1)
    d, f = 16, 24
    slab = synth.expert_slab(5, d, f, None)
    # x = 0 -> y = 0
    assert np.all(oracle.expert(np.zeros(d, np.float32), slab, d, f) == 0)
    # W3 = 0 -> y = 0
    s2 = slab.copy()
    s2[f * d: 2 * f * d] = 0
    assert np.all(oracle.expert(rng.standard_normal(d).astype(np.float32), s2, d, f) == 0)
    # large gate: SiLU(g) -> g, so y -> W2 (g * u)
    x = np.zeros(4, np.float32)
    x[0] = 40.0
    s3 = _slab_from(np.eye(4), np.eye(4), np.eye(4))
    y = oracle.expert(x, s3, 4, 4)
    assert abs(float(y[0]) - 1600.0) < 1e-3 and np.all(y[1:] == 0)
    # large negative gate: SiLU(g) -> 0
    x[0] = -40.0
    y = oracle.expert(x, s3, 4, 4)
    assert abs(float(y[0])) < 1e-12


@pytest.mark.parametrize("d,f,std", [(8, 16, None), (32, 48, None), (64, 128, 0.02), (256, 512, None)])
def test_brute_force_fp64(d, f, std):
    slab = synth.expert_slab(17 + d, d, f, std)
    rng = np.random.default_rng(d * 7 + f)
    for _ in range(3):
        x = rng.standard_normal(d).astype(np.float32)
        y = oracle.expert(x, slab, d, f).astype(np.float64)
        ref = _np_expert(x, slab, d, f)
        rms = math.sqrt(float(np.mean(ref ** 2)))
        # the oracle rounds g, u, h and y to fp32; the brute force does not
        assert np.max(np.abs(y - ref)) <= 1e-6 * max(rms, 1e-30), (np.max(np.abs(y - ref)), rms)


def test_bf16_widening_exact():
    a = np.random.default_rng(0).standard_normal(1000).astype(np.float32)
    b = synth.bf16_bits(a)
    w = synth.bf16_to_f32(b)
    assert np.array_equal(synth.bf16_bits(w), b)           # round trip of bf16 values is exact
    assert np.all(np.abs(w - a) <= np.abs(a) * 2.0 ** -8)   # RNE to 8 mantissa bits


def test_combine_and_decomposition():
    d, f, n, k = 48, 40, 6, 3
    rng = np.random.default_rng(9)
    wr = (rng.standard_normal((n, d)) / math.sqrt(d)).astype(np.float32)
    slabs = [synth.expert_slab(100 + e, d, f, None) for e in range(n)]
    shared = synth.expert_slab(999, d, 56, None)
    for t in range(5):
        x = rng.standard_normal(d).astype(np.float32)
        idx, w, out, gap = oracle.moe_token(x, wr, slabs, k, f)
        ys = np.stack([oracle.expert(x, slabs[e], d, f) for e in idx])
        ref = (w.astype(np.float64)[:, None] * ys.astype(np.float64)).sum(0)
        assert np.allclose(out, ref, rtol=1e-6, atol=1e-7)
        # fp64 brute force of the whole layer (router from numpy logits)
        l = wr.astype(np.float64) @ x.astype(np.float64)
        order = sorted(range(n), key=lambda i: (-l[i], i))[:k]
        assert list(idx) == order
        p = np.exp(l[order] - l[order[0]])
        p /= p.sum()
        full = sum(p[j] * _np_expert(x, slabs[e], d, f) for j, e in enumerate(order))
        rms = math.sqrt(float(np.mean(full ** 2)))
        assert np.max(np.abs(out - full)) <= 1e-6 * rms
        # shared expert adds with weight 1
        idx2, w2, out2, _ = oracle.moe_token(x, wr, slabs, k, f, shared_slab=shared, f_shared=56)
        ysh = _np_expert(x, shared, d, 56)
        assert np.max(np.abs(out2 - (full + ysh))) <= 1e-6 * math.sqrt(float(np.mean((full + ysh) ** 2)))


def test_thread_count_independent():
    d, f = 128, 320
    slab = synth.expert_slab(3, d, f, None)
    x = np.random.default_rng(2).standard_normal(d).astype(np.float32)
    old = oracle.get_threads()
    try:
        oracle.set_threads(1)
        y1 = oracle.expert(x, slab, d, f)
        oracle.set_threads(4)
        y4 = oracle.expert(x, slab, d, f)
    finally:
        oracle.set_threads(old)
    assert np.array_equal(y1, y4)
