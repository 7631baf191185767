"""Pins of the fp32 rounding bounds in ``oracle/tieband.py``.

The bound is pinned by the arithmetic it bounds, simulated independently in
numpy float32: dot products of bf16 values accumulated in random orders,
the scale multiply, the window softmax in base 2 with the fp32 constant
log2(e), the fp32 sums, the reciprocal and the weight products.  For every
window key the simulated fp32 score must lie within the bound of the exact
fp64 score, also when every logit is pushed to the edge of its own error
bound; the bound must stay small (a band that accepts everything would pin
nothing); and the tie test must accept exactly the picks inside it.
"""

import numpy as np
import pytest

from oracle import tieband


def bf16(x):
    """Round fp64 values to bf16 (nearest even) and return them as fp64."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def f32_seq_sum(x, rng, axis=-1):
    """fp32 sum along ``axis`` in a random order, one rounding per add."""
    x = np.moveaxis(np.asarray(x, np.float32), axis, -1)
    perm = rng.permutation(x.shape[-1])
    return np.cumsum(x[..., perm], axis=-1, dtype=np.float32)[..., -1]


def simulate(q_group, keys, scale, rng, push=None):
    """fp32 scores of the window keys as the device computes them.
    ``push`` (None, or +-1 per key) moves each fp32 logit by two thirds of
    its error bound before the softmax (the fp32 rounding of the moved
    value, at most u |s|, adds at most the last third)."""
    qg = np.atleast_2d(q_group)
    prods = qg.astype(np.float32)[:, None, :] * keys.astype(np.float32)[None, :, :]
    dots = f32_seq_sum(prods, rng)
    s = (dots * np.float32(scale)).astype(np.float32)
    if push is not None:
        for h in range(qg.shape[0]):
            band = tieband.logit_band(qg[h], keys, scale)
            s[h] = (s[h].astype(np.float64) + push[h] * band * (2 / 3)).astype(np.float32)
    if qg.shape[0] == 1:
        return s[0].astype(np.float64)
    L2E = np.float32(1.4426950408889634)
    m = s.max(axis=1, keepdims=True)
    e = np.exp2((L2E * (s - m).astype(np.float32)).astype(np.float32)).astype(np.float32)
    Z = f32_seq_sum(e, rng)
    inv = (np.float32(1.0) / Z).astype(np.float32)
    w = (e * inv[:, None]).astype(np.float32)
    return f32_seq_sum(w, rng, axis=0).astype(np.float64)


CASES = [(1, 64, 40), (1, 128, 300), (2, 128, 29), (4, 128, 205), (4, 64, 400), (8, 128, 97)]


@pytest.mark.parametrize("g,d,n", CASES)
def test_bound_holds_on_simulated_fp32(g, d, n):
    rng = np.random.default_rng(g * 1000 + n)
    worst = 0.0
    for trial in range(6):
        q = bf16(rng.standard_normal((g, d)))
        keys = rng.standard_normal((n, d))
        if trial % 2:  # outlier keys (x8), as in the Emu3-like workload
            keys[rng.random(n) < 0.05] *= 8
        keys = bf16(keys)
        scale = 1 / np.sqrt(d)
        exact, err = tieband.score_bounds(q, keys, scale)
        for push in ((None,) if g == 1 else (None, 1.0, -1.0)):
            pv = None if push is None else [push * np.where(rng.random(n) < 0.5, 1, -1)
                                           for _ in range(g)]
            got = simulate(q, keys, scale, rng, pv)
            dev = np.abs(got - exact)
            assert (dev <= err).all(), (trial, push, (dev / err).max())
            worst = max(worst, (dev / err).max())
        # the bound is not vacuous (the worst-case dot-product term
        # gamma_d * sum |q_i k_i| dominates it): below 0.1% of the largest
        # logit for one query head, below 1% of each key's own score for a
        # group
        if g == 1:
            assert err.max() <= 1e-3 * np.abs(exact).max()
        else:
            assert (err <= 1e-2 * exact).all()
    assert worst > 1e-3  # the simulated errors come within reach of the bound


def test_tie_decisions():
    rng = np.random.default_rng(11)
    d, n = 128, 50
    scale = 1 / np.sqrt(d)
    for g in (1, 4):
        q = bf16(rng.standard_normal((g, d)))
        keys = bf16(rng.standard_normal((n, d)))
        score, err = tieband.score_bounds(q, keys, scale)
        j_ref = int(np.argmin(score))
        assert tieband.within_tie_band(q, keys, scale, j_ref, j_ref)
        order = np.argsort(score)
        j2 = int(order[1])
        gap = score[j2] - score[j_ref]
        inside = gap <= err[j2] + err[j_ref]
        assert tieband.within_tie_band(q, keys, scale, j2, j_ref) == inside
        # a key clearly above the minimum is rejected
        j_far = int(order[-1])
        assert not tieband.within_tie_band(q, keys, scale, j_far, j_ref)
        assert not tieband.within_tie_band(q, keys, scale, n + 3, j_ref)
    # an exact duplicate of the minimum key is a tie either way
    q = bf16(rng.standard_normal((2, d)))
    keys = bf16(rng.standard_normal((10, d)))
    score, _ = tieband.score_bounds(q, keys, scale)
    j = int(np.argmin(score))
    keys2 = np.concatenate([keys, keys[j:j + 1]])
    assert tieband.within_tie_band(q, keys2, scale, 10, j)
    assert tieband.within_tie_band(q, keys2, scale, j, 10)
