"""Pins of the oracle's fp64 attention, selection score and decode step.

* textbook routine: dense decoding equals fp64 ``scaled_dot_product_attention``
  on the CPU, and the diagonal mode with nothing skipped equals dense;
* closed forms: a zero query averages the attended value rows, a single key
  returns its value row, constant values return the constant, two keys give
  the logistic weights;
* invariants: the weights sum to one, permuting the keys does not change the
  output, attention split into two halves and merged by log-sum-exp equals a
  single pass, the window softmax sums to one per query head so the GQA score
  sums to the group size;
* selection: at group size 1 the argmin of the softmax is the argmin of the
  logits, ties go to the oldest key, identical queries in a group reduce to
  the single-head rule.
"""

import math

import numpy as np
import pytest
import torch

from oracle import attention, step


def rnd(*shape, seed=0):
    return np.random.default_rng(seed).standard_normal(shape)


def test_weights_sum_to_one_and_permutation_invariance():
    q, K, V = rnd(64, seed=1), rnd(37, 64, seed=2), rnd(37, 64, seed=3)
    out, w = attention.attend(q, K, V, 0.125)
    assert abs(w.sum() - 1.0) < 1e-12
    perm = np.random.default_rng(4).permutation(37)
    out2, _ = attention.attend(q, K[perm], V[perm], 0.125)
    np.testing.assert_allclose(out, out2, rtol=0, atol=1e-13)


def test_closed_forms():
    K, V = rnd(9, 16, seed=5), rnd(9, 16, seed=6)
    out, w = attention.attend(np.zeros(16), K, V, 0.25)
    np.testing.assert_allclose(out, V.mean(axis=0), atol=1e-14)
    out, _ = attention.attend(rnd(16, seed=7), K[:1], V[:1], 0.25)
    np.testing.assert_array_equal(out, V[0])
    out, _ = attention.attend(rnd(16, seed=8), K, np.ones((9, 16)), 0.25)
    np.testing.assert_allclose(out, 1.0, atol=1e-14)
    # two keys along the query: w1 = 1 / (1 + exp(s0 - s1))
    q = np.array([1.0, 0.0])
    K2 = np.array([[0.5, 3.0], [2.0, -1.0]])
    V2 = np.array([[1.0, 0.0], [0.0, 1.0]])
    out, w = attention.attend(q, K2, V2, 1.0)
    w1 = 1.0 / (1.0 + math.exp(0.5 - 2.0))
    np.testing.assert_allclose(w, [1 - w1, w1], atol=1e-15)
    np.testing.assert_allclose(out, [1 - w1, w1], atol=1e-15)


def test_split_merge_equals_single_pass():
    q, K, V = rnd(32, seed=9), rnd(50, 32, seed=10), rnd(50, 32, seed=11)
    scale = 1 / math.sqrt(32)
    full, _ = attention.attend(q, K, V, scale)
    parts = []
    for lo, hi in ((0, 17), (17, 50)):
        s = attention.logits(q, K[lo:hi], scale)
        m = s.max()
        e = np.exp(s - m)
        parts.append((m, e.sum(), e @ V[lo:hi]))
    M = max(p[0] for p in parts)
    num = sum(math.exp(m - M) * a for m, _, a in parts)
    den = sum(math.exp(m - M) * l for m, l, _ in parts)
    np.testing.assert_allclose(num / den, full, atol=1e-14)


@pytest.mark.parametrize("t", [0, 1, 5, 40])
def test_dense_step_matches_torch_sdpa(t):
    Hq, Hkv, d, Lp, L = 6, 3, 16, 5, 41
    q = rnd(Hq, d, seed=12)
    Kp, Vp = rnd(Hkv, Lp, d, seed=13), rnd(Hkv, Lp, d, seed=14)
    K, V = rnd(Hkv, L, d, seed=15), rnd(Hkv, L, d, seed=16)
    res = step.request_step(t, q, Kp, Vp, K, V, 1 / math.sqrt(d), mode="dense")
    g = Hq // Hkv
    keys = torch.from_numpy(np.concatenate([Kp, K[:, :t + 1]], axis=1)).repeat_interleave(g, 0)
    vals = torch.from_numpy(np.concatenate([Vp, V[:, :t + 1]], axis=1)).repeat_interleave(g, 0)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[:, None, :], keys, vals)[:, 0, :].numpy()
    np.testing.assert_allclose(res.out, ref, rtol=0, atol=1e-12)


def test_no_skip_diagonal_equals_dense():
    Hq, d, Lp, L = 4, 8, 3, 20
    rng = np.random.default_rng(17)
    Q = rng.standard_normal((L, Hq, d))
    Kp, Vp = rng.standard_normal((2, Hq, Lp, d))
    K, V = rng.standard_normal((2, Hq, L, d))
    diag = step.trajectory(Q, Kp, Vp, K, V, 0.3, N_r=L, N_att=L)
    dense = step.trajectory(Q, Kp, Vp, K, V, 0.3, N_r=L, N_att=L, mode="dense")
    for a, b in zip(diag, dense):
        np.testing.assert_array_equal(a.out, b.out)


def test_select_mha_is_argmin_of_logits_with_oldest_tie():
    rng = np.random.default_rng(18)
    for _ in range(50):
        q, K = rng.standard_normal(16), rng.standard_normal((23, 16))
        j, sigma = attention.select(q, K, 0.25)
        assert j == int(np.argmin(K @ q))
        assert abs(sigma.sum() - 1.0) < 1e-12
    # exact tie between keys 1 and 3 (identical rows): the older (1) wins
    K = np.array([[1.0, 0.0], [-1.0, 0.0], [0.5, 0.0], [-1.0, 0.0]])
    assert attention.select(np.array([1.0, 0.0]), K, 1.0)[0] == 1


def test_select_gqa_reductions():
    rng = np.random.default_rng(19)
    q, K = rng.standard_normal(16), rng.standard_normal((30, 16))
    j1, s1 = attention.select(q, K, 0.25)
    j4, s4 = attention.select(np.stack([q] * 4), K, 0.25)
    assert j1 == j4
    np.testing.assert_allclose(s4, 4 * s1, atol=1e-14)
    qg = rng.standard_normal((4, 16))
    _, sg = attention.select(qg, K, 0.25)
    assert abs(sg.sum() - 4.0) < 1e-12


def test_step_uses_group_kv_head_and_prompt():
    """Each query head reads KV head h // g; the prompt is always attended."""
    Hq, Hkv, d, Lp, L = 4, 2, 8, 2, 12
    rng = np.random.default_rng(20)
    q = rng.standard_normal((Hq, d))
    Kp, Vp = rng.standard_normal((2, Hkv, Lp, d))
    K, V = rng.standard_normal((2, Hkv, L, d))
    states = step.new_states(Hkv, 6, 2)
    for t in range(9):
        res = step.request_step(t, q, Kp, Vp, K, V, 0.5, states=states)
    for h in range(Hq):
        kvh = h // 2
        idx = res.heads[kvh].idx
        keys = np.concatenate([Kp[kvh], K[kvh][idx]])
        vals = np.concatenate([Vp[kvh], V[kvh][idx]])
        s = 0.5 * keys @ q[h]
        w = np.exp(s - s.max())
        np.testing.assert_allclose(res.out[h], (w / w.sum()) @ vals, atol=1e-13)
