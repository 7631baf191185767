"""Pins of the C oracle (``oracle/c/dsa_oracle.c``) to the Python oracle and
to the paper's worked example (section 4, "Detailed explanation").

* the worked example (N_r = 7, N_att = 4) replayed through the C Algorithm 1;
* the C Algorithm 1 equals the Python one on every (N_r, N_att) up to 10,
  over random choice paths and every stopping step, and on a long window;
* one decode step of a request (attention of every query head, the window
  softmax selection) equals the Python step: outputs within fp64 rounding,
  the same picks and the same states afterwards, in diagonal and dense mode,
  at group sizes 1, 2 and 4, with any number of threads.
"""

import copy
import json
import os
import random

import numpy as np
import pytest

from oracle import alg1, coracle, step as ostep


def test_worked_example_c(golden_dir):
    fx = json.load(open(os.path.join(golden_dir, "worked_example.json")))
    N_r, N_att, L = fx["N_r"], fx["N_att"], 12
    # the paper's picks: K_0 at t = 3 (index 0 of [0,1,2,3]), K_2 at t = 4
    # (index 1 of [0,2,3,4]); t = 5 picks its oldest kept key
    rand = [0, 1, 0]
    for key, want in fx["steps"].items():
        t = int(key)
        skip, idx = coracle.alg1_replay(N_r, N_att, L, t, rand)
        assert idx == want["idx"]
        assert skip == want["skip_before_append"]
    for t in range(N_r, L):
        skip, idx = coracle.alg1_replay(N_r, N_att, L, t, rand)
        assert len(idx) == fx["attended_count_phase3"]
        assert len(skip) == fx["max_skip_len"]
        assert fx["evict_at_t7"] not in idx and min(idx) >= t - N_r + 1
    for t in fx["phase1_steps"]:
        assert coracle.alg1_replay(N_r, N_att, L, t, rand) == ([], list(range(t + 1)))


@pytest.mark.parametrize("N_r", range(1, 11))
def test_c_alg1_equals_python(N_r):
    rng = random.Random(N_r)
    L = 2 * N_r + 3
    for N_att in range(1, N_r + 1):
        for _ in range(4):
            rand = [rng.randrange(1 << 40) for _ in range(N_r)]
            for t_end in range(L):
                st = alg1.HeadState(N_r, N_att)
                ch = alg1.uniform(rand)
                for t in range(t_end):
                    st.step(t, ch)
                rec = st.step(t_end, lambda t_, i_: 0)
                skip, idx = coracle.alg1_replay(N_r, N_att, L, t_end, rand)
                assert idx == rec.idx, (N_r, N_att, t_end)
                assert skip == rec.skip_idx, (N_r, N_att, t_end)


def test_c_alg1_long_window():
    rng = random.Random(5)
    N_r, N_att, L = 300, 37, 700
    rand = [rng.randrange(1 << 40) for _ in range(N_r)]
    for t_end in (N_att - 2, N_att - 1, 150, N_r - 2, N_r - 1, N_r, 699):
        st = alg1.HeadState(N_r, N_att)
        ch = alg1.uniform(rand)
        for t in range(t_end):
            st.step(t, ch)
        rec = st.step(t_end, lambda t_, i_: 0)
        assert coracle.alg1_replay(N_r, N_att, L, t_end, rand) == (rec.skip_idx, rec.idx)


def test_c_alg1_rejects_short_random_stream():
    with pytest.raises(ValueError):
        coracle.alg1_replay(8, 3, 20, 10, [1, 2])


@pytest.mark.parametrize("g", [1, 2, 4])
def test_c_request_step_equals_python(g):
    rng = np.random.default_rng(g)
    Hkv, d, Lp, N_r, N_att, L = 3, 16, 5, 12, 4, 30
    Hq = Hkv * g
    Kp, Vp = rng.standard_normal((2, Hkv, Lp, d))
    K, V = rng.standard_normal((2, Hkv, L, d))
    Q = rng.standard_normal((L, Hq, d))
    scale = 0.25
    py_states = ostep.new_states(Hkv, N_r, N_att)
    c_states = coracle.States.from_heads(py_states, L)
    for t in range(L):
        res = ostep.request_step(t, Q[t], Kp, Vp, K, V, scale, "diagonal", py_states)
        out, picked = coracle.request_step(t, Q[t], Kp, Vp, K, V, scale, "diagonal", c_states)
        assert np.abs(out - res.out).max() <= 1e-12 * np.abs(res.out).max()
        for h in range(Hkv):
            sel = res.heads[h].selected
            assert picked[h] == (-1 if sel is None else sel), (t, h)
            assert c_states.skip[h, :c_states.n_skip[h]].tolist() == py_states[h].skip_idx
        dres = ostep.request_step(t, Q[t], Kp, Vp, K, V, scale, "dense")
        dout, _ = coracle.request_step(t, Q[t], Kp, Vp, K, V, scale, "dense")
        assert np.abs(dout - dres.out).max() <= 1e-12 * np.abs(dres.out).max()


def test_c_request_step_threads_and_empty_prompt():
    rng = np.random.default_rng(3)
    Hkv, g, d, N_r, N_att, L = 8, 2, 32, 20, 6, 40
    Kp = Vp = np.zeros((Hkv, 0, d))
    K, V = rng.standard_normal((2, Hkv, L, d))
    q = rng.standard_normal((Hkv * g, d))
    heads = ostep.random_states(Hkv, N_r, N_att, 17, list(rng.integers(0, 1 << 30, 200)))
    base = coracle.States.from_heads(heads, L)
    outs = []
    for th in (1, 3, 8):
        st = base.copy()
        outs.append((coracle.request_step(17, q, Kp, Vp, K, V, 0.2, "diagonal", st, threads=th), st))
    for (o, p), st in outs[1:]:
        assert np.array_equal(o, outs[0][0][0]) and np.array_equal(p, outs[0][0][1])
        assert np.array_equal(st.skip, outs[0][1].skip)
    res = ostep.request_step(17, q, Kp, Vp, K, V, 0.2, "diagonal", copy.deepcopy(heads))
    assert np.abs(outs[0][0][0] - res.out).max() <= 1e-12 * np.abs(res.out).max()


def test_replay_head_is_the_state_before_the_step():
    rng = random.Random(9)
    for N_r, N_att, L in ((7, 4, 20), (12, 3, 40), (30, 30, 70)):
        for t in range(L):
            rand = [rng.randrange(1 << 40) for _ in range(N_r)]
            st, kept = coracle.replay_head(N_r, N_att, L, t, rand)
            ref = alg1.HeadState(N_r, N_att)
            ch = alg1.uniform(rand)
            for u in range(t):
                ref.step(u, ch)
            assert st.skip_idx == ref.skip_idx and st.evicted == ref.evicted, (N_r, N_att, t)
            assert ref.step(t, lambda t_, i_: 0).idx == kept
