"""Pins of the oracle's Algorithm 1 (section 4) against facts fixed outside it.

* the worked example the paper prints (N_r = 7, N_att = 4), as a fixture;
* the counts the paper states: the attended decode count grows to N_att and
  then stays there, the skip list grows by one per step up to N_r - N_att,
  the footprint never exceeds N_r decode rows;
* the special cases that reduce to textbook rules: N_att = N_r is a sliding
  window over the last N_r decode tokens, N_att = N_r >= L_dec is dense
  causal attention;
* brute force on tiny inputs: every possible choice path for small N_r, and
  an independent formulation (relative offsets, which never change because a
  skip entry and t both advance by one per step) on random paths.
"""

import itertools
import json
import os
import random

import pytest

from oracle import alg1


def offset_form(N_r, N_att, T, choose):
    """Independent formulation: a set of offsets d = t - j.  The window is
    offsets 0 .. min(t, N_r - 1); a phase-2 step adds t - idx[j*]."""
    D = []
    out = []
    for t in range(T):
        kept = [t - d for d in range(min(t, N_r - 1), -1, -1) if d not in D]
        sel = None
        if N_att - 1 <= t < N_r and len(D) < N_r - N_att:
            j = choose(t, list(kept))
            sel = kept[j]
            D.append(t - sel)
        out.append((kept, sel))
    return out


def test_worked_example(golden_dir):
    fx = json.load(open(os.path.join(golden_dir, "worked_example.json")))
    N_r, N_att = fx["N_r"], fx["N_att"]
    # the paper names the choices at t=3 and t=4; t=5 picks the oldest kept key
    picks = {3: fx["steps"]["3"]["choose_position"], 4: fx["steps"]["4"]["choose_position"], 5: 0}
    st = alg1.HeadState(N_r, N_att)
    recs = [st.step(t, alg1.by_position(picks)) for t in range(12)]
    for t in fx["phase1_steps"]:
        assert recs[t].phase == 1 and recs[t].idx == list(range(t + 1))
    for key, want in fx["steps"].items():
        r = recs[int(key)]
        assert r.phase == 2
        assert r.idx == want["idx"]
        assert r.skip_idx == want["skip_before_append"]
        if "choose_position" in want:
            assert r.selected == want["choose_position"]
    assert max(len(r.skip_idx) + (r.selected is not None) for r in recs) == fx["max_skip_len"]
    assert recs[7].phase == 3 and fx["evict_at_t7"] in st.evicted
    assert fx["evict_at_t7"] not in recs[7].idx
    for r in recs[7:]:
        assert len(r.idx) == fx["attended_count_phase3"]


def _random_chooser(rng):
    return lambda t, idx: rng.randrange(len(idx))


@pytest.mark.parametrize("N_r", range(1, 13))
def test_counts_and_footprint(N_r):
    rng = random.Random(N_r)
    for N_att in range(1, N_r + 1):
        for _ in range(20):
            T = 3 * N_r + 5
            st = alg1.HeadState(N_r, N_att)
            for t in range(T):
                r = st.step(t, _random_chooser(rng))
                # attended decode count: min(t + 1, N_att) in every phase
                assert len(r.idx) == min(t + 1, N_att)
                assert r.idx == sorted(set(r.idx))
                # the skip list grows one per phase-2 step, up to N_r - N_att
                assert len(st.skip_idx) == max(0, min(t - N_att + 2, N_r - N_att))
                # kept rows lie in the live window: footprint <= N_r decode rows
                assert all(max(0, t - N_r + 1) <= j <= t for j in r.idx)
                # the oldest live row is never a skip target (its offset is N_r - 1)
                if t >= N_r - 1:
                    assert (t - N_r + 1) not in st.skip_idx
                # skip entries stay inside the live window, never evicted rows
                assert all(t - N_r + 1 <= j <= t for j in st.skip_idx)


@pytest.mark.parametrize("N_r", range(1, 11))
def test_offset_form_matches_literal_random_paths(N_r):
    rng = random.Random(1000 + N_r)
    for N_att in range(1, N_r + 1):
        for rep in range(30):
            seq = [rng.randrange(1 << 30) for _ in range(N_r)]
            T = 2 * N_r + 7
            lit = alg1.run(N_r, N_att, T, alg1.uniform(seq))
            off = offset_form(N_r, N_att, T, alg1.uniform(seq))
            for r, (kept, sel) in zip(lit, off):
                assert r.idx == kept
                assert r.selected == sel


@pytest.mark.parametrize("N_r", range(1, 8))
def test_offset_form_matches_literal_every_path(N_r):
    """Exhaustive over all choice paths for N_r <= 7."""
    for N_att in range(1, N_r + 1):
        n_sel = N_r - N_att
        T = 2 * N_r + 3
        for path in itertools.product(range(N_att), repeat=n_sel):
            lit = alg1.run(N_r, N_att, T, alg1.scripted(path))
            off = offset_form(N_r, N_att, T, alg1.scripted(path))
            assert [r.idx for r in lit] == [k for k, _ in off]


@pytest.mark.parametrize("N_r", [1, 2, 5, 16])
def test_sliding_window_special_case(N_r):
    """N_att = N_r never selects: the kept set is the last N_r decode tokens."""
    for r in alg1.run(N_r, N_r, 4 * N_r, None):
        assert r.selected is None
        assert r.idx == list(range(max(0, r.t - N_r + 1), r.t + 1))


@pytest.mark.parametrize("L_dec", [1, 7, 33])
def test_dense_special_case(L_dec):
    """N_att = N_r >= L_dec: every step attends all decode tokens 0 .. t."""
    N_r = L_dec + 3
    for r in alg1.run(N_r, N_r, L_dec, None):
        assert r.idx == list(range(r.t + 1))


def test_phase_boundaries():
    st = alg1.HeadState(10, 4)
    phases = [st.step(t, lambda t, idx: 0).phase for t in range(15)]
    assert phases == [1, 1, 1] + [2] * 7 + [3] * 5
    # selections happen at t = N_att - 1 .. N_r - 2 only
    st = alg1.HeadState(10, 4)
    sel = [t for t in range(15) if st.step(t, lambda t, idx: 0).selected is not None]
    assert sel == list(range(3, 9))


def test_invalid_parameters():
    with pytest.raises(ValueError):
        alg1.HeadState(4, 5)
    with pytest.raises(ValueError):
        alg1.HeadState(4, 0)


@pytest.mark.parametrize("N_r", [2, 3, 6, 11, 24])
def test_next_kept_offsets_follow_from_the_selection(N_r):
    """The property the selection state's kept lists rest on, on the literal
    Algorithm 1: after a phase-2 selection at step t (k entries before it),
    the kept offsets of step t + 1, oldest first, are the new oldest offset
    N_att + k followed by step t's kept offsets without the selected one;
    once the selections are over, the kept offsets stay the same."""
    rng = random.Random(77 + N_r)
    for N_att in range(1, N_r + 1):
        for rep in range(10):
            T = 2 * N_r + 5
            recs = alg1.run(N_r, N_att, T, alg1.uniform([rng.randrange(1 << 30) for _ in range(N_r)]))
            for a, b in zip(recs, recs[1:]):
                t = a.t
                offs_t = [t - j for j in a.idx]
                offs_next = [t + 1 - j for j in b.idx]
                if a.selected is not None:
                    k = t - (N_att - 1)
                    assert offs_next == [N_att + k] + [d for d in offs_t if d != t - a.selected]
                elif t >= N_r - 1:
                    assert offs_next == offs_t
