"""Pins of the oracle's sink modes (section 5.1): Diagonal+Sink keeps the
first S decode tokens and runs Algorithm 1 on the later ones; StreamingLLM
keeps the S sinks plus the most recent tokens.  Sinks count against N_att.

* a small case of each mode worked by hand (fixture);
* closed forms: StreamingLLM is {0 .. S-1} plus the last N_att - S tokens,
  with S = 0 the sliding window;
* Diagonal+Sink with S = 0 is plain Algorithm 1 on every choice path;
* the attended decode count is min(t + 1, N_att) in every mode, the sinks
  are always kept once decoded, a selection never picks a sink, and the
  footprint is at most S + N_r decode rows;
* an independent offset formulation (the one the library's kernels use) on
  random choice paths.
"""

import itertools
import json
import os
import random

import pytest

from oracle import alg1
from oracle import step as ostep


def run_mode(mode, N_r, N_att, S, T, choose):
    st = ostep.new_states(1, N_r, N_att, mode, S)[0]
    return [ostep.kept_with_sinks(t, S, st, choose) for t in range(T)]


def oldest(t, idx):
    return 0


def test_hand_worked_example(golden_dir):
    with open(os.path.join(golden_dir, "sink_example.json")) as f:
        g = json.load(f)
    ds = g["diagonal_sink"]
    recs = run_mode("diagonal_sink", ds["N_r"], ds["N_att"], ds["sinks"], 8, oldest)
    for t, kept in ds["kept"].items():
        assert recs[int(t)].idx == kept, t
    sel = {str(r.t): r.selected for r in recs if r.selected is not None}
    assert sel == ds["selected"]
    sm = g["streaming"]
    recs = run_mode("streaming", 0, sm["N_att"], sm["sinks"], 10, None)
    for t, kept in sm["kept"].items():
        assert recs[int(t)].idx == kept, t
        assert recs[int(t)].selected is None


@pytest.mark.parametrize("S", [0, 1, 4])
def test_streaming_closed_form(S):
    for N_att in range(S + 1, S + 12):
        for r in run_mode("streaming", 0, N_att, S, 3 * N_att + 5, None):
            t = r.t
            want = sorted(set(range(min(S, t + 1))) | set(range(max(0, t - (N_att - S) + 1), t + 1)))
            assert r.idx == want
            assert r.selected is None


def test_streaming_without_sinks_is_sliding_window():
    for N_att in (1, 3, 9):
        for r in run_mode("streaming", 0, N_att, 0, 30, None):
            assert r.idx == list(range(max(0, r.t - N_att + 1), r.t + 1))


@pytest.mark.parametrize("N_r", range(1, 8))
def test_diagonal_sink_zero_is_algorithm_1(N_r):
    for N_att in range(1, N_r + 1):
        for path in itertools.product(range(N_att), repeat=N_r - N_att):
            T = 2 * N_r + 3
            plain = alg1.run(N_r, N_att, T, alg1.scripted(path))
            sink0 = run_mode("diagonal_sink", N_r, N_att, 0, T, alg1.scripted(path))
            assert [r.idx for r in plain] == [r.idx for r in sink0]
            assert [r.selected for r in plain] == [r.selected for r in sink0]


def offset_form_sinks(N_r, N_att, S, T, choose):
    """Independent formulation: sinks, then the window offsets
    0 .. min(t - S, N_r - 1) minus the first n stored offsets, where
    n = clamp(t - N_att + 1, 0, N_r - N_att + S); a selecting step stores
    t - idx[j*] over the kept window keys (sinks excluded)."""
    D = []
    out = []
    for t in range(T):
        n = min(max(t - N_att + 1, 0), N_r - N_att + S)
        skip = set(D[:n])
        win = [t - d for d in range(min(t - S, N_r - 1), -1, -1) if d not in skip]
        kept = list(range(min(S, t + 1))) + win
        sel = None
        if N_att - 1 <= t <= N_r + S - 2:
            j = choose(t, list(win))
            sel = win[j]
            D.append(t - sel)
        out.append((kept, sel))
    return out


@pytest.mark.parametrize("S", [1, 2, 4])
def test_diagonal_sink_offset_form(S):
    rng = random.Random(77 + S)
    for N_r in range(1, 10):
        for N_att in range(S + 1, S + N_r + 1):
            for rep in range(12):
                seq = [rng.randrange(1 << 30) for _ in range(N_r + S)]
                T = 2 * (N_r + S) + 5
                lit = run_mode("diagonal_sink", N_r, N_att, S, T, alg1.uniform(seq))
                off = offset_form_sinks(N_r, N_att, S, T, alg1.uniform(seq))
                for r, (kept, sel) in zip(lit, off):
                    assert r.idx == kept, (N_r, N_att, S, r.t)
                    assert r.selected == sel


@pytest.mark.parametrize("mode", ["diagonal_sink", "streaming"])
def test_counts_sinks_and_footprint(mode):
    rng = random.Random(5)
    for S in (1, 4):
        for N_r in (3, 8, 13):
            for N_att in range(S + 1, S + N_r + 1):
                seq = [rng.randrange(1 << 30) for _ in range(64)]
                for r in run_mode(mode, N_r, N_att, S, 3 * (N_r + S), alg1.uniform(seq)):
                    t = r.t
                    assert len(r.idx) == min(t + 1, N_att)
                    assert r.idx == sorted(set(r.idx))
                    assert set(range(min(S, t + 1))) <= set(r.idx)
                    assert r.selected is None or r.selected >= S
                    span = N_r if mode == "diagonal_sink" else N_att - S
                    assert all(j < S or j > t - span for j in r.idx)
