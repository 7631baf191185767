"""One decode step of one request, and whole decode trajectories, in fp64.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

For every KV head of a request this runs Algorithm 1 (section 4) with the
attention-derived argmin of ``oracle.attention.select`` (or one of the sink
modes of section 5.1, see ``kept_with_sinks``) and computes
``Attn(Q_t, K_p + K[idx], V_p + V[idx])`` for each query head that reads
that KV head.  Dense mode ("no sparsity", the baseline of section 5) attends
``K_p`` plus every decode row ``0 .. t``.

Arrays (float64, or anything ``numpy.asarray`` turns into float64):

* ``q``       ``[Hq, d]``       the step's queries
* ``Kp, Vp``  ``[Hkv, L_p, d]`` prompt KV
* ``K, V``    ``[Hkv, n, d]``   decode KV; row ``j`` is decode position ``j``
                               and rows ``0 .. t`` must be present

Query head ``h`` reads KV head ``h // (Hq / Hkv)``.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, List, Optional

import numpy as np

from . import alg1, attention

# decide(kvh, t, idx, j_oracle, sigma) -> j used for the append.  The default
# keeps the oracle's own argmin; tests may substitute another valid choice.
Decider = Callable[[int, int, List[int], int, np.ndarray], int]


@dataclass
class HeadResult:
    idx: List[int]                 # kept decode positions (ascending)
    phase: int
    selected: Optional[int]        # position appended to skip_idx, or None
    j_oracle: Optional[int]        # the oracle's own argmin (index into idx)
    sigma: Optional[np.ndarray]    # selection score per kept window key
    window_logits: np.ndarray      # [g, len(idx)] scale * q.k over the window


@dataclass
class StepResult:
    out: np.ndarray                # [Hq, d]
    heads: List[HeadResult]        # one per KV head


SINK_MODES = ("streaming", "diagonal_sink")


def new_states(num_kv_heads: int, N_r: int, N_att: int, mode: str = "diagonal",
               sinks: int = 0) -> List[alg1.HeadState]:
    """Per-KV-head Algorithm 1 states.  In the sink modes the algorithm runs
    on the decode stream after the ``sinks`` first tokens: Diagonal+Sink
    with window ``N_r`` and ``N_att - sinks`` tokens to attend, StreamingLLM
    as a plain recent window of ``N_att - sinks`` tokens (``N_att = N_r``
    never skips)."""
    if mode == "diagonal_sink":
        N_r, N_att = N_r, N_att - sinks
    elif mode == "streaming":
        N_r = N_att = N_att - sinks
    return [alg1.HeadState(N_r, N_att) for _ in range(num_kv_heads)]


def kept_with_sinks(t: int, sinks: int, state: alg1.HeadState, choose) -> alg1.StepRecord:
    """The sink modes of section 5.1 ("Diagonal+Sink4" and the StreamingLLM
    baseline): decode tokens ``0 .. sinks-1`` are always attended; the other
    slots follow Algorithm 1 on the stream of later tokens, whose step
    ``t - sinks`` sees positions shifted down by ``sinks``."""
    if t < sinks:
        return alg1.StepRecord(t=t, phase=1, window=list(range(t + 1)), skip_idx=[],
                               idx=list(range(t + 1)), selected=None)
    shifted = None if choose is None else (lambda t_, idx_: choose(t_ + sinks, [j + sinks for j in idx_]))
    rec = state.step(t - sinks, shifted)
    rec.idx = list(range(sinks)) + [j + sinks for j in rec.idx]
    rec.selected = None if rec.selected is None else rec.selected + sinks
    rec.t = t
    return rec


def request_step(t: int, q, Kp, Vp, K, V, scale: float, mode: str = "diagonal",
                 states: Optional[List[alg1.HeadState]] = None,
                 decide: Optional[Decider] = None, sinks: int = 0) -> StepResult:
    q = np.asarray(q, dtype=np.float64)
    Hq, d = q.shape
    Hkv = len(Kp)
    if Hq % Hkv:
        raise ValueError("query heads must be a multiple of KV heads")
    g = Hq // Hkv
    out = np.zeros((Hq, d))
    heads: List[HeadResult] = []
    for kvh in range(Hkv):
        qg = q[kvh * g:(kvh + 1) * g]
        Kd = np.asarray(K[kvh], dtype=np.float64)
        note = {"j": None, "sigma": None}
        if mode == "dense":
            idx, phase, selected = list(range(t + 1)), 0, None
        elif mode == "diagonal" or mode in SINK_MODES:
            def choose(t_, idx_, kvh=kvh, qg=qg, Kd=Kd, note=note):
                j, sigma = attention.select(qg, Kd[idx_], scale)
                note["j"], note["sigma"] = j, sigma
                return j if decide is None else decide(kvh, t_, idx_, j, sigma)
            if mode == "diagonal":
                rec = states[kvh].step(t, choose)
            else:
                rec = kept_with_sinks(t, sinks, states[kvh], choose)
            idx, phase, selected = rec.idx, rec.phase, rec.selected
        else:
            raise ValueError(f"unknown mode {mode!r}")
        keys = np.concatenate([np.asarray(Kp[kvh], np.float64), Kd[idx]], axis=0)
        vals = np.concatenate([np.asarray(Vp[kvh], np.float64),
                               np.asarray(V[kvh], np.float64)[idx]], axis=0)
        for i in range(g):
            out[kvh * g + i] = attention.attend(qg[i], keys, vals, scale)[0]
        wl = np.stack([attention.logits(qg[i], Kd[idx], scale) for i in range(g)])
        heads.append(HeadResult(idx=idx, phase=phase, selected=selected,
                                j_oracle=note["j"], sigma=note["sigma"], window_logits=wl))
    return StepResult(out=out, heads=heads)


def trajectory(Q, Kp, Vp, K, V, scale: float, N_r: int, N_att: int, mode: str = "diagonal",
               steps: Optional[int] = None, decide: Optional[Decider] = None,
               sinks: int = 0) -> List[StepResult]:
    """All steps ``t = 0 .. steps-1`` of one request; ``Q[t]`` is ``[Hq, d]``."""
    T = len(Q) if steps is None else steps
    states = new_states(len(Kp), N_r, N_att, mode, sinks) if mode != "dense" else None
    return [request_step(t, Q[t], Kp, Vp, K, V, scale, mode, states, decide, sinks)
            for t in range(T)]


def random_states(num_kv_heads: int, N_r: int, N_att: int, t_end: int,
                  random_ints, mode: str = "diagonal", sinks: int = 0) -> List[alg1.HeadState]:
    """Selection states after steps ``0 .. t_end-1`` with the argmin replaced
    by externally drawn random choices (``random_ints``, one per selection,
    consumed head by head)."""
    it = iter(random_ints)
    states = new_states(num_kv_heads, N_r, N_att, mode, sinks)
    shift = sinks if mode in SINK_MODES else 0
    for st in states:
        for t in range(shift, t_end):
            st.step(t - shift, lambda t_, idx_: int(next(it)) % len(idx_))
    return states
