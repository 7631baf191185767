"""ctypes access to the C oracle (``oracle/c/dsa_oracle.c``), built with gcc.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

The C oracle restates Algorithm 1 and the fp64 decode step of
``oracle.alg1`` / ``oracle.step`` in plain C so that long selection
histories and whole requests run in seconds; ``tests/test_oracle_c.py`` pins
it to the Python oracle and to the paper's worked example.  ``build()``
compiles it (``__graft_entry__.build()`` calls it); ``lib()`` loads it.
"""

from __future__ import annotations

import ctypes as C
import os
import shutil
import subprocess
from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "c", "dsa_oracle.c")
LIB_PATH = os.path.join(_HERE, "libdsa_oracle.so")

_lib = None


def build(verbose: bool = False) -> str:
    """Compile the C oracle into ``oracle/libdsa_oracle.so``."""
    cc = shutil.which("gcc") or "gcc"
    tmp = LIB_PATH + ".tmp"
    cmd = [cc, "-O2", "-std=c11", "-fopenmp", "-shared", "-fPIC", "-fvisibility=hidden",
           "-Wall", "-o", tmp, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"C oracle build failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = C.CDLL(LIB_PATH)
        P = C.c_void_p
        L.orc_alg1_replay.restype = C.c_int
        L.orc_alg1_replay.argtypes = [C.c_int32] * 4 + [P, C.c_int64, P, P, P, P, P]
        L.orc_request_step.restype = C.c_int
        L.orc_request_step.argtypes = [P, C.c_int32, P, P, P, P, P, C.c_int32, C.c_double,
                                       P, P, P, P, P, C.c_int32]
        _lib = L
    return _lib


def _p(a: np.ndarray) -> int:
    return a.ctypes.data


def alg1_replay(N_r: int, N_att: int, L: int, t_end: int,
                rand: Sequence[int]) -> Tuple[List[int], List[int]]:
    """Algorithm 1 of one head over steps ``0 .. t_end - 1`` with the k-th
    choice ``rand[k] mod |idx|``, then step ``t_end`` without a choice.
    Returns ``(skip_idx used at t_end, kept positions at t_end)``."""
    r = np.ascontiguousarray(np.asarray(rand, dtype=np.int64))
    skip = np.zeros(max(N_r - N_att, 1), dtype=np.int32)
    ns = np.zeros(1, dtype=np.int32)
    ev = np.zeros(L, dtype=np.uint8)
    idx = np.zeros(N_r + 1, dtype=np.int32)
    ni = np.zeros(1, dtype=np.int32)
    st = lib().orc_alg1_replay(N_r, N_att, L, t_end, _p(r), len(r), _p(skip), _p(ns), _p(ev),
                               _p(idx), _p(ni))
    if st != 0:
        raise ValueError(f"orc_alg1_replay failed ({st})")
    return skip[:ns[0]].tolist(), idx[:ni[0]].tolist()


def replay_head(N_r: int, N_att: int, L: int, t: int, rand: Sequence[int]):
    """Algorithm 1 state of one head before step ``t`` (after steps
    ``0 .. t-1`` with the k-th choice ``rand[k] mod |idx|``) as an
    ``oracle.alg1.HeadState``, plus the positions step ``t`` attends.  The
    C replay also runs step ``t`` (without a choice); the state before it is
    its skip list one position back along each diagonal when step ``t``
    shifted it (phase 2 or 3), and the positions evicted at steps before
    ``t`` (``t' - N_r`` for ``N_r <= t' < t``)."""
    from . import alg1
    skip_used, kept = alg1_replay(N_r, N_att, L, t, rand)
    st = alg1.HeadState(N_r, N_att)
    st.skip_idx = [j - 1 for j in skip_used] if st.phase(t) >= 2 else list(skip_used)
    st.evicted = set(range(0, max(0, t - N_r)))
    return st, kept


@dataclass
class States:
    """Algorithm 1 states of the KV heads of one request, in the C oracle's
    arrays: ``skip[h, :n_skip[h]]`` absolute positions, ``evicted[h, j]``."""
    N_r: int
    N_att: int
    L: int
    skip: np.ndarray
    n_skip: np.ndarray
    evicted: np.ndarray

    @classmethod
    def empty(cls, Hkv: int, N_r: int, N_att: int, L: int) -> "States":
        return cls(N_r, N_att, L, np.zeros((Hkv, max(N_r - N_att, 1)), np.int32),
                   np.zeros(Hkv, np.int32), np.zeros((Hkv, L), np.uint8))

    @classmethod
    def from_heads(cls, heads, L: int) -> "States":
        """From ``oracle.alg1.HeadState`` objects."""
        s = cls.empty(len(heads), heads[0].N_r, heads[0].N_att, L)
        for h, hs in enumerate(heads):
            s.n_skip[h] = len(hs.skip_idx)
            s.skip[h, :len(hs.skip_idx)] = hs.skip_idx
            for j in hs.evicted:
                s.evicted[h, j] = 1
        return s

    def copy(self) -> "States":
        return States(self.N_r, self.N_att, self.L, self.skip.copy(), self.n_skip.copy(),
                      self.evicted.copy())


def request_step(t: int, q, Kp, Vp, K, V, scale: float, mode: str = "diagonal",
                 states: Optional[States] = None, L: Optional[int] = None,
                 threads: int = 1):
    """One decode step of one request (all KV heads) in the C oracle.
    Arrays as ``oracle.step.request_step``; ``states`` is updated in place.
    Returns ``(out [Hq, d], picked [Hkv])`` with ``picked[h] = -1`` where
    head ``h`` added no skip entry."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    Kp = np.ascontiguousarray(Kp, dtype=np.float64)
    Vp = np.ascontiguousarray(Vp, dtype=np.float64)
    K = np.ascontiguousarray(K, dtype=np.float64)
    V = np.ascontiguousarray(V, dtype=np.float64)
    Hq, d = q.shape
    Hkv, Lp = Kp.shape[0], Kp.shape[1]
    rows = K.shape[1]
    if mode == "dense":
        Ltot = L if L is not None else rows
        st = States.empty(Hkv, 1, 1, Ltot)
        m = 0
    elif mode == "diagonal":
        st = states
        m = 1
    else:
        raise ValueError(f"unknown mode {mode!r}")
    dims = np.array([Hq, Hkv, d, Lp, st.N_r, st.N_att, st.L, m], dtype=np.int32)
    out = np.zeros((Hq, d), np.float64)
    picked = np.full(Hkv, -1, np.int32)
    if Lp == 0:  # a valid pointer for an empty prompt
        Kp = Vp = np.zeros((Hkv, 1, d), np.float64)
    rc = lib().orc_request_step(_p(dims), t, _p(q), _p(Kp), _p(Vp), _p(K), _p(V), rows,
                                float(scale), _p(st.skip), _p(st.n_skip), _p(st.evicted),
                                _p(out), _p(picked), int(threads))
    if rc != 0:
        raise ValueError(f"orc_request_step failed ({rc})")
    return out, picked
