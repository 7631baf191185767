"""Algorithm 1 (section 4) -- the selection state of one attention head.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

The state is exactly the algorithm's: a list ``skip_idx`` of absolute decode
positions, shifted by +1 at every phase-2 and phase-3 step, and the set of
decode positions whose KV has been evicted.  No reformulation (offsets,
bitmaps) is used here; the tests compare this literal form against other
formulations.

Readings of the paper taken here:

* Phase boundaries follow the algorithm box: phase 1 while ``t < N_att-1``,
  phase 2 while ``t < N_r``, phase 3 afterwards.  The prose sentence that
  says phase 2 starts at ``t >= N_att`` is outvoted by the box and by the
  worked example, where the first selection happens at ``t = 3`` with
  ``N_att = 4``.
* ``window = [max(0, t-N_r), ..., t]`` is inclusive and contains the current
  token ``t``; in phase 3 the entry ``K[t-N_r]`` is evicted in the same step,
  so it is never attended (the attended count then stays at ``N_att``).
* The entry appended at a phase-2 step is not skipped at that step: the
  append happens after ``idx`` has been formed and used.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, List, Optional, Sequence, Set

# choose(t, idx) -> j*, the position *within idx* of the key to skip next.
Chooser = Callable[[int, List[int]], int]


@dataclass
class StepRecord:
    t: int
    phase: int                 # 1, 2 or 3
    window: List[int]          # [max(0, t-N_r) .. t] as written in the algorithm
    skip_idx: List[int]        # skip list used to form idx (after the shift)
    idx: List[int]             # kept decode positions, ascending
    selected: Optional[int]    # absolute position appended to skip_idx, or None


@dataclass
class HeadState:
    """Selection state of one head (one KV head under GQA).

    ``N_r``: recent window size; ``N_att``: number of decode tokens to attend.
    """

    N_r: int
    N_att: int
    skip_idx: List[int] = field(default_factory=list)
    evicted: Set[int] = field(default_factory=set)

    def __post_init__(self):
        if not (1 <= self.N_att <= self.N_r):
            raise ValueError("Algorithm 1 needs 1 <= N_att <= N_r")

    def phase(self, t: int) -> int:
        """Which of the algorithm's three regimes step ``t`` is in: 1 before
        the first selection (``t < N_att - 1``), 2 while the window still
        grows (``t < N_r``), 3 once the window slides."""
        if t < self.N_att - 1:
            return 1
        return 2 if t < self.N_r else 3

    def needs_choice(self, t: int) -> bool:
        """True when step ``t`` (about to run) adds a skip entry: only in
        phase 2, and only until the list holds ``N_r - N_att`` entries."""
        return self.phase(t) == 2 and len(self.skip_idx) < self.N_r - self.N_att

    def _advance(self, t: int, phase: int) -> None:
        """State changes at the start of step ``t``: once the window slides,
        its oldest position ``t - N_r`` leaves the cache; from phase 2 on,
        every skipped position moves one step along its diagonal (+1)."""
        if phase == 3:
            self.evicted.add(t - self.N_r)
        if phase >= 2:
            self.skip_idx = [j + 1 for j in self.skip_idx]

    def kept(self, t: int) -> List[int]:
        """Decode positions step ``t`` attends, ascending: the window
        ``[max(0, t - N_r), t]`` minus what was evicted and what is skipped."""
        gone = self.evicted | set(self.skip_idx)
        return [j for j in range(max(0, t - self.N_r), t + 1) if j not in gone]

    def step(self, t: int, choose: Optional[Chooser]) -> StepRecord:
        """Run decode step ``t`` and return what it attends.

        ``choose`` is called only when the step adds a skip entry
        (``needs_choice``).  It receives ``t`` and the kept list ``idx`` and
        returns ``j*``, an index into ``idx``.  The entry it names joins the
        skip list after ``idx`` was formed, so it is still attended at step
        ``t``."""
        phase = self.phase(t)
        adds = self.needs_choice(t)
        self._advance(t, phase)
        used_skip = list(self.skip_idx)
        idx = self.kept(t)
        selected = None
        if adds:
            if choose is None:
                raise ValueError(f"step {t} needs a choice but no chooser was given")
            j_star = int(choose(t, list(idx)))
            if not (0 <= j_star < len(idx)):
                raise ValueError("chooser returned an index outside idx")
            selected = idx[j_star]
            self.skip_idx.append(selected)
        return StepRecord(t=t, phase=phase, window=list(range(max(0, t - self.N_r), t + 1)),
                          skip_idx=used_skip, idx=idx, selected=selected)


def run(N_r: int, N_att: int, T: int, choose: Optional[Chooser]) -> List[StepRecord]:
    """Steps ``t = 0 .. T-1`` of one head from an empty skip list."""
    st = HeadState(N_r, N_att)
    return [st.step(t, choose) for t in range(T)]


def scripted(choices: Sequence[int]) -> Chooser:
    """A chooser that returns the given ``j*`` values in order."""
    it = iter(choices)
    return lambda t, idx: next(it)


def by_position(positions: dict) -> Chooser:
    """A chooser that skips a given absolute position at given steps:
    ``positions[t]`` is the decode position to append at step ``t``."""
    return lambda t, idx: idx.index(positions[t])


def uniform(random_ints: Sequence[int]) -> Chooser:
    """A chooser driven by externally drawn non-negative integers: the k-th
    choice is ``random_ints[k] mod |idx|``."""
    it = iter(random_ints)
    return lambda t, idx: int(next(it)) % len(idx)


def offsets_of(state: HeadState, t: int) -> List[int]:
    """The skip entries as distances from the current step ``t``, in append
    order (``t - j`` for each ``j`` in ``skip_idx`` after step ``t``)."""
    return [t - j for j in state.skip_idx]
