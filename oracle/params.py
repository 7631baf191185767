"""Parameter rules of the method.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

* ``L_dec = H * W``: the decode length is the number of visual tokens of the
  ``H x W`` token grid (section 3.1, Table 1).
* ``N_r = 0.5 * L_dec`` is the paper's default recent window ("Parameter
  selection" paragraph of section 4); an explicit window overrides it.
* Sparsity is the fraction of decode KV not attended relative to the maximum
  decode length, ``s = 1 - N_att / L_dec`` (section 5.1, "Our methods").
  Solving for ``N_att`` and rounding half up gives ``N_att``; it is clamped
  to ``[1, N_r]`` since the algorithm needs ``N_att <= N_r``.
"""

from __future__ import annotations

from fractions import Fraction


def decode_length(grid_h: int, grid_w: int) -> int:
    return int(grid_h) * int(grid_w)


def default_window(grid_h: int, grid_w: int) -> int:
    """``N_r = 0.5 * L_dec`` (at least 1)."""
    return max(1, decode_length(grid_h, grid_w) // 2)


def n_att_from_sparsity(grid_h: int, grid_w: int, window: int, sparsity_permille: int) -> int:
    """``N_att = round((1 - s) * L_dec)`` clamped to ``[1, N_r]``, with
    ``s = sparsity_permille / 1000`` in exact rational arithmetic and ties
    rounded up."""
    if not (0 <= sparsity_permille <= 1000):
        raise ValueError("sparsity must be within [0, 1000] permille")
    exact = Fraction(1000 - sparsity_permille, 1000) * decode_length(grid_h, grid_w)
    n = int(exact + Fraction(1, 2))  # floor(x + 1/2) for x >= 0
    return max(1, min(int(window), n))


def sparsity_of(grid_h: int, grid_w: int, n_att: int) -> float:
    """The realised sparsity ``1 - N_att / L_dec``."""
    return 1.0 - n_att / decode_length(grid_h, grid_w)
