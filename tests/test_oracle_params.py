"""Pins of the parameter rules against values worked by hand from the
definitions (sparsity ``1 - N_att / L_dec`` of section 5.1, ``N_r = 0.5 L_dec``
of section 4)."""

import pytest

from oracle import params


@pytest.mark.parametrize("h,w,window,permille,want", [
    (24, 24, 128, 950, 29),     # 0.05 * 576 = 28.8
    (24, 24, 256, 900, 58),     # 0.10 * 576 = 57.6
    (64, 64, 512, 950, 205),    # 0.05 * 4096 = 204.8
    (16, 16, 64, 950, 13),      # 12.8
    (16, 16, 64, 900, 26),      # 25.6
    (32, 32, 512, 950, 51),     # 51.2 (1024 visual tokens)
    (96, 96, 64, 950, 64),      # 460.8 clamped to the window
    (2, 2, 4, 1000, 1),         # zero budget clamped to one key
    (2, 2, 4, 875, 1),          # 0.5 rounds half up -> 1
    (4, 4, 8, 0, 8),            # no sparsity: clamped to N_r
])
def test_n_att(h, w, window, permille, want):
    assert params.n_att_from_sparsity(h, w, window, permille) == want


def test_default_window_and_sparsity():
    assert params.default_window(24, 24) == 288
    assert params.default_window(1, 1) == 1
    assert abs(params.sparsity_of(24, 24, 29) - (1 - 29 / 576)) < 1e-15
    with pytest.raises(ValueError):
        params.n_att_from_sparsity(4, 4, 8, 1001)
