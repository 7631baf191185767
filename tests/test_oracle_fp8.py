"""Pins of the oracle's E4M3 decoding against facts fixed outside it: values
worked by hand from the OCP definition, torch's own float8_e4m3fn
conversion for all 256 codes, and the structure of the format (sign
symmetry, monotone magnitudes, exact round trips)."""

import math

import numpy as np
import torch

from oracle import fp8


def test_hand_values():
    want = {
        0x00: 0.0, 0x38: 1.0, 0x40: 2.0, 0x30: 0.5, 0x3C: 1.5, 0x7E: 448.0,
        0x08: 2.0 ** -6, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9, 0x2A: 0.3125,
        0xB8: -1.0, 0xFE: -448.0,
    }
    got = fp8.decode_e4m3(list(want))
    assert got.tolist() == list(want.values())
    assert math.copysign(1.0, fp8.decode_e4m3([0x80])[0]) == -1.0
    assert np.isnan(fp8.decode_e4m3([0x7F, 0xFF])).all()


def test_all_codes_match_torch():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = fp8.decode_e4m3(np.arange(256))
    nan = np.isnan(ref)
    assert (np.isnan(got) == nan).all() and nan.sum() == 2
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def test_structure():
    pos = fp8.decode_e4m3(np.arange(0x7F))           # 0x00 .. 0x7E
    assert np.all(np.diff(pos) > 0)                   # strictly increasing
    assert np.array_equal(fp8.decode_e4m3(np.arange(0x80, 0xFF)), -pos)
    # every finite code round-trips through torch's float -> E4M3 conversion
    back = torch.tensor(pos).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert back.tolist() == list(range(0x7F))


def test_dequantize_scales_exactly():
    codes = np.array([0x38, 0x7E, 0x01, 0xC0])
    assert fp8.dequantize(codes, 0.25).tolist() == [0.25, 112.0, 2.0 ** -11, -0.5]
