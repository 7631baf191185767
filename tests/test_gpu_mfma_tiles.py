"""The grouped-head (MFMA) tile's wave-to-tile mapping against the oracle.

A split's tiles (prompt tiles, then window tiles, 32 rows each) are dealt
to the workgroup's waves in blocks of consecutive tiles whose size follows
from the split's rows alone, and a wave computes its tiles two at a time.
These cases put one request in one split (256 (request, KV head) pairs, so
the launch is not split further) and choose the prompt length and N_att so
that a split has

* fewer tiles than waves (one tile per wave),
* 14 tiles on 8 waves, one wave holding the last prompt tile and the first
  window tile,
* 17 tiles on 8 waves (blocks of three: a pair, then a single tile),

and, in dense mode, splits of eight tiles on two waves (two pairs per
wave); two of the cases also over fp8 caches.  Positions cover an unused slot, the first decode steps (fewer kept
rows than N_att, so some waves get no tile), every phase boundary of
Algorithm 1 and ragged ones.  Kept sets must match bit for bit, outputs
within the tolerance and every phase-2 pick the oracle's argmin or a
certified near tie, for the fused step and for the separate calls."""

import math
import random

import pytest
import torch

from paper_2609_19702_amd import binding as B
from paper_2609_19702_amd import synth
from tests.gpu_util import (DEV, c_replay_states, check_layer_vs_oracle, fp8_request_arrays,
                            request_arrays, say, states_to_buffer)

pytestmark = pytest.mark.gpu

CASES = [
    # name, B, Hq, Hkv, d, L_p, grid, N_r, N_att, tiles per split (sparse)
    ("g4_7tiles", 32, 32, 8, 128, 96, 16, 160, 100, 7),
    ("g2_14tiles_mixed_wave", 32, 16, 8, 64, 270, 20, 300, 150, 14),
    ("g4_17tiles_blocks_of_3", 32, 32, 8, 128, 300, 20, 300, 212, 17),
    ("g8_4tiles", 64, 32, 4, 128, 64, 12, 100, 60, 4),
]


def positions(Bn, L, N_r, N_att, seed):
    rng = random.Random(seed)
    fixed = [-1, 0, 1, N_att // 3, N_att - 2, N_att - 1, N_att, (N_att + N_r) // 2,
             N_r - 2, N_r - 1, N_r, L - 1]
    fixed = [min(t, L - 1) for t in fixed]
    return (fixed + [rng.randrange(L) for _ in range(Bn - len(fixed))])[:Bn]


def run(p, s, q, kv, pos, st, fused, lay=None):
    bufs = B.alloc_buffers(p, s, DEV)
    st = st.clone() if st is not None else None
    scale = 1 / math.sqrt(s.head_dim)
    lay = B.kv_layout(kv.k) if lay is None else lay
    sparse = p.mode != B.MODE_DENSE
    if fused:
        B.decode_step(p, s, q, kv.k, kv.v, lay, pos, st, bufs.plan, scale, bufs.out, bufs.logits,
                      bufs.workspace)
    else:
        B.plan(p, s, pos, st if sparse else None, bufs.plan)
        B.decode_attention(p, s, q, kv.k, kv.v, lay, pos, bufs.plan if sparse else None, scale,
                           bufs.out, bufs.logits if sparse else None, bufs.workspace)
        if sparse:
            B.select(p, s, pos, bufs.plan, bufs.logits, st)
    torch.cuda.synchronize()
    return bufs, st


@pytest.mark.parametrize("fused", [True, False], ids=["fused", "separate"])
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_mfma_tile_mapping_matches_oracle(case, fused):
    name, Bn, Hq, Hkv, d, Lp, grid, N_r, N_att, tiles = case
    L = grid * grid
    p = B.make_params(Lp, grid, grid, N_r, N_att)
    s = B.make_shape(Bn, Hq, Hkv, d)
    info = B.launch_info(p, s)
    say("mfma tiles", name, "fused" if fused else "separate", "splits", info.max_splits,
        "rows", info.rows_per_split, "waves", info.waves_per_group)
    # the shape this case is about: one split per request, the stated tile count
    assert info.kernel_variant == 100 and info.max_splits == 1
    assert -(-Lp // 32) + -(-N_att // 32) == tiles
    assert info.waves_per_group == min(8, tiles)
    ts = positions(Bn, L, N_r, N_att, seed=tiles)
    rng = random.Random(tiles * 31 + Hkv)
    w = synth.Workload(name, 1, Bn, Hq, Hkv, d, Lp, grid, grid, N_r, outlier_frac=0.01)
    kv = synth.layer_kv(w, 0, DEV)
    q = synth.layer_query(w, 0, DEV)
    states, _ = c_replay_states(N_r, N_att, L, ts, Hkv, rng)
    st0 = states_to_buffer(p, s, states, ts)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    bufs, st = run(p, s, q, kv, pos, st0, fused)
    arrays = [request_arrays(kv, b, Lp) for b in range(Bn)]
    forced = check_layer_vs_oracle(p, s, q, arrays, ts, states, bufs.plan, bufs.out, st,
                                   bufs.logits)
    say(f"  near-tie picks adopted: {forced}")
    assert forced <= 2


@pytest.mark.parametrize("case", CASES[1:3], ids=[c[0] for c in CASES[1:3]])
def test_mfma_tile_mapping_fp8(case):
    """The same mapping over fp8 (E4M3) caches with per-(request, KV head)
    scales: two k-steps per 16-byte K load and half the V registers per
    tile, fused step."""
    name, Bn, Hq, Hkv, d, Lp, grid, N_r, N_att, tiles = case
    L = grid * grid
    p = B.make_params(Lp, grid, grid, N_r, N_att)
    s = B.make_shape(Bn, Hq, Hkv, d)
    info = B.launch_info(p, s)
    assert info.kernel_variant == 100 and info.max_splits == 1
    say("mfma tiles fp8", name, "waves", info.waves_per_group)
    ts = positions(Bn, L, N_r, N_att, seed=tiles + 1)
    rng = random.Random(tiles * 37 + Hkv)
    w = synth.Workload(name, 1, Bn, Hq, Hkv, d, Lp, grid, grid, N_r, outlier_frac=0.01)
    kv = synth.to_fp8(synth.layer_kv(w, 0, DEV))
    q = synth.layer_query(w, 0, DEV)
    states, _ = c_replay_states(N_r, N_att, L, ts, Hkv, rng)
    st0 = states_to_buffer(p, s, states, ts)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    lay = B.kv_layout(kv.k, k_scale=kv.k_scale, v_scale=kv.v_scale)
    bufs, st = run(p, s, q, kv, pos, st0, True, lay)
    arrays = [fp8_request_arrays(kv, b, Lp, Hkv) for b in range(Bn)]
    forced = check_layer_vs_oracle(p, s, q, arrays, ts, states, bufs.plan, bufs.out, st)
    say(f"  near-tie picks adopted: {forced}")
    assert forced <= 2


def test_mfma_dense_two_pairs_per_wave():
    """Dense mode: splits of 256 rows (eight tiles) on two waves, so every wave
    computes two pairs of tiles; ragged lengths leave partial last splits."""
    name, Bn, Hq, Hkv, d, Lp, grid = "dense_g4", 32, 32, 8, 128, 100, 24
    L = grid * grid
    pd = B.make_params(Lp, grid, grid, L, L, B.MODE_DENSE)
    s = B.make_shape(Bn, Hq, Hkv, d)
    info = B.launch_info(pd, s)
    say("mfma dense", "splits", info.max_splits, "rows", info.rows_per_split,
        "waves", info.waves_per_group)
    assert info.kernel_variant == 100 and info.rows_per_split == 256
    assert info.waves_per_group == 2 and info.max_splits > 1
    ts = positions(Bn, L, L, L, seed=3)
    w = synth.Workload(name, 1, Bn, Hq, Hkv, d, Lp, grid, grid, L)
    kv = synth.layer_kv(w, 0, DEV)
    q = synth.layer_query(w, 0, DEV)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    bufs, _ = run(pd, s, q, kv, pos, None, False)
    arrays = [request_arrays(kv, b, Lp) for b in range(Bn)]
    check_layer_vs_oracle(pd, s, q, arrays, ts, None, bufs.plan, bufs.out)
