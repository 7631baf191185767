"""The selection paths that only long windows reach, against the oracle.

* Grouped query heads with more than 256 kept window keys: the phase-2
  score (sum of the group's window softmaxes) is then computed by the
  streaming form of the device argmin, in the separate select kernel and in
  the fused step's combine.  Every pick is compared with the oracle's argmin
  over the same kept keys (equal, or inside the certified fp32 tie band).
* One query head per KV head with more than 256 kept window keys in a
  single split: the fused decode kernel runs the streaming argmin itself.
* Grouped query heads with more than 256 kept window keys in a single split
  (enough (request, KV head) pairs that no request is split): the fused
  decode kernel takes the selection itself, each head's window softmax on a
  wave of its own, then the score sum and argmin on one wave.  Checked
  against the oracle and bit for bit against the separate calls (same plan,
  logits, outputs and stored offsets).
* Windows of 4096, 16384 and 20000 positions: selection states replayed by
  the literal Algorithm 1 of the C oracle (every choice random), then the
  plan's kept sets compared bit for bit with the oracle's, the outputs with
  the oracle's attention, and every pick the step makes with the oracle's
  argmin.
"""

import math
import random

import numpy as np
import pytest
import torch

from paper_2609_19702_amd import binding as B
from paper_2609_19702_amd import synth
from tests.gpu_util import (DEV, c_replay_states, check_layer_vs_oracle, request_arrays, say,
                            states_to_buffer)

pytestmark = pytest.mark.gpu


def run_step(p, s, q, kv, pos, st, fused):
    bufs = B.alloc_buffers(p, s, DEV)
    st = st.clone()
    scale = 1 / math.sqrt(s.head_dim)
    lay = B.kv_layout(kv.k)
    if fused:
        B.decode_step(p, s, q, kv.k, kv.v, lay, pos, st, bufs.plan, scale, bufs.out, bufs.logits,
                      bufs.workspace)
    else:
        B.plan(p, s, pos, st, bufs.plan)
        B.decode_attention(p, s, q, kv.k, kv.v, lay, pos, bufs.plan, scale, bufs.out,
                           bufs.logits, bufs.workspace)
        B.select(p, s, pos, bufs.plan, bufs.logits, st)
    torch.cuda.synchronize()
    return bufs, st


LONG = [
    # Hq, Hkv, d, L_p, grid, N_r, N_att
    (4, 2, 128, 16, 30, 700, 400),    # G = 2
    (8, 2, 64, 16, 30, 700, 300),     # G = 4
    (16, 2, 128, 0, 30, 700, 500),    # G = 8
    (128, 128, 64, 16, 30, 700, 400),  # G = 1, one split per request in the fused step
]


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("case", LONG, ids=[str(c) for c in LONG])
def test_selection_over_long_windows(case, fused):
    Hq, Hkv, d, Lp, grid, N_r, N_att = case
    L = grid * grid
    ts = [N_att - 1, (N_att + N_r) // 2, N_r - 2, L - 1]  # first, middle, last select; phase 3
    Bn = len(ts)
    say("long-window selection", case, "fused" if fused else "separate")
    rng = random.Random(N_att * 7 + Hq)
    w = synth.Workload("longsel", 1, Bn, Hq, Hkv, d, Lp, grid, grid, N_r, outlier_frac=0.01)
    kv = synth.layer_kv(w, 0, DEV)
    q = synth.layer_query(w, 0, DEV)
    p = B.make_params(Lp, grid, grid, N_r, N_att)
    s = B.make_shape(Bn, Hq, Hkv, d)
    info = B.launch_info(p, s)
    if Hq == Hkv and fused:
        assert info.max_splits == 1  # the fused kernel selects on its own
    states, _ = c_replay_states(N_r, N_att, L, ts, Hkv, rng)
    st0 = states_to_buffer(p, s, states, ts)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    bufs, st = run_step(p, s, q, kv, pos, st0, fused)
    arrays = [request_arrays(kv, b, Lp) for b in range(Bn)]
    forced = check_layer_vs_oracle(p, s, q, arrays, ts, states, bufs.plan, bufs.out, st,
                                   bufs.logits)
    say(f"  near-tie picks adopted: {forced}")
    assert forced <= 2


@pytest.mark.parametrize("window,n_att,grid,fused", [
    (4096, 405, 90, True),       # a 720x720 Emu3-like image (8100 tokens), N_r = L/2
    (16384, 1000, 130, True),    # the fused step's largest window
    (20000, 2000, 150, False),   # beyond it: the separate calls
])
def test_large_windows_literal(window, n_att, grid, fused):
    rng = random.Random(window)
    L = grid * grid
    ts = [L - 1, window - 2, n_att - 1, rng.randrange(n_att, window - 2), window + 7]
    Bn, Hq, Hkv, d, Lp = len(ts), 4, 2, 64, 16
    p = B.make_params(Lp, grid, grid, window, n_att)
    s = B.make_shape(Bn, Hq, Hkv, d)
    say("large window", window, n_att, grid, "fused" if fused else "separate")
    states, kept = c_replay_states(window, n_att, L, ts, Hkv, rng)
    st0 = states_to_buffer(p, s, states, ts)
    w = synth.Workload("big", 1, Bn, Hq, Hkv, d, Lp, grid, grid, window)
    kv = synth.layer_kv(w, 0, DEV)
    q = synth.layer_query(w, 0, DEV)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    if not fused:
        with pytest.raises(B.DSAError) as e:
            B.decode_step(p, s, q, kv.k, kv.v, B.kv_layout(kv.k), pos, st0.clone(),
                          B.alloc_buffers(p, s, DEV).plan, 0.125, torch.empty_like(q, dtype=torch.float32),
                          B.alloc_buffers(p, s, DEV).logits, None)
        assert e.value.status == B.ERR_UNSUPPORTED
    bufs, st = run_step(p, s, q, kv, pos, st0, fused)
    # kept sets: the C oracle's literal replay, bit for bit
    cnt, flg, idx = (x.cpu().numpy() for x in B.plan_views(p, s, bufs.plan))
    assert not flg.any()
    for b in range(Bn):
        for h in range(Hkv):
            assert idx[b * Hkv + h, :cnt[b * Hkv + h]].tolist() == kept[b][h], (b, h)
    # outputs, logits and every pick against the Python oracle's step
    arrays = [request_arrays(kv, b, Lp) for b in range(Bn)]
    forced = check_layer_vs_oracle(p, s, q, arrays, ts, states, bufs.plan, bufs.out, st,
                                   bufs.logits)
    assert forced <= 2


SINGLE_SPLIT_GQA = [
    # Hq, Hkv, d, L_p, grid, N_r, N_att, copies of the four positions
    (64, 32, 128, 16, 30, 700, 400, 2),    # G = 2
    (128, 32, 64, 16, 30, 700, 300, 2),    # G = 4
    (256, 32, 128, 0, 30, 700, 470, 2),    # G = 8
    (128, 32, 128, 256, 30, 700, 200, 2),  # G = 4, at most 256 window keys
]


@pytest.mark.parametrize("case", SINGLE_SPLIT_GQA, ids=[str(c) for c in SINGLE_SPLIT_GQA])
def test_fused_grouped_selection_single_split(case):
    Hq, Hkv, d, Lp, grid, N_r, N_att, copies = case
    L = grid * grid
    ts = [N_att - 1, (N_att + N_r) // 2, N_r - 2, L - 1] * copies
    Bn = len(ts)
    say("fused grouped selection, one split", case)
    rng = random.Random(N_att * 11 + Hq)
    w = synth.Workload("gqasel", 1, Bn, Hq, Hkv, d, Lp, grid, grid, N_r, outlier_frac=0.01)
    kv = synth.layer_kv(w, 0, DEV)
    q = synth.layer_query(w, 0, DEV)
    p = B.make_params(Lp, grid, grid, N_r, N_att)
    s = B.make_shape(Bn, Hq, Hkv, d)
    assert B.launch_info(p, s).max_splits == 1  # the decode kernel selects on its own
    states, _ = c_replay_states(N_r, N_att, L, ts, Hkv, rng)
    st0 = states_to_buffer(p, s, states, ts)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    fb, fst = run_step(p, s, q, kv, pos, st0, True)
    sb, sst = run_step(p, s, q, kv, pos, st0, False)
    assert torch.equal(fst, sst)
    assert torch.equal(fb.plan, sb.plan)
    assert torch.equal(fb.out, sb.out)
    assert torch.equal(fb.logits, sb.logits)
    arrays = [request_arrays(kv, b, Lp) for b in range(Bn)]
    forced = check_layer_vs_oracle(p, s, q, arrays, ts, states, fb.plan, fb.out, fst, fb.logits)
    say(f"  near-tie picks adopted: {forced}")
    assert forced <= 2
