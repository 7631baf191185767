"""Edge cases and less-travelled paths of the GPU library:

* windows at the size limits: the fused step up to N_r = 16384, the separate
  plan beyond it (checked against the oracle on a few pairs and against
  properties that hold at any size: count, order, window, skipped offsets);
* every slot unused; no prompt with a single key; N_att = 1;
* state reset of a subset of requests;
* two independent layers on two streams at once;
* argument errors of the fused step.
"""

import copy
import math
import random

import numpy as np
import pytest
import torch

from oracle import alg1, step as ostep
from paper_2609_19702_amd import binding as B
from paper_2609_19702_amd import synth, workload
from tests.gpu_util import DEV, TOL, rel_err, request_arrays, run_layer, say, states_to_buffer

pytestmark = pytest.mark.gpu


def random_offsets_state(p, s, ts, rng):
    """A valid state for positions ``ts`` drawn in the offset form directly
    (each selection step picks a kept offset at random) -- used where the
    literal oracle replay would be too slow; the oracle checks a few pairs."""
    Hkv = s.num_kv_heads
    buf = torch.zeros(B.state_bytes(p, s), dtype=torch.uint8)
    cnt, _, off = B.state_views(p, s, buf)
    sets = []
    for b, t in enumerate(ts):
        for h in range(Hkv):
            D = []
            avail = list(range(p.n_att - 1))  # kept offsets before the first selection
            for u in range(p.n_att - 1, min(t - 1, p.window - 2) + 1):
                avail.append(u)               # the window reaches offset u at step u
                k = rng.randrange(len(avail))
                avail[k], avail[-1] = avail[-1], avail[k]
                D.append(avail.pop())
            pair = b * Hkv + h
            cnt[pair] = len(D)
            if D:
                off[pair, :len(D)] = torch.tensor(np.array(D, dtype=np.uint16).view(np.int16))
            sets.append(D)
    return buf, sets


def check_plan_properties(p, ts, Hkv, sets, cnt, idx):
    for b, t in enumerate(ts):
        for h in range(Hkv):
            pair = b * Hkv + h
            n = int(cnt[pair])
            assert n == min(t + 1, p.n_att)
            pos = idx[pair, :n].tolist()
            assert pos == sorted(pos) and len(set(pos)) == n
            assert all(max(0, t - p.window + 1) <= j <= t for j in pos)
            skipped = {t - d for d in sets[pair][:max(0, min(t - p.n_att + 1, p.window - p.n_att))]}
            assert not (skipped & set(pos))


@pytest.mark.parametrize("window,n_att,grid,fused", [
    (4096, 405, 90, True),       # 720x720 Emu3 output length (8100 tokens), N_r = L/2
    (16384, 1000, 130, True),    # the fused step's largest window
    (20000, 2000, 150, False),   # beyond it: the separate calls
])
def test_large_windows(window, n_att, grid, fused):
    rng = random.Random(window)
    L = grid * grid
    ts = [L - 1, window - 2, n_att - 1, rng.randrange(L), window + 7]
    p = B.make_params(16, grid, grid, window, n_att)
    s = B.make_shape(len(ts), 4, 2, 64)
    say("large window", window, n_att, grid, "fused" if fused else "separate")
    st, sets = random_offsets_state(p, s, ts, rng)
    w = synth.Workload("big", 1, len(ts), 4, 2, 64, 16, grid, grid, window)
    kv = synth.layer_kv(w, 0, DEV)
    q = synth.layer_query(w, 0, DEV)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    bufs = B.alloc_buffers(p, s, DEV)
    st = st.to(DEV)
    if fused:
        B.decode_step(p, s, q, kv.k, kv.v, B.kv_layout(kv.k), pos, st, bufs.plan, 0.125, bufs.out,
                      bufs.logits, bufs.workspace)
    else:
        with pytest.raises(B.DSAError) as e:
            B.decode_step(p, s, q, kv.k, kv.v, B.kv_layout(kv.k), pos, st, bufs.plan, 0.125,
                          bufs.out, bufs.logits, bufs.workspace)
        assert e.value.status == B.ERR_UNSUPPORTED
        B.plan(p, s, pos, st, bufs.plan)
        B.decode_attention(p, s, q, kv.k, kv.v, B.kv_layout(kv.k), pos, bufs.plan, 0.125,
                           bufs.out, bufs.logits, bufs.workspace)
        B.select(p, s, pos, bufs.plan, bufs.logits, st)
    cnt, flg, idx = (x.cpu().numpy() for x in B.plan_views(p, s, bufs.plan))
    assert not flg.any()
    check_plan_properties(p, ts, 2, sets, cnt, idx)
    # outputs of two pairs against the oracle (attention over the GPU's kept set)
    qn = q.double().cpu().numpy()
    out = bufs.out.double().cpu().numpy()
    for b in (0, 3):
        Kp, Vp, K, V = request_arrays(kv, b, 16)
        for h in range(2):
            kept = idx[b * 2 + h, :cnt[b * 2 + h]].tolist()
            keys = np.concatenate([Kp[h], K[h][kept]])
            vals = np.concatenate([Vp[h], V[h][kept]])
            for i in range(2):
                from oracle import attention
                ref, _ = attention.attend(qn[b, h * 2 + i], keys, vals, 0.125)
                assert rel_err(out[b, h * 2 + i], ref) <= TOL


def test_all_slots_unused_and_single_key():
    p = B.make_params(0, 4, 4, 8, 3)
    s = B.make_shape(3, 2, 2, 64)
    w = synth.Workload("edge", 1, 3, 2, 2, 64, 0, 4, 4, 8)
    kv = synth.layer_kv(w, 0, DEV)
    q = synth.layer_query(w, 0, DEV)
    bufs = B.alloc_buffers(p, s, DEV)
    B.state_reset(p, s, bufs.state)
    for fused in (False, True):
        pos = torch.full((3,), -1, dtype=torch.int32, device=DEV)
        bufs.out.fill_(7.0)
        if fused:
            B.decode_step(p, s, q, kv.k, kv.v, B.kv_layout(kv.k), pos, bufs.state, bufs.plan, 0.125,
                          bufs.out, bufs.logits, bufs.workspace)
        else:
            run_layer(p, s, q, kv, pos, bufs.state, bufs)
        cnt, flg, _ = (x.cpu().numpy() for x in B.plan_views(p, s, bufs.plan))
        assert torch.all(bufs.out == 0) and not cnt.any() and (flg == B.FLAG_INACTIVE).all()
        # no prompt, t = 0: the only key is decode row 0, the output is its value row
        pos = torch.tensor([0, 0, -1], dtype=torch.int32, device=DEV)
        if fused:
            B.decode_step(p, s, q, kv.k, kv.v, B.kv_layout(kv.k), pos, bufs.state, bufs.plan, 0.125,
                          bufs.out, bufs.logits, bufs.workspace)
        else:
            run_layer(p, s, q, kv, pos, bufs.state, bufs)
        for b in (0, 1):
            for h in range(2):
                assert torch.equal(bufs.out[b, h], kv.v[b, h, 0].float())


def test_state_reset_mask():
    p = B.make_params(4, 6, 6, 16, 5)
    s = B.make_shape(4, 2, 2, 64)
    st = torch.zeros(B.state_bytes(p, s), dtype=torch.uint8)
    cnt, flg, _ = B.state_views(p, s, st)
    cnt[:] = 7
    flg[:] = 3
    st = st.to(DEV)
    mask = torch.tensor([1, 0, 1, 0], dtype=torch.int32, device=DEV)
    B.state_reset(p, s, st, mask)
    cnt, flg, _ = B.state_views(p, s, st.cpu())
    assert cnt.tolist() == [0, 0, 7, 7, 0, 0, 7, 7]
    assert flg.tolist() == [0, 0, 3, 3, 0, 0, 3, 3]


def test_two_streams_concurrently():
    w = synth.Workload("streams", 2, 16, 8, 8, 64, 50, 16, 16, 64)
    bt = workload.make_batch(w)
    workload.build_histories(bt)
    state0 = [Lr.bufs.state.clone() for Lr in bt.layers]
    workload.step(bt, fused=True)
    torch.cuda.synchronize()
    ref = [(Lr.bufs.out.clone(), Lr.bufs.state.clone()) for Lr in bt.layers]
    for Lr, st in zip(bt.layers, state0):
        Lr.bufs.state.copy_(st)
        Lr.bufs.out.zero_()
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for Lr, stream in zip(bt.layers, streams):
        with torch.cuda.stream(stream):
            workload.fused_layer(bt, Lr)
    torch.cuda.synchronize()
    for Lr, (o, st) in zip(bt.layers, ref):
        assert torch.equal(Lr.bufs.out, o) and torch.equal(Lr.bufs.state, st)


def test_decode_step_argument_errors():
    w = synth.Workload("args", 1, 2, 4, 4, 64, 8, 6, 6, 12)
    bt = workload.make_batch(w)
    L = bt.layers[0]
    lay = B.kv_layout(L.kv.k)
    args = (bt.p, bt.s, L.q, L.kv.k, L.kv.v, lay, bt.pos)
    with pytest.raises(B.DSAError) as e:   # no window logits buffer
        B.decode_step(*args, L.bufs.state, L.bufs.plan, bt.scale, L.bufs.out, None, L.bufs.workspace)
    assert e.value.status == B.ERR_INVALID_ARG
    with pytest.raises(B.DSAError) as e:   # no state
        B.decode_step(*args, None, L.bufs.plan, bt.scale, L.bufs.out, L.bufs.logits, L.bufs.workspace)
    assert e.value.status == B.ERR_INVALID_ARG
    small = torch.zeros(B.plan_bytes(bt.p, bt.s) - 256, dtype=torch.uint8, device=DEV)
    with pytest.raises(B.DSAError) as e:   # plan buffer too small
        B.decode_step(*args, L.bufs.state, small, bt.scale, L.bufs.out, L.bufs.logits, L.bufs.workspace)
    assert e.value.status == B.ERR_WORKSPACE
    with pytest.raises(B.DSAError) as e:   # non-finite scale
        B.decode_step(*args, L.bufs.state, L.bufs.plan, float("nan"), L.bufs.out, L.bufs.logits,
                      L.bufs.workspace)
    assert e.value.status == B.ERR_INVALID_ARG
