"""Edge cases and less-travelled paths of the GPU library:

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
    tags, lists = B.kept_views(p, s, st)
    tags[:] = 9
    lists[:] = 5
    st = st.to(DEV)
    mask = torch.tensor([1, 0, 1, 0], dtype=torch.int32, device=DEV)
    B.state_reset(p, s, st, mask)
    cnt, flg, _ = B.state_views(p, s, st.cpu())
    assert cnt.tolist() == [0, 0, 7, 7, 0, 0, 7, 7]
    assert flg.tolist() == [0, 0, 3, 3, 0, 0, 3, 3]
    # the kept lists of the reset requests are dropped (both tags 0); the
    # others keep theirs; the list contents themselves are not touched
    tags, lists = B.kept_views(p, s, st.cpu())
    assert tags.tolist() == [[0, 0]] * 2 + [[9, 9]] * 2 + [[0, 0]] * 2 + [[9, 9]] * 2
    assert (lists == 5).all()


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
