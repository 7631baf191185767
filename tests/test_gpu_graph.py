"""A decode step (separate calls, dense, or the fused step) captured as a
HIP graph replays to exactly the eager result, replay after replay, with
unrelated eager work and synchronisations between the replays (the library
records no memset nodes: every buffer it clears is cleared by a kernel).
The timed launch variants compute the same output as the plain ones."""

import pytest
import torch

from paper_2609_19702_amd import binding as B
from paper_2609_19702_amd import synth, workload
from tests.gpu_util import DEV, say

pytestmark = pytest.mark.gpu


def snapshot(bt):
    return [(L.bufs.out.clone(), L.bufs.state.clone(), L.bufs.plan.clone(), L.bufs.logits.clone())
            for L in bt.layers]


@pytest.mark.parametrize("mode,kv_heads,d", [
    ("separate", 4, 128),  # plan -> attention -> select, grouped heads (MFMA tile)
    ("dense", 4, 128),
    ("fused", 4, 128),     # the fused step, grouped heads
    ("fused", 8, 64),      # the fused step, one query head per KV head (vector-ALU tile)
])
def test_graph_replay_matches_eager(mode, kv_heads, d):
    dense, fused = mode == "dense", mode == "fused"
    w = synth.Workload("graph", 3, 12, 8, kv_heads, d, 40, 12, 12, 48)
    bt = workload.make_batch(w)
    workload.build_histories(bt)
    workload.step(bt, dense=dense, fused=fused)
    torch.cuda.synchronize()
    ref = snapshot(bt)
    ref_dense = bt.dense_bufs.out.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        workload.step(bt, dense=dense, fused=fused)
    for rep in range(4):
        for L in bt.layers:  # scribble over the outputs between replays
            L.bufs.out.fill_(float("nan"))
        bt.dense_bufs.out.fill_(float("nan"))
        x = torch.randn(1000, device=DEV).sum()  # unrelated eager work
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        say(f"replay {rep} ({mode}, {kv_heads} KV heads, d={d}) {float(x):.3f}")
        if dense:
            assert torch.equal(bt.dense_bufs.out, ref_dense)
        else:
            for L, (o, st, pl, lg) in zip(bt.layers, ref):
                assert torch.equal(L.bufs.out, o)
                assert torch.equal(L.bufs.state, st)
                assert torch.equal(L.bufs.plan, pl)


@pytest.mark.parametrize("fused", [False, True])
def test_timed_launch_same_output(fused):
    w = synth.Workload("timed", 2, 8, 16, 4, 64, 20, 10, 10, 40)
    bt = workload.make_batch(w)
    workload.build_histories(bt)
    workload.step(bt, fused=fused)
    torch.cuda.synchronize()
    ref = [L.bufs.out.clone() for L in bt.layers]
    timers = [B.timing_events() for _ in bt.layers]
    workload.step(bt, timers=timers, fused=fused)
    torch.cuda.synchronize()
    for L, o, (a, b) in zip(bt.layers, ref, timers):
        assert torch.equal(L.bufs.out, o)
        assert 0.0 < a.elapsed_time(b) < 1000.0
