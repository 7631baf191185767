"""Lockstep decode trajectories on the GPU against the oracle: every step of
the tiny workload (prompt 32, 16x16 grid, 8 heads, d=64, window 64) runs
``dsa_plan -> dsa_decode_attention -> dsa_select`` on the GPU and Algorithm 1
in fp64 on the CPU from the same inputs.

Each step compares the kept index sets bit for bit and the outputs within
the tolerance.  The phase-2 argmin must agree exactly, or else fall within
the rounding band of the fp32 logits (a near tie).  In that case the oracle
continues with the GPU's pick and the test counts it."""

import math

import numpy as np
import pytest
import torch

from oracle import step as ostep
from paper_2609_19702_amd import binding as B
from paper_2609_19702_amd import synth
from tests.gpu_util import DEV, TOL, offsets_from_buffer, rel_err, say, within_tie_band

pytestmark = pytest.mark.gpu


def tiny_cache():
    T = synth.tiny_tensors()
    k = torch.cat([T["Kp"], T["K"]], 0).permute(1, 0, 2).unsqueeze(0).contiguous()
    v = torch.cat([T["Vp"], T["V"]], 0).permute(1, 0, 2).unsqueeze(0).contiguous()
    return T, synth.LayerKV(k.to(DEV), v.to(DEV), k.shape[2])


def run_trajectory(kv, Q, Lp, gh, gw, N_r, N_att, Hq, Hkv, d, steps):
    p = B.make_params(Lp, gh, gw, N_r, N_att, B.MODE_DIAGONAL)
    s = B.make_shape(1, Hq, Hkv, d)
    bufs = B.alloc_buffers(p, s, DEV)
    B.state_reset(p, s, bufs.state)
    scale = 1 / math.sqrt(d)
    k64 = kv.k[0].to(torch.float64).cpu().numpy()
    v64 = kv.v[0].to(torch.float64).cpu().numpy()
    Kp, Vp, K, V = k64[:, :Lp], v64[:, :Lp], k64[:, Lp:], v64[:, Lp:]
    Q64 = Q.to(torch.float64).numpy()
    states = ostep.new_states(Hkv, N_r, N_att)
    g = Hq // Hkv
    forced, worst = 0, 0.0
    for t in range(steps):
        pos = torch.tensor([t], dtype=torch.int32, device=DEV)
        q = Q[t].unsqueeze(0).contiguous().to(DEV)
        B.plan(p, s, pos, bufs.state, bufs.plan)
        B.decode_attention(p, s, q, kv.k, kv.v, B.kv_layout(kv.k), pos, bufs.plan, scale,
                           bufs.out, bufs.logits, bufs.workspace)
        B.select(p, s, pos, bufs.plan, bufs.logits, bufs.state)
        cnt, flg, idx = (x.cpu().numpy() for x in B.plan_views(p, s, bufs.plan))
        scnt, sflg, soff = offsets_from_buffer(p, s, bufs.state)
        out = bufs.out.cpu().numpy().astype(np.float64)[0]

        def decide(kvh, t_, idx_, j_ref, sigma):
            nonlocal forced
            k = t_ - (N_att - 1)
            assert scnt[kvh] == k + 1, (t_, kvh, scnt[kvh])
            j_gpu = idx_.index(t_ - int(soff[kvh, k]))
            if j_gpu != j_ref:
                qg = Q64[t_][kvh * g:(kvh + 1) * g]
                assert within_tie_band(qg, K[kvh][idx_], scale, j_gpu, j_ref), (t_, kvh, j_gpu, j_ref)
                forced += 1
            return j_gpu

        res = ostep.request_step(t, Q64[t], Kp, Vp, K, V, scale, "diagonal", states, decide)
        for h in range(Hkv):
            assert flg[h] == 0 and sflg[h] == 0
            assert idx[h, :cnt[h]].tolist() == res.heads[h].idx, (t, h)
        for h in range(Hq):
            e = rel_err(out[h], res.out[h])
            worst = max(worst, e)
            assert e <= TOL, (t, h, e)
    return forced, worst


@pytest.mark.parametrize("n_att", [13, 26, 1, 64])
def test_tiny_full_trajectory(n_att):
    T, kv = tiny_cache()
    say("tiny trajectory N_att", n_att)
    forced, worst = run_trajectory(kv, T["Q"], 32, 16, 16, 64, n_att, 8, 8, 64, 256)
    say(f"  forced near-tie choices: {forced}, worst rel err {worst:.2e}")
    assert forced <= 2


@pytest.mark.parametrize("case", [
    # Hq, Hkv, d, L_p, gh, gw, N_r, N_att
    (8, 2, 128, 16, 8, 8, 24, 6),
    (16, 2, 64, 8, 6, 6, 20, 5),
])
def test_gqa_trajectory(case):
    Hq, Hkv, d, Lp, gh, gw, N_r, N_att = case
    say("gqa trajectory", case)
    w = synth.Workload("gqa_traj", 1, 1, Hq, Hkv, d, Lp, gh, gw, N_r, outlier_frac=0.01, seed=4)
    kv = synth.layer_kv(w, 0, DEV)
    L = gh * gw
    Q = torch.stack([synth.step_query(w, 0, t)[0] for t in range(L)])
    forced, worst = run_trajectory(kv, Q, Lp, gh, gw, N_r, N_att, Hq, Hkv, d, L)
    say(f"  forced near-tie choices: {forced}, worst rel err {worst:.2e}")
    assert forced <= 2
