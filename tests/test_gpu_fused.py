"""The fused decode step (``dsa_decode_step``) against the three separate
calls (``dsa_plan -> dsa_decode_attention -> dsa_select``): plan, window
logits, output and selection state must be identical bit for bit, with one
split or several, at phase-1, phase-2 and phase-3 positions, with unused
slots and with grouped query heads.  A tiny decode trajectory driven only by
the fused step stays in lockstep with the oracle.

The fused step reads its kept window rows from the kept list the previous
selection stored (when it matches the step) instead of rebuilding them from
the skip entries: with the lists removed it must give the same plan, logits,
outputs and stored offsets, and every stored list must equal the window
part of the plan, as offsets from the decode position, largest first."""

import math

import numpy as np
import pytest
import torch

from oracle import step as ostep
from paper_2609_19702_amd import binding as B
from paper_2609_19702_amd import synth, workload
from tests.gpu_util import DEV, TOL, offsets_from_buffer, rel_err, say, within_tie_band

pytestmark = pytest.mark.gpu

CASES = [
    # name, layers, batch, Hq, Hkv, d, L_p, gh, gw, window
    ("mha64", 2, 24, 8, 8, 64, 40, 16, 16, 64),
    ("mha128_split", 2, 16, 4, 4, 128, 300, 12, 12, 100),
    ("gqa4", 2, 10, 16, 4, 128, 64, 20, 20, 160),
    ("gqa8_d64", 1, 6, 16, 2, 64, 10, 8, 8, 40),
    ("gqa2_noprompt", 1, 9, 4, 2, 64, 0, 9, 9, 30),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_fused_equals_separate_calls(case):
    name, nl, Bn, Hq, Hkv, d, Lp, gh, gw, win = case
    w = synth.Workload(name, nl, Bn, Hq, Hkv, d, Lp, gh, gw, win, sparsity_permille=900,
                       outlier_frac=0.01)
    L = gh * gw
    rng = np.random.default_rng(5)
    pos = rng.integers(0, L, Bn).tolist()
    pos[0] = -1
    pos[1] = L - 1
    p0 = B.params_from_sparsity(Lp, gh, gw, win, 900)
    pos[2] = p0.n_att - 1          # first phase-2 step
    pos[3 % Bn] = p0.window - 2    # last phase-2 step
    bt = workload.make_batch(w, positions=pos)
    workload.build_histories(bt)
    info = B.launch_info(bt.p, bt.s)
    say(name, "splits", info.max_splits, "rows", info.rows_per_split, "n_att", bt.p.n_att)
    # separate calls on a copy of the state
    states = [Lr.bufs.state.clone() for Lr in bt.layers]
    workload.step(bt)
    torch.cuda.synchronize()
    ref = [(Lr.bufs.out.clone(), Lr.bufs.state.clone(), Lr.bufs.plan.clone(), Lr.bufs.logits.clone())
           for Lr in bt.layers]
    for Lr, st in zip(bt.layers, states):
        Lr.bufs.state.copy_(st)
        Lr.bufs.out.fill_(float("nan"))
        Lr.bufs.plan.fill_(0x5A)
        Lr.bufs.logits.fill_(float("nan"))
    workload.step(bt, fused=True)
    torch.cuda.synchronize()
    for li, (Lr, (o, st, pl, lg)) in enumerate(zip(bt.layers, ref)):
        cnt, flg, idx = B.plan_views(bt.p, bt.s, Lr.bufs.plan)
        rcnt, rflg, ridx = B.plan_views(bt.p, bt.s, pl)
        assert torch.equal(cnt, rcnt) and torch.equal(flg, rflg), li
        for pair in range(Bn * Hkv):
            n = int(rcnt[pair])
            assert torch.equal(idx[pair, :n], ridx[pair, :n]), (li, pair)
        assert torch.equal(Lr.bufs.out, o), li
        assert torch.equal(Lr.bufs.state, st), li
        lg_f = Lr.bufs.logits.view(Bn, Hq, -1)
        lg_r = lg.view(Bn, Hq, -1)
        for b in range(Bn):
            n = int(rcnt[b * Hkv])
            assert torch.equal(lg_f[b, :, :n], lg_r[b, :, :n]), (li, b)


LIST_CASES = CASES[:4] + [
    # many (request, KV head) pairs and skip lists of 770-864 entries: lists on,
    # three splits per request (the combine stores the next step's list)
    ("wide_gqa2", 1, 33, 4, 2, 64, 16, 40, 40, 1024),
    ("wide_mha", 1, 70, 1, 1, 64, 8, 36, 36, 900),
    # few pairs with kept lists longer than the 256 offsets loaded ahead
    # (N_att 360 and 410; several splits per request)
    ("long_lists", 1, 40, 2, 1, 64, 16, 60, 60, 2048),
    ("long_lists_gqa4", 1, 12, 16, 4, 128, 0, 64, 64, 1500),
]


@pytest.mark.parametrize("case", LIST_CASES, ids=[c[0] for c in LIST_CASES])
def test_fused_kept_list_equals_rebuild(case):
    name, nl, Bn, Hq, Hkv, d, Lp, gh, gw, win = case
    w = synth.Workload(name, nl, Bn, Hq, Hkv, d, Lp, gh, gw, win, sparsity_permille=900,
                       outlier_frac=0.01)
    L = gh * gw
    rng = np.random.default_rng(11)
    pos = rng.integers(0, L, Bn).tolist()
    p0 = B.params_from_sparsity(Lp, gh, gw, win, 900)
    pos[0] = p0.n_att - 1          # first phase-2 step: no list yet
    pos[1] = p0.n_att              # first step that has one
    pos[2] = p0.window - 2         # last phase-2 step
    pos[3] = p0.window - 1         # first phase-3 step
    bt = workload.make_batch(w, positions=pos)
    workload.build_histories(bt)
    p, s = bt.p, bt.s
    lay = B.state_layout(p, s)
    assert lay.kept_cap == p.n_att - p.sinks
    info = B.launch_info(p, s)
    reads = info.kept_read
    # lists for launches of few pairs or long skip lists, of at most 256 kept offsets
    assert reads == ((Bn * Hkv <= 64 and lay.kept_cap <= 512)
                     or (lay.cap > 512 and lay.kept_cap <= 256))
    if name.startswith("wide"):
        assert reads and info.max_splits > 1
    if name.startswith("long"):
        assert reads and lay.kept_cap > 256
    say(name, "kept_cap", lay.kept_cap, "reads lists", reads, "positions", pos)
    states = [Lr.bufs.state.clone() for Lr in bt.layers]
    # every list the histories stored matches the plan of its step
    workload.step(bt, fused=True)
    torch.cuda.synchronize()
    ref = [(Lr.bufs.out.clone(), Lr.bufs.state.clone(), Lr.bufs.plan.clone(), Lr.bufs.logits.clone())
           for Lr in bt.layers]
    # the same step again on the state it left (as a benchmark repeats it): its
    # list is still in its slot, and every result is the same
    workload.step(bt, fused=True)
    torch.cuda.synchronize()
    for li, (Lr, (o, st, pl, lg)) in enumerate(zip(bt.layers, ref)):
        assert torch.equal(Lr.bufs.out, o) and torch.equal(Lr.bufs.state, st), li
        assert torch.equal(Lr.bufs.plan, pl), li
    used = 0
    for Lr, st0 in zip(bt.layers, states):
        tags, lists = B.kept_views(p, s, st0)
        if not reads:  # launches that keep no lists never write them
            assert not tags.any()
            continue
        cnt, _, idx = B.plan_views(p, s, Lr.bufs.plan)
        for pair in range(Bn * Hkv):
            t = pos[pair // Hkv]
            k = min(t - (p.n_att - 1), lay.cap)
            if k < 1:
                continue
            sl = k & 1
            assert int(tags[pair, sl]) == k + 1, (pair, t, k)
            used += 1
            got = (lists[pair, sl, :lay.kept_cap].to(torch.int64) & 0xFFFF).tolist()
            n = int(cnt[pair])
            want = [t - int(j) for j in idx[pair, p.sinks:n].tolist()]
            assert got == want, (pair, t)
    assert used > 0 or not reads
    # the same step with every list removed: the kept rows are rebuilt
    for Lr, st in zip(bt.layers, states):
        st2 = st.clone()
        tags, _ = B.kept_views(p, s, st2)
        tags.zero_()
        Lr.bufs.state.copy_(st2)
        Lr.bufs.out.fill_(float("nan"))
        Lr.bufs.plan.fill_(0x5A)
        Lr.bufs.logits.fill_(float("nan"))
    workload.step(bt, fused=True)
    torch.cuda.synchronize()
    for li, (Lr, (o, st, pl, lg)) in enumerate(zip(bt.layers, ref)):
        assert torch.equal(Lr.bufs.out, o), li
        cnt, flg, idx = B.plan_views(p, s, Lr.bufs.plan)
        rcnt, rflg, ridx = B.plan_views(p, s, pl)
        assert torch.equal(cnt, rcnt) and torch.equal(flg, rflg), li
        for pair in range(Bn * Hkv):
            n = int(rcnt[pair])
            assert torch.equal(idx[pair, :n], ridx[pair, :n]), (li, pair)
        lg_a, lg_r = Lr.bufs.logits.view(Bn, Hq, -1), lg.view(Bn, Hq, -1)
        for b in range(Bn):
            n = int(rcnt[b * Hkv])
            assert torch.equal(lg_a[b, :, :n], lg_r[b, :, :n]), (li, b)
        a_cnt, a_flg, a_off = B.state_views(p, s, Lr.bufs.state)
        r_cnt, r_flg, r_off = B.state_views(p, s, st)
        assert torch.equal(a_cnt, r_cnt) and torch.equal(a_flg, r_flg) and torch.equal(a_off, r_off)
        # the list each selection stored for the next step (other slot)
        a_tags, a_lists = B.kept_views(p, s, Lr.bufs.state)
        r_tags, r_lists = B.kept_views(p, s, st)
        if not reads:
            assert not a_tags.any() and not r_tags.any()
            continue
        for pair in range(Bn * Hkv):
            t = pos[pair // Hkv]
            k = t - (p.n_att - 1)
            if 0 <= k < lay.cap:
                sl = (k + 1) & 1
                assert int(a_tags[pair, sl]) == k + 2 == int(r_tags[pair, sl]), (li, pair)
                assert torch.equal(a_lists[pair, sl, :lay.kept_cap], r_lists[pair, sl, :lay.kept_cap])


def test_fused_tiny_trajectory():
    T = synth.tiny_tensors()
    Lp, H, d, N_r, N_att = 32, 8, 64, 64, 13
    k = torch.cat([T["Kp"], T["K"]], 0).permute(1, 0, 2).unsqueeze(0).contiguous().to(DEV)
    v = torch.cat([T["Vp"], T["V"]], 0).permute(1, 0, 2).unsqueeze(0).contiguous().to(DEV)
    p = B.make_params(Lp, 16, 16, N_r, N_att)
    s = B.make_shape(1, H, H, d)
    bufs = B.alloc_buffers(p, s, DEV)
    B.state_reset(p, s, bufs.state)
    scale = 1 / math.sqrt(d)
    k64, v64 = k[0].double().cpu().numpy(), v[0].double().cpu().numpy()
    Q64 = T["Q"].double().numpy()
    states = ostep.new_states(H, N_r, N_att)
    assert B.launch_info(p, s).kept_read == 1  # every step after the first selection reads a list
    cap = B.state_layout(p, s).cap
    forced = 0
    for t in range(256):
        pos = torch.tensor([t], dtype=torch.int32, device=DEV)
        B.decode_step(p, s, T["Q"][t].unsqueeze(0).contiguous().to(DEV), k, v, B.kv_layout(k), pos,
                      bufs.state, bufs.plan, scale, bufs.out, bufs.logits, bufs.workspace)
        cnt, flg, idx = (x.cpu().numpy() for x in B.plan_views(p, s, bufs.plan))
        scnt, sflg, soff = offsets_from_buffer(p, s, bufs.state)
        kk = t - (N_att - 1)
        if 0 <= kk < cap:  # this step selected: the next step's list is stored, tagged
            tags, _ = B.kept_views(p, s, bufs.state)
            assert (tags[:, (kk + 1) & 1] == kk + 2).all(), t

        def decide(kvh, t_, idx_, j_ref, sigma):
            nonlocal forced
            j = idx_.index(t_ - int(soff[kvh, t_ - N_att + 1]))
            if j != j_ref:
                assert within_tie_band(Q64[t_][kvh], k64[kvh, Lp:][idx_], scale, j, j_ref)
                forced += 1
            return j

        res = ostep.request_step(t, Q64[t], k64[:, :Lp], v64[:, :Lp], k64[:, Lp:], v64[:, Lp:],
                                 scale, "diagonal", states, decide)
        out = bufs.out[0].double().cpu().numpy()
        for h in range(H):
            assert flg[h] == 0
            assert idx[h, :cnt[h]].tolist() == res.heads[h].idx, (t, h)
            assert rel_err(out[h], res.out[h]) <= TOL
    say("fused trajectory forced near-ties:", forced)
    assert forced <= 2
