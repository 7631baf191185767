"""GPU parity of ``dsa_plan``: the kept decode positions must equal the
oracle's Algorithm 1 ``idx`` bit for bit, given the same selection history.

Histories are drawn by the oracle itself (Algorithm 1 with seeded random
choices standing in for the argmin), converted to the library's offset form
and uploaded; the plan of step ``t_b`` is then compared with the oracle's
``idx`` at ``t_b``."""

import copy
import random

import numpy as np
import pytest
import torch

from oracle import alg1, step as ostep
from paper_2609_19702_amd import binding as B
from tests.gpu_util import DEV, say, states_to_buffer

pytestmark = pytest.mark.gpu


def edge_positions(L_dec, N_r, N_att):
    ts = {0, N_att - 2, N_att - 1, N_att, N_r - 2, N_r - 1, N_r, N_r + 1, L_dec - 1, L_dec // 2}
    return sorted(t for t in ts if 0 <= t < L_dec)


CASES = [
    # B, Hkv, L_p, gh, gw, N_r, N_att
    (4, 8, 32, 16, 16, 64, 13),
    (3, 3, 0, 7, 9, 20, 1),
    (2, 2, 5, 8, 8, 16, 16),
    (6, 4, 120, 24, 24, 128, 29),
    (2, 2, 256, 24, 24, 256, 29),
    (1, 2, 256, 64, 64, 512, 205),
    (5, 1, 3, 3, 3, 9, 4),
    (2, 3, 0, 40, 40, 100, 99),
]


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_plan_matches_oracle(case):
    Bn, Hkv, Lp, gh, gw, N_r, N_att = case
    L_dec = gh * gw
    say("plan case", case)
    rng = random.Random(hash(case) & 0xFFFF)
    edges = edge_positions(L_dec, N_r, N_att)
    t_list = [edges[i % len(edges)] if i < len(edges) else rng.randrange(L_dec) for i in range(Bn * 2)]
    for rep in range(2):
        ts = t_list[rep * Bn:(rep + 1) * Bn]
        p = B.make_params(Lp, gh, gw, N_r, N_att, B.MODE_DIAGONAL)
        s = B.make_shape(Bn, Hkv, Hkv, 64)
        states = []
        for b, t in enumerate(ts):
            ints = [rng.randrange(1 << 30) for _ in range(Hkv * N_r)]
            states.append(ostep.random_states(Hkv, N_r, N_att, t, ints))
        st_buf = states_to_buffer(p, s, states, ts)
        plan = torch.zeros(B.plan_bytes(p, s), dtype=torch.uint8, device=DEV)
        pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
        B.plan(p, s, pos, st_buf, plan)
        cnt, flg, idx = (x.cpu().numpy() for x in B.plan_views(p, s, plan))
        for b, t in enumerate(ts):
            for h in range(Hkv):
                rec = copy.deepcopy(states[b][h]).step(t, lambda t_, i_: 0)
                pair = b * Hkv + h
                assert flg[pair] == 0, (b, h, t, flg[pair])
                assert cnt[pair] == len(rec.idx) == min(t + 1, N_att)
                assert idx[pair, :cnt[pair]].tolist() == rec.idx, (b, h, t)


def test_worked_example_through_gpu(golden_dir):
    import json
    import os
    fx = json.load(open(os.path.join(golden_dir, "worked_example.json")))
    N_r, N_att = fx["N_r"], fx["N_att"]
    picks = {3: 0, 4: 2, 5: 1, 6: 6}  # paper's picks at t=3,4; t=5,6 any valid choice
    p = B.make_params(2, 3, 4, N_r, N_att, B.MODE_DIAGONAL)
    s = B.make_shape(1, 1, 1, 64)
    st = alg1.HeadState(N_r, N_att)
    for t in range(12):
        buf = states_to_buffer(p, s, [[st]], [t])
        plan = torch.zeros(B.plan_bytes(p, s), dtype=torch.uint8, device=DEV)
        B.plan(p, s, torch.tensor([t], dtype=torch.int32, device=DEV), buf, plan)
        cnt, flg, idx = (x.cpu().numpy() for x in B.plan_views(p, s, plan))
        rec = st.step(t, alg1.by_position(picks))
        assert idx[0, :cnt[0]].tolist() == rec.idx
        if str(t) in fx["steps"]:
            assert rec.idx == fx["steps"][str(t)]["idx"]


def test_dense_plan_and_flags():
    Lp, gh, gw, N_r, N_att = 4, 5, 6, 12, 5
    L_dec = gh * gw
    s = B.make_shape(6, 2, 2, 64)
    pos = torch.tensor([-1, 0, 7, L_dec - 1, L_dec + 9, 11], dtype=torch.int32, device=DEV)
    p = B.make_params(Lp, gh, gw, N_r, N_att, B.MODE_DENSE)
    plan = torch.zeros(B.plan_bytes(p, s), dtype=torch.uint8, device=DEV)
    B.plan(p, s, pos, None, plan)
    cnt, flg, _ = (x.cpu().numpy() for x in B.plan_views(p, s, plan))
    assert cnt.reshape(6, 2)[:, 0].tolist() == [0, 1, 8, L_dec, L_dec, 12]
    assert flg.reshape(6, 2)[:, 0].tolist() == [B.FLAG_INACTIVE, 0, 0, 0, B.FLAG_POS_CLAMPED, 0]

    # diagonal: a state that is behind, an offset out of range, a clamped position
    p = B.make_params(Lp, gh, gw, N_r, N_att, B.MODE_DIAGONAL)
    st = torch.zeros(B.state_bytes(p, s), dtype=torch.uint8)
    scnt, _, soff = B.state_views(p, s, st)
    scnt[:] = 0                    # every request: no skip entries stored
    scnt[5 * 2] = 3                # request 5 (t=11 needs 7): behind
    soff[3 * 2, :7] = torch.tensor([0, 1, 2, 3, 4, 5, 6], dtype=torch.int16)
    scnt[3 * 2] = 7                # request 3 at t = L_dec-1: full list, valid
    soff[1 * 2, 0] = N_r - 1       # request 1 is at t=0: entry unused, never read
    scnt[1 * 2] = 1
    plan = torch.zeros(B.plan_bytes(p, s), dtype=torch.uint8, device=DEV)
    B.plan(p, s, pos, st.to(DEV), plan)
    cnt, flg, idx = (x.cpu().numpy() for x in B.plan_views(p, s, plan))
    f = flg.reshape(6, 2)[:, 0].tolist()
    assert f[0] == B.FLAG_INACTIVE and cnt[0] == 0
    assert f[1] == 0 and cnt[2] == 1
    assert f[3] == 0 and idx[6, :cnt[6]].tolist() == list(range(L_dec - N_r, L_dec - 7))
    assert f[4] == B.FLAG_POS_CLAMPED | B.FLAG_STATE_BEHIND
    assert f[5] == B.FLAG_STATE_BEHIND
    # bad offset in a used slot
    scnt[5 * 2] = 7
    soff[5 * 2, :7] = torch.tensor([0, 1, 2, N_r - 1, 4, 5, 6], dtype=torch.int16)
    B.plan(p, s, pos, st.to(DEV), plan)
    _, flg, _ = (x.cpu().numpy() for x in B.plan_views(p, s, plan))
    assert flg[10] == B.FLAG_BAD_OFFSET


def test_plan_rejects_small_buffer():
    p = B.make_params(4, 5, 6, 12, 5, B.MODE_DIAGONAL)
    s = B.make_shape(2, 2, 2, 64)
    st = torch.zeros(B.state_bytes(p, s), dtype=torch.uint8, device=DEV)
    small = torch.zeros(B.plan_bytes(p, s) - 4, dtype=torch.uint8, device=DEV)
    pos = torch.zeros(2, dtype=torch.int32, device=DEV)
    with pytest.raises(B.DSAError) as e:
        B.plan(p, s, pos, st, small)
    assert e.value.status == B.ERR_WORKSPACE
