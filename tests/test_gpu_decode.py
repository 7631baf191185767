"""GPU parity of ``dsa_decode_attention`` (split-K decode + combine) against
the fp64 oracle, element by element, at sizes that span several splits and
ragged tails; plus properties that hold at any size."""

import copy
import math
import os
import random

import numpy as np
import pytest
import torch

from oracle import step as ostep
from paper_2609_19702_amd import binding as B
from paper_2609_19702_amd import synth
from tests.gpu_util import DEV, TOL, dot_band, rel_err, request_arrays, run_layer, say, states_to_buffer

pytestmark = pytest.mark.gpu

CASES = [
    # B, Hq, Hkv, d, L_p, gh, gw, N_r, N_att, outlier_frac
    (3, 8, 8, 64, 32, 16, 16, 64, 13, 0.0),
    (4, 4, 4, 128, 17, 8, 9, 40, 11, 0.0),
    (2, 8, 2, 128, 0, 10, 10, 30, 7, 0.0),
    (2, 16, 2, 64, 5, 6, 6, 20, 20, 0.0),
    (2, 4, 2, 128, 300, 12, 12, 100, 50, 0.0),
    (3, 8, 2, 128, 40, 16, 16, 64, 21, 0.01),
    (2, 2, 1, 64, 1, 5, 5, 9, 1, 0.0),
]


def make_case(case, mode, seed=0):
    Bn, Hq, Hkv, d, Lp, gh, gw, N_r, N_att, out_frac = case
    w = synth.Workload("case", 1, Bn, Hq, Hkv, d, Lp, gh, gw, N_r, outlier_frac=out_frac, seed=seed)
    kv = synth.layer_kv(w, 0, DEV)
    q = synth.layer_query(w, 0, DEV)
    rng = random.Random(seed * 7919 + Bn)
    L = gh * gw
    ts = [L - 1, rng.randrange(L)] + [rng.randrange(L) for _ in range(Bn - 2)]
    ts = ts[:Bn]
    p = B.make_params(Lp, gh, gw, N_r, N_att, mode)
    s = B.make_shape(Bn, Hq, Hkv, d)
    states = [ostep.random_states(Hkv, N_r, N_att, t, [rng.randrange(1 << 30) for _ in range(Hkv * N_r)])
              for t in ts]
    return w, kv, q, ts, p, s, states


def oracle_outputs(w, kv, q, ts, p, s, states, mode):
    outs, heads = [], []
    qn = q.to(torch.float64).cpu().numpy()
    for b, t in enumerate(ts):
        Kp, Vp, K, V = request_arrays(kv, b, w.prompt_len)
        st = copy.deepcopy(states[b]) if mode == B.MODE_DIAGONAL else None
        r = ostep.request_step(t, qn[b], Kp, Vp, K, V, 1 / math.sqrt(s.head_dim),
                               "diagonal" if mode == B.MODE_DIAGONAL else "dense", st)
        outs.append(r.out)
        heads.append(r.heads)
    return np.stack(outs), heads


@pytest.mark.parametrize("mode", [B.MODE_DIAGONAL, B.MODE_DENSE])
@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_decode_matches_oracle(case, mode):
    say("decode case", case, "mode", mode)
    w, kv, q, ts, p, s, states = make_case(case, mode)
    st_buf = states_to_buffer(p, s, states, ts)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    bufs = run_layer(p, s, q, kv, pos, st_buf)
    torch.cuda.synchronize()
    out = bufs.out.cpu().numpy().astype(np.float64)
    ref, heads = oracle_outputs(w, kv, q, ts, p, s, states, mode)
    g = s.num_q_heads // s.num_kv_heads
    worst = 0.0
    for b in range(s.batch):
        for h in range(s.num_q_heads):
            e = rel_err(out[b, h], ref[b, h])
            worst = max(worst, e)
            assert e <= TOL, (b, h, e)
    say("  worst rel err", worst)
    if mode == B.MODE_DIAGONAL:
        cnt, flg, idx = (x.cpu().numpy() for x in B.plan_views(p, s, bufs.plan))
        wl = bufs.logits.cpu().numpy().reshape(s.batch, s.num_q_heads, -1)
        qn = q.to(torch.float64).cpu().numpy()
        for b in range(s.batch):
            Kp, Vp, K, V = request_arrays(kv, b, w.prompt_len)
            for kvh in range(s.num_kv_heads):
                pair = b * s.num_kv_heads + kvh
                hr = heads[b][kvh]
                assert idx[pair, :cnt[pair]].tolist() == hr.idx
                for i in range(g):
                    qh = qn[b, kvh * g + i]
                    band = dot_band(qh, K[kvh][hr.idx], 1 / math.sqrt(s.head_dim)) + 1e-6
                    got = wl[b, kvh * g + i, :len(hr.idx)]
                    assert np.all(np.abs(got - hr.window_logits[i]) <= band + 4e-7 * np.abs(got))


def test_dense_equals_identity_gather_bitwise():
    """Nothing skipped (N_att = N_r >= L_dec): the gathered path reads the same
    rows in the same order as the dense path, so the outputs are identical."""
    case = (3, 8, 4, 128, 24, 6, 7, 64, 64, 0.0)
    w, kv, q, ts, p, s, states = make_case(case, B.MODE_DIAGONAL, seed=3)
    st_buf = states_to_buffer(p, s, states, ts)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    a = run_layer(p, s, q, kv, pos, st_buf).out.clone()
    pd = B.make_params(p.prompt_len, p.grid_h, p.grid_w, p.window, p.n_att, B.MODE_DENSE)
    d = run_layer(pd, s, q, kv, pos).out.clone()
    assert torch.equal(a, d)


def test_constant_values_and_unused_slot():
    case = (3, 4, 4, 64, 10, 8, 8, 32, 9, 0.0)
    w, kv, q, ts, p, s, states = make_case(case, B.MODE_DIAGONAL, seed=5)
    kv.v.fill_(1.0)
    ts = [ts[0], -1, 5]
    states[1] = ostep.random_states(s.num_kv_heads, p.window, p.n_att, 0, [])
    states[2] = ostep.random_states(s.num_kv_heads, p.window, p.n_att, 5, list(range(1, 99)))
    st_buf = states_to_buffer(p, s, states, [max(t, 0) for t in ts])
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    out = run_layer(p, s, q, kv, pos, st_buf).out.cpu()
    assert torch.allclose(out[0], torch.ones_like(out[0]), atol=2e-6)
    assert torch.all(out[1] == 0)
    assert torch.allclose(out[2], torch.ones_like(out[2]), atol=2e-6)


def test_split_size_invariance():
    """The same request merged from different numbers of splits gives the
    same attention (within fp32) and matches the oracle.  The split rule
    depends only on the shape, so the request is placed in batches of 1, 32
    and 128 copies: the smaller the batch, the more splits per request."""
    case = (1, 8, 2, 128, 300, 12, 12, 100, 50, 0.0)
    w, kv, q, ts, p, s, states = make_case(case, B.MODE_DENSE, seed=9)
    ref, _ = oracle_outputs(w, kv, q, ts, p, s, states, B.MODE_DENSE)
    outs, splits = [], []
    for nb in (1, 32, 128):
        sb = B.make_shape(nb, s.num_q_heads, s.num_kv_heads, s.head_dim)
        kvb = synth.LayerKV(kv.k.expand(nb, -1, -1, -1).contiguous(),
                            kv.v.expand(nb, -1, -1, -1).contiguous(), kv.rows)
        qb = q.expand(nb, -1, -1).contiguous()
        info = B.launch_info(p, sb)
        splits.append(info.max_splits)
        say("batch", nb, "splits", info.max_splits)
        pos = torch.tensor(ts * nb, dtype=torch.int32, device=DEV)
        o = run_layer(p, sb, qb, kvb, pos).out.cpu().double()
        for b in range(nb):
            assert torch.equal(o[b], o[0])
        outs.append(o[0])
    assert len(set(splits)) == 3
    for o in outs:
        assert (o - outs[0]).abs().max() <= 1e-5 * outs[0].abs().max()
        for h in range(s.num_q_heads):
            assert rel_err(o[h].numpy(), ref[0, h]) <= TOL


def test_token_major_layout_with_row_base():
    """A ragged token-major cache addressed through per-request row bases
    gives the same result as the head-major cache."""
    case = (3, 4, 2, 64, 6, 5, 5, 12, 4, 0.0)
    w, kv, q, ts, p, s, states = make_case(case, B.MODE_DIAGONAL, seed=11)
    st_buf = states_to_buffer(p, s, states, ts)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    ref = run_layer(p, s, q, kv, pos, st_buf).out.clone()
    rows = [w.prompt_len + t + 1 for t in ts]
    Hkv, d = s.num_kv_heads, s.head_dim
    packed_k = torch.cat([kv.k[b, :, :rows[b]].transpose(0, 1).reshape(-1) for b in range(s.batch)])
    packed_v = torch.cat([kv.v[b, :, :rows[b]].transpose(0, 1).reshape(-1) for b in range(s.batch)])
    base = torch.tensor(np.cumsum([0] + [r * Hkv * d for r in rows[:-1]]), dtype=torch.int64, device=DEV)
    lay = B.KVLayout(base.data_ptr(), 0, d, Hkv * d, 0)
    bufs = B.alloc_buffers(p, s, DEV)
    B.plan(p, s, pos, st_buf, bufs.plan)
    B.decode_attention(p, s, q, packed_k, packed_v, lay, pos, bufs.plan, 1 / math.sqrt(d),
                       bufs.out, None, bufs.workspace)
    assert torch.equal(bufs.out, ref)


def test_decode_argument_errors():
    case = (2, 4, 4, 64, 300, 12, 12, 100, 50, 0.0)
    w, kv, q, ts, p, s, states = make_case(case, B.MODE_DENSE)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    bufs = B.alloc_buffers(p, s, DEV)
    lay = B.kv_layout(kv.k)
    assert B.workspace_bytes(p, s) > 0
    with pytest.raises(B.DSAError) as e:
        B.decode_attention(p, s, q, kv.k, kv.v, lay, pos, None, 0.125, bufs.out, None, None)
    assert e.value.status == B.ERR_WORKSPACE
    pdg = B.make_params(300, 12, 12, 100, 50, B.MODE_DIAGONAL)
    with pytest.raises(B.DSAError) as e:
        B.decode_attention(pdg, s, q, kv.k, kv.v, lay, pos, None, 0.125, bufs.out, None,
                           bufs.workspace)
    assert e.value.status == B.ERR_INVALID_ARG
    bad = B.KVLayout(None, lay.stride_batch, lay.stride_head, 60, 0)
    with pytest.raises(B.DSAError) as e:
        B.decode_attention(p, s, q, kv.k, kv.v, bad, pos, None, 0.125, bufs.out, None, bufs.workspace)
    assert e.value.status == B.ERR_INVALID_ARG
