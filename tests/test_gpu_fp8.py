"""fp8 (OCP E4M3) KV caches on the GPU against the oracle.

* every finite E4M3 byte widens exactly, read back through the window logits
  (one-hot queries, unit scales) on the vector-ALU and the MFMA tiles;
* with unit scales an fp8 cache gives the kept sets of the bf16 cache
  holding the same values, and its outputs and window logits within fp32
  rounding (an fp8 lane loads 16 elements, a bf16 lane 8, so the sums run
  in different orders), in both modes and both tiles;
* scaled caches from the synthetic quantizer match the oracle, which decodes
  the bytes exactly and multiplies by the scales in fp64, within the
  tolerance; the fused step reproduces the separate calls bit for bit, a
  ring reproduces the linear cache bit for bit and matches the oracle;
* argument errors: scales on a bf16 cache, unknown element types."""

import copy
import math
import random

import numpy as np
import pytest
import torch

from oracle import fp8 as ofp8
from oracle import step as ostep
from paper_2609_19702_amd import binding as B
from paper_2609_19702_amd import synth
from tests.gpu_util import (DEV, TOL, check_layer_vs_oracle, dot_band, fp8_request_arrays,
                            offsets_from_buffer, rel_err, say, states_to_buffer, within_tie_band)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("Hq,Hkv,d", [(1, 1, 64), (1, 1, 128), (2, 1, 64), (4, 1, 128)])
def test_every_code_widens_exactly(Hq, Hkv, d):
    say("fp8 codes", Hq, Hkv, d)
    L = 256
    p = B.make_params(0, 16, 16, L, L, B.MODE_DIAGONAL)
    s = B.make_shape(1, Hq, Hkv, d)
    codes = torch.arange(256, dtype=torch.int32)
    codes[0x7F] = 0
    codes[0xFF] = 0
    k = torch.zeros((1, Hkv, L, d), dtype=torch.uint8)
    k[0, :, :, 0] = codes.to(torch.uint8)
    k = k.to(DEV)
    v = torch.zeros_like(k)
    q = torch.zeros((1, Hq, d), dtype=torch.bfloat16)
    q[:, :, 0] = 1.0
    q = q.to(DEV)
    bufs = B.alloc_buffers(p, s, DEV)
    pos = torch.tensor([L - 1], dtype=torch.int32, device=DEV)
    B.plan(p, s, pos, bufs.state, bufs.plan)
    B.decode_attention(p, s, q, k, v, B.kv_layout(k), pos, bufs.plan, 1.0, bufs.out, bufs.logits,
                       bufs.workspace)
    torch.cuda.synchronize()
    got = bufs.logits.view(Hq, L).cpu().numpy().astype(np.float64)
    want = ofp8.decode_e4m3(codes.numpy())
    for h in range(Hq):
        assert np.array_equal(got[h], want), h


CASES = [
    # B, Hq, Hkv, d, L_p, gh, gw, N_r, N_att
    (3, 8, 8, 64, 32, 16, 16, 64, 13),
    (2, 8, 2, 128, 0, 10, 10, 30, 7),
    (2, 4, 2, 128, 300, 12, 12, 100, 50),
    (3, 8, 2, 128, 40, 16, 16, 64, 21),
    (2, 16, 2, 64, 5, 6, 6, 20, 20),
]


def make_case(case, mode, seed):
    Bn, Hq, Hkv, d, Lp, gh, gw, N_r, N_att = case
    w = synth.Workload("fp8", 1, Bn, Hq, Hkv, d, Lp, gh, gw, N_r, outlier_frac=0.01, seed=seed)
    kv = synth.to_fp8(synth.layer_kv(w, 0, DEV))
    q = synth.layer_query(w, 0, DEV)
    rng = random.Random(seed * 31 + Bn)
    L = gh * gw
    ts = [L - 1] + [rng.randrange(L) for _ in range(Bn - 1)]
    p = B.make_params(Lp, gh, gw, N_r, N_att, mode)
    s = B.make_shape(Bn, Hq, Hkv, d)
    states = [ostep.random_states(Hkv, N_r, N_att, t, [rng.randrange(1 << 30) for _ in range(Hkv * N_r)])
              for t in ts]
    return w, kv, q, ts, p, s, states


@pytest.mark.parametrize("mode", [B.MODE_DIAGONAL, B.MODE_DENSE])
@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_fp8_matches_oracle(case, mode):
    say("fp8 case", case, "mode", mode)
    w, kv, q, ts, p, s, states = make_case(case, mode, seed=2)
    Hkv, g = s.num_kv_heads, s.num_q_heads // s.num_kv_heads
    scale = 1 / math.sqrt(s.head_dim)
    st_buf = states_to_buffer(p, s, states, ts)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    bufs = B.alloc_buffers(p, s, DEV)
    lay = B.kv_layout(kv.k, k_scale=kv.k_scale, v_scale=kv.v_scale)
    sparse = mode != B.MODE_DENSE
    B.plan(p, s, pos, st_buf if sparse else None, bufs.plan)
    B.decode_attention(p, s, q, kv.k, kv.v, lay, pos, bufs.plan if sparse else None, scale,
                       bufs.out, bufs.logits if sparse else None, bufs.workspace)
    torch.cuda.synchronize()
    out = bufs.out.cpu().numpy().astype(np.float64)
    qn = q.to(torch.float64).cpu().numpy()
    cnt, _, idx = (x.cpu().numpy() for x in B.plan_views(p, s, bufs.plan))
    wl = bufs.logits.cpu().numpy().reshape(s.batch, s.num_q_heads, -1) if sparse else None
    worst = 0.0
    for b, t in enumerate(ts):
        Kp, Vp, K, V = fp8_request_arrays(kv, b, w.prompt_len, Hkv)
        st = copy.deepcopy(states[b]) if sparse else None
        r = ostep.request_step(t, qn[b], Kp, Vp, K, V, scale, "diagonal" if sparse else "dense", st)
        for h in range(s.num_q_heads):
            e = rel_err(out[b, h], r.out[h])
            worst = max(worst, e)
            assert e <= TOL, (b, h, e)
        if sparse:
            for kvh in range(Hkv):
                pair = b * Hkv + kvh
                hr = r.heads[kvh]
                assert idx[pair, :cnt[pair]].tolist() == hr.idx
                for i in range(g):
                    qh = qn[b, kvh * g + i]
                    band = dot_band(qh, K[kvh][hr.idx], scale) + 1e-6
                    got = wl[b, kvh * g + i, :len(hr.idx)]
                    assert np.all(np.abs(got - hr.window_logits[i]) <= band + 4e-7 * np.abs(got))
    say("  worst rel err", worst)


@pytest.mark.parametrize("mode", [B.MODE_DIAGONAL, B.MODE_DENSE])
@pytest.mark.parametrize("case", CASES[:4], ids=[str(c) for c in CASES[:4]])
def test_unit_scale_fp8_matches_bf16(case, mode):
    """Bytes with unit scales (given, or absent) and the bf16 cache of their
    values: the same kept sets and, within fp32 rounding, the same outputs
    and window logits.  (Not bit for bit: an fp8 lane loads 16 elements, a
    bf16 lane 8, so the two sum in different orders.)  A unit scale and no
    scale give identical bits.  Each selection either agrees or both picks
    lie inside the certified tie band."""
    say("fp8 ~ bf16", case, mode)
    w, kv, q, ts, p, s, states = make_case(case, mode, seed=4)
    kb = kv.k.view(torch.float8_e4m3fn).to(torch.bfloat16)
    vb = kv.v.view(torch.float8_e4m3fn).to(torch.bfloat16)
    st_buf = states_to_buffer(p, s, states, ts)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    sparse = mode != B.MODE_DENSE
    ones = torch.ones(s.batch * s.num_kv_heads, dtype=torch.float32, device=DEV)
    outs = []
    for k, v, sc in ((kb, vb, None), (kv.k, kv.v, None), (kv.k, kv.v, ones)):
        bufs = B.alloc_buffers(p, s, DEV)
        st = st_buf.clone()
        lay = B.kv_layout(k, k_scale=sc, v_scale=sc)
        if sparse:
            B.decode_step(p, s, q, k, v, lay, pos, st, bufs.plan, 0.125, bufs.out, bufs.logits,
                          bufs.workspace)
        else:
            B.decode_attention(p, s, q, k, v, lay, pos, None, 0.125, bufs.out, None, bufs.workspace)
        torch.cuda.synchronize()
        outs.append((bufs.out.clone(), st.clone(), bufs.logits.clone(), bufs.plan.clone()))
    assert all(torch.equal(x, y) for x, y in zip(outs[1], outs[2]))
    (o0, s0, l0, p0), (o1, s1, l1, p1) = outs[0], outs[1]
    d = (o1 - o0).abs().amax(dim=-1) / o0.abs().amax(dim=-1).clamp_min(1e-30)
    assert d.max().item() <= 1e-5, d.max().item()
    if not sparse:
        return
    assert torch.equal(p0, p1)
    assert (l1 - l0).abs().max().item() <= 1e-5 * max(1.0, l0.abs().max().item())
    if torch.equal(s0, s1):
        return
    # a selection that differs: both picks must be near ties of the exact scores
    Hkv, g = s.num_kv_heads, s.num_q_heads // s.num_kv_heads
    cnt, _, idx = (x.cpu().numpy() for x in B.plan_views(p, s, p0))
    _, _, off0 = offsets_from_buffer(p, s, s0)
    c1, _, off1 = offsets_from_buffer(p, s, s1)
    qn = q.double().cpu().numpy()
    for b, t in enumerate(ts):
        Kp, Vp, K, V = fp8_request_arrays(kv, b, w.prompt_len, Hkv)
        k_slot = t - (p.n_att - 1)
        for h in range(Hkv):
            pair = b * Hkv + h
            if not (0 <= k_slot < off0.shape[1]) or off0[pair, k_slot] == off1[pair, k_slot]:
                continue
            kept = idx[pair, :cnt[pair]].tolist()
            j0 = kept.index(t - int(off0[pair, k_slot]))
            j1 = kept.index(t - int(off1[pair, k_slot]))
            qg = qn[b][h * g:(h + 1) * g]
            from oracle.attention import select
            j_ref, _ = select(qg, K[h][kept], 0.125)
            assert within_tie_band(qg, K[h][kept], 0.125, j0, j_ref)
            assert within_tie_band(qg, K[h][kept], 0.125, j1, j_ref)


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_fp8_fused_equals_separate(case):
    say("fp8 fused", case)
    w, kv, q, ts, p, s, states = make_case(case, B.MODE_DIAGONAL, seed=6)
    st0 = states_to_buffer(p, s, states, ts)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    lay = B.kv_layout(kv.k, k_scale=kv.k_scale, v_scale=kv.v_scale)
    a, b = B.alloc_buffers(p, s, DEV), B.alloc_buffers(p, s, DEV)
    sa, sb = st0.clone(), st0.clone()
    B.decode_step(p, s, q, kv.k, kv.v, lay, pos, sa, a.plan, 0.1, a.out, a.logits, a.workspace)
    B.plan(p, s, pos, sb, b.plan)
    B.decode_attention(p, s, q, kv.k, kv.v, lay, pos, b.plan, 0.1, b.out, b.logits, b.workspace)
    B.select(p, s, pos, b.plan, b.logits, sb)
    torch.cuda.synchronize()
    assert torch.equal(a.out, b.out) and torch.equal(sa, sb) and torch.equal(a.plan, b.plan)


def test_fp8_ring_equals_linear():
    Bn, Hq, Hkv, d, Lp, gh, gw, N_r, N_att, R = 5, 8, 2, 128, 12, 10, 10, 30, 7, 33
    w = synth.Workload("fp8_ring", 1, Bn, Hq, Hkv, d, Lp, gh, gw, N_r, outlier_frac=0.01)
    kv = synth.to_fp8(synth.layer_kv(w, 0, DEV))
    q = synth.layer_query(w, 0, DEV)
    rng = random.Random(3)
    L = gh * gw
    ts = [L - 1, N_r - 1, N_att - 1, 0, rng.randrange(L)]
    p = B.make_params(Lp, gh, gw, N_r, N_att)
    s = B.make_shape(Bn, Hq, Hkv, d)
    states = [ostep.random_states(Hkv, N_r, N_att, t, [rng.randrange(1 << 30) for _ in range(Hkv * N_r)])
              for t in ts]
    st0 = states_to_buffer(p, s, states, ts)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    rk = kv.k[:, :, :Lp + R].clone()
    rv = kv.v[:, :, :Lp + R].clone()
    rk[:, :, Lp:] = 0x7E  # 448: a read of a slot the step must not read would show
    rv[:, :, Lp:] = 0xFE
    for b, t in enumerate(ts):
        for j in range(max(0, t - R + 1), t + 1):
            rk[b, :, Lp + j % R] = kv.k[b, :, Lp + j]
            rv[b, :, Lp + j % R] = kv.v[b, :, Lp + j]
    res = []
    for k, v, ring in ((kv.k, kv.v, 0), (rk, rv, R)):
        bufs = B.alloc_buffers(p, s, DEV)
        st = st0.clone()
        lay = B.kv_layout(k, ring_rows=ring, k_scale=kv.k_scale, v_scale=kv.v_scale)
        B.decode_step(p, s, q, k, v, lay, pos, st, bufs.plan, 0.1, bufs.out, bufs.logits,
                      bufs.workspace)
        torch.cuda.synchronize()
        res.append((bufs.out.clone(), st.clone(), bufs.plan.clone(), bufs.logits.clone()))
    assert torch.equal(res[0][0], res[1][0]) and torch.equal(res[0][1], res[1][1])
    # the ring's results against the oracle on the dequantized cache
    arrays = [fp8_request_arrays(kv, b, Lp, Hkv) for b in range(Bn)]
    o1, s1, p1, l1 = res[1]
    assert check_layer_vs_oracle(p, s, q, arrays, ts, states, p1, o1, s1, l1, scale=0.1) <= 1


def test_fp8_argument_errors():
    p = B.make_params(4, 4, 4, 8, 4)
    s = B.make_shape(2, 4, 2, 64)
    w = synth.Workload("fp8_err", 1, 2, 4, 2, 64, 4, 4, 4, 8)
    kv = synth.layer_kv(w, 0, DEV)
    q = synth.layer_query(w, 0, DEV)
    bufs = B.alloc_buffers(p, s, DEV)
    pos = torch.tensor([3, 9], dtype=torch.int32, device=DEV)
    B.plan(p, s, pos, bufs.state, bufs.plan)
    ones = torch.ones(4, dtype=torch.float32, device=DEV)
    bad = [B.kv_layout(kv.k, k_scale=ones), B.kv_layout(kv.k, v_scale=ones)]
    odd = B.kv_layout(kv.k)
    odd.dtype = 7
    bad.append(odd)
    for lay in bad:
        with pytest.raises(B.DSAError) as e:
            B.decode_attention(p, s, q, kv.k, kv.v, lay, pos, bufs.plan, 0.1, bufs.out, None,
                               bufs.workspace)
        assert e.value.status == B.ERR_INVALID_ARG
