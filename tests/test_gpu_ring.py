"""Ring-buffer KV (physical eviction, section 4 "Cost analysis"): a cache of
L_p + R rows per (request, KV head) in which decode position j lives in slot
j mod R.  Its plans, outputs, window logits and stored selections are
checked against the oracle's step from the same selection states (kept sets
bit for bit, outputs within the tolerance, picks equal to the oracle's
argmin or inside the certified tie band), and must equal the linear cache's
results bit for bit.  Only the live window of each request is copied into
the ring; every other slot holds a large decoy value, so a read of an
evicted row would show."""

import random

import numpy as np
import pytest
import torch

from oracle import step as ostep
from paper_2609_19702_amd import binding as B
from paper_2609_19702_amd import synth
from tests.gpu_util import DEV, check_layer_vs_oracle, request_arrays, say, states_to_buffer

pytestmark = pytest.mark.gpu

CASES = [
    # B, Hq, Hkv, d, L_p, gh, gw, N_r, N_att, ring
    (6, 8, 8, 64, 20, 12, 12, 40, 10, 40),
    (6, 8, 8, 64, 0, 12, 12, 40, 10, 47),
    (5, 8, 2, 128, 33, 10, 10, 30, 7, 30),
    (4, 16, 2, 64, 8, 9, 9, 24, 24, 29),
]


def to_ring(kv, Lp, ts, R):
    k = kv.k[:, :, :Lp + R].clone()
    v = kv.v[:, :, :Lp + R].clone()
    k[:, :, Lp:] = 1e4
    v[:, :, Lp:] = -1e4
    for b, t in enumerate(ts):
        if t < 0:
            continue
        for j in range(max(0, t - R + 1), t + 1):
            k[b, :, Lp + j % R] = kv.k[b, :, Lp + j]
            v[b, :, Lp + j % R] = kv.v[b, :, Lp + j]
    return k, v


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_ring_equals_linear(case, fused):
    Bn, Hq, Hkv, d, Lp, gh, gw, N_r, N_att, R = case
    say("ring", case, "fused" if fused else "separate")
    rng = random.Random(R * 7 + Bn)
    L = gh * gw
    ts = [L - 1, N_r - 1, N_att - 1] + [rng.randrange(L) for _ in range(Bn - 3)]
    ts[-1] = -1
    w = synth.Workload("ring", 1, Bn, Hq, Hkv, d, Lp, gh, gw, N_r, outlier_frac=0.01)
    kv = synth.layer_kv(w, 0, DEV)
    q = synth.layer_query(w, 0, DEV)
    p = B.make_params(Lp, gh, gw, N_r, N_att)
    s = B.make_shape(Bn, Hq, Hkv, d)
    states = [ostep.random_states(Hkv, N_r, N_att, max(t, 0), [rng.randrange(1 << 30) for _ in range(Hkv * N_r)])
              for t in ts]
    st0 = states_to_buffer(p, s, states, [max(t, 0) for t in ts])
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    rk, rv = to_ring(kv, Lp, ts, R)
    results = []
    for k, v, ring in ((kv.k, kv.v, 0), (rk, rv, R)):
        bufs = B.alloc_buffers(p, s, DEV)
        st = st0.clone()
        lay = B.kv_layout(k, ring_rows=ring)
        if fused:
            B.decode_step(p, s, q, k, v, lay, pos, st, bufs.plan, 0.125, bufs.out, bufs.logits,
                          bufs.workspace)
        else:
            B.plan(p, s, pos, st, bufs.plan)
            B.decode_attention(p, s, q, k, v, lay, pos, bufs.plan, 0.125, bufs.out, bufs.logits,
                               bufs.workspace)
            B.select(p, s, pos, bufs.plan, bufs.logits, st)
        torch.cuda.synchronize()
        results.append((bufs.out.clone(), st.clone(), bufs.plan.clone(), bufs.logits.clone()))
    (o0, s0, p0, _), (o1, s1, p1, l1) = results
    assert torch.isfinite(o1).all()
    arrays = [request_arrays(kv, b, Lp) for b in range(Bn)]
    forced = check_layer_vs_oracle(p, s, q, arrays, ts, states, p1, o1, s1, l1, scale=0.125)
    assert forced <= 1
    assert torch.equal(o0, o1)
    assert torch.equal(s0, s1)
    assert torch.equal(p0, p1)


def test_ring_too_small_rejected():
    w = synth.Workload("ring_bad", 1, 2, 4, 4, 64, 4, 6, 6, 12)
    kv = synth.layer_kv(w, 0, DEV)
    q = synth.layer_query(w, 0, DEV)
    p = B.make_params(4, 6, 6, 12, 5)
    s = B.make_shape(2, 4, 4, 64)
    bufs = B.alloc_buffers(p, s, DEV)
    pos = torch.tensor([3, 20], dtype=torch.int32, device=DEV)
    B.plan(p, s, pos, bufs.state, bufs.plan)
    with pytest.raises(B.DSAError) as e:
        B.decode_attention(p, s, q, kv.k, kv.v, B.kv_layout(kv.k, ring_rows=11), pos, bufs.plan,
                           0.125, bufs.out, None, bufs.workspace)
    assert e.value.status == B.ERR_INVALID_ARG
    pd = B.make_params(4, 6, 6, 12, 5, B.MODE_DENSE)
    with pytest.raises(B.DSAError) as e:  # dense mode reads every decode row
        B.decode_attention(pd, s, q, kv.k, kv.v, B.kv_layout(kv.k, ring_rows=20), pos, None,
                           0.125, bufs.out, None, B.alloc_buffers(pd, s, DEV).workspace)
    assert e.value.status == B.ERR_INVALID_ARG
