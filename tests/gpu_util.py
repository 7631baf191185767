"""Helpers shared by the GPU parity tests: running one layer step through the
C ABI, and moving selection states between the oracle's form (Algorithm 1's
``skip_idx`` list) and the library's form (offsets in append order)."""

from __future__ import annotations

import math
import sys

import numpy as np
import torch

from oracle import alg1
from oracle import fp8 as ofp8
from oracle.tieband import dot_band, logit_band, within_tie_band  # noqa: F401
from paper_2609_19702_amd import binding as B

DEV = "cuda"
TOL = 2e-3  # max |o_gpu - o_ref| / max |o_ref| per (request, query head)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def states_to_buffer(p, s, states, t_list, device=DEV):
    """Library state buffer holding the oracle states ``states[b][h]`` (each
    after steps ``0 .. t_list[b]-1``).  With sinks the oracle's state counts
    steps from the first position after the sinks; offsets are the same in
    both frames."""
    buf = torch.zeros(B.state_bytes(p, s), dtype=torch.uint8)
    if B.state_layout(p, s).cap == 0:  # nothing is ever selected: empty lists
        return buf.to(device)
    cnt, flg, off = B.state_views(p, s, buf)
    Hkv = s.num_kv_heads
    for b, per_head in enumerate(states):
        for h, st in enumerate(per_head):
            pair = b * Hkv + h
            t_state = t_list[b] - p.sinks  # steps the state has seen
            d = alg1.offsets_of(st, t_state - 1) if t_state > 0 else []
            assert len(d) == len(st.skip_idx)
            cnt[pair] = len(d)
            if d:
                off[pair, :len(d)] = torch.tensor(np.array(d, dtype=np.uint16).view(np.int16))
    return buf.to(device)


def offsets_from_buffer(p, s, buf):
    cnt, flg, off = B.state_views(p, s, buf.cpu())
    off = off.numpy().view(np.uint16)
    return cnt.numpy().copy(), flg.numpy().copy(), off


def run_layer(p, s, q, kv, pos, state=None, bufs=None, logits=True, stream=None):
    """plan + decode (+ combine) for one layer; returns the buffers."""
    if bufs is None:
        bufs = B.alloc_buffers(p, s, DEV)
    sparse = p.mode != B.MODE_DENSE
    B.plan(p, s, pos, state if sparse else None, bufs.plan, stream=stream)
    B.decode_attention(p, s, q, kv.k, kv.v, B.kv_layout(kv.k), pos,
                       bufs.plan if sparse else None,
                       1.0 / math.sqrt(s.head_dim), bufs.out,
                       bufs.logits if (logits and sparse) else None,
                       bufs.workspace, stream=stream)
    return bufs


def rel_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    den = np.abs(ref).max()
    return float(np.abs(gpu - ref).max() / (den if den > 0 else 1.0))


def request_arrays(kv, b, Lp):
    """fp64 (Kp, Vp, K, V) of request b from a head-major bf16 cache."""
    k = kv.k[b].to(torch.float64).cpu().numpy()
    v = kv.v[b].to(torch.float64).cpu().numpy()
    return k[:, :Lp], v[:, :Lp], k[:, Lp:], v[:, Lp:]


def fp8_request_arrays(kv, b, Lp, Hkv):
    """fp64 (Kp, Vp, K, V) of request b of an fp8 cache, decoded and scaled
    by the oracle."""
    kc = kv.k[b].cpu().numpy()
    vc = kv.v[b].cpu().numpy()
    ks = kv.k_scale.cpu().numpy()[b * Hkv:(b + 1) * Hkv]
    vs = kv.v_scale.cpu().numpy()[b * Hkv:(b + 1) * Hkv]
    k = np.stack([ofp8.dequantize(kc[h], ks[h]) for h in range(Hkv)])
    v = np.stack([ofp8.dequantize(vc[h], vs[h]) for h in range(Hkv)])
    return k[:, :Lp], v[:, :Lp], k[:, Lp:], v[:, Lp:]


def check_layer_vs_oracle(p, s, q, arrays, ts, states, plan_buf, out, state_after=None,
                          logits=None, scale=None):
    """One layer step of the library against the oracle's step from the same
    selection states: kept sets bit for bit, every query head's output
    within ``TOL``, the window logits (when given) within their fp32 bound,
    and every phase-2 pick the library stored equal to the oracle's argmin
    or inside the certified tie band (the oracle then adopts it).

    ``arrays[b]`` holds request b's ``(Kp, Vp, K, V)`` as fp64 values of the
    cache (dequantized for fp8); ``states[b]`` its per-KV-head oracle
    states before the step (not modified).  Returns the number of near-tie
    picks adopted."""
    import copy
    from oracle import step as ostep
    mode = {B.MODE_DENSE: "dense", B.MODE_DIAGONAL: "diagonal",
            B.MODE_WINDOW: "streaming"}[p.mode]
    if p.mode == B.MODE_DIAGONAL and p.sinks:
        mode = "diagonal_sink"
    scale = 1.0 / math.sqrt(s.head_dim) if scale is None else scale
    Hkv, g = s.num_kv_heads, s.num_q_heads // s.num_kv_heads
    sparse = p.mode != B.MODE_DENSE
    if sparse:
        cnt, flg, idx = (x.cpu().numpy() for x in B.plan_views(p, s, plan_buf))
    if state_after is not None:
        scnt, sflg, soff = offsets_from_buffer(p, s, state_after)
        assert not sflg.any()
    o = out.double().cpu().numpy()
    qn = q.double().cpu().numpy()
    wl = None if logits is None else logits.view(s.batch, s.num_q_heads, -1).cpu().numpy()
    forced = 0
    for b, t in enumerate(ts):
        if t < 0:
            assert not o[b].any()
            continue
        Kp, Vp, K, V = arrays[b]

        def decide(kvh, t_, idx_, j_ref, sigma, b=b):
            nonlocal forced
            if state_after is None:
                return j_ref
            pair = b * Hkv + kvh
            k = t_ - (p.n_att - 1)
            assert scnt[pair] == k + 1, (b, kvh, t_, scnt[pair])
            j_gpu = idx_.index(t_ - int(soff[pair, k]))
            if j_gpu != j_ref:
                qg = qn[b][kvh * g:(kvh + 1) * g]
                assert within_tie_band(qg, K[kvh][idx_], scale, j_gpu, j_ref), (b, kvh, t_)
                forced += 1
            return j_gpu

        st = copy.deepcopy(states[b]) if states is not None and sparse else None
        res = ostep.request_step(t, qn[b], Kp, Vp, K, V, scale, mode, st, decide, p.sinks)
        for h in range(Hkv):
            pair = b * Hkv + h
            if sparse:
                assert flg[pair] == 0, (b, h, flg[pair])
                assert idx[pair, :cnt[pair]].tolist() == res.heads[h].idx, (b, h, t)
                if wl is not None:
                    kept = res.heads[h].idx
                    for i in range(g):
                        ref = res.heads[h].window_logits[i]
                        band = logit_band(qn[b][h * g + i], K[h][kept], scale) + 1e-7
                        got = wl[b, h * g + i, :len(kept)]
                        assert (np.abs(got - ref) <= band).all(), (b, h, i)
            for i in range(g):
                e = rel_err(o[b, h * g + i], res.out[h * g + i])
                assert e <= TOL, (b, h * g + i, e)
    return forced


def c_replay_states(N_r, N_att, L, ts, Hkv, rng, threads=8):
    """Algorithm 1 states of every (request, KV head) before step ``ts[b]``,
    each drawn by the C oracle's literal replay with random choices (fast
    enough for windows of tens of thousands of positions).  Returns
    ``(states, kept)``: ``states[b][h]`` an ``oracle.alg1.HeadState`` equal
    to the literal state after steps ``0 .. t-1``, and ``kept[b][h]`` the
    positions step ``t`` attends."""
    from concurrent.futures import ThreadPoolExecutor
    from oracle import coracle
    jobs = [(b, h, max(t, 0), [rng.randrange(1 << 40) for _ in range(N_r)])
            for b, t in enumerate(ts) for h in range(Hkv)]

    def one(job):
        b, h, t, rand = job
        st, kept = coracle.replay_head(N_r, N_att, L, t, rand)
        return b, h, st, kept

    states = [[None] * Hkv for _ in ts]
    kept = [[None] * Hkv for _ in ts]
    with ThreadPoolExecutor(threads) as ex:
        for b, h, st, kp in ex.map(one, jobs):
            states[b][h], kept[b][h] = st, kp
    return states, kept
