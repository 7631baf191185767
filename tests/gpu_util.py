"""Helpers shared by the GPU parity tests: running one layer step through the
C ABI, and moving selection states between the oracle's form (Algorithm 1's
``skip_idx`` list) and the library's form (offsets in append order)."""

from __future__ import annotations

import math
import sys

import numpy as np
import torch

from oracle import alg1
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


def dot_band(q, keys, scale):
    """Forward-error bound of an fp32 dot product of length d, per key:
    gamma_d * scale * sum_i |q_i k_i| with gamma_d = d u / (1 - d u)."""
    d = q.shape[-1]
    u = 2.0 ** -24
    gamma = d * u / (1 - d * u)
    return gamma * scale * (np.abs(keys) @ np.abs(q))


def within_tie_band(q_group, window_keys, scale, j_gpu, j_ref) -> bool:
    """Is the GPU's argmin ``j_gpu`` as good as the oracle's ``j_ref`` up to
    the rounding the fp32 path may commit?

    Group size 1: the GPU compares fp32 logits, each within ``dot_band`` of
    the exact logit (plus the rounding of the scale multiply), so any pick
    whose exact logit exceeds the minimum by at most the two bands is valid.
    Larger groups: a logit error of at most ``beta_h`` changes each window
    softmax weight by a factor within ``exp(+-2 beta_h)``; with the fp32
    exp/divide rounding this bounds the error of the summed score."""
    q_group = np.atleast_2d(np.asarray(q_group, np.float64))
    keys = np.asarray(window_keys, np.float64)
    if j_gpu == j_ref:
        return True
    if q_group.shape[0] == 1:
        s = scale * keys @ q_group[0]
        band = dot_band(q_group[0], keys, scale) + 2.0 ** -23 * np.abs(s)
        return s[j_gpu] - s[j_ref] <= band[j_gpu] + band[j_ref]
    sig = np.zeros(len(keys))
    slack = 1e-7 * q_group.shape[0]
    for q in q_group:
        s = scale * keys @ q
        w = np.exp(s - s.max())
        w /= w.sum()
        sig += w
        beta = (dot_band(q, keys, scale) + 2.0 ** -23 * np.abs(s)).max()
        slack += (w[j_gpu] + w[j_ref]) * (2 * beta + 8e-6)
    return sig[j_gpu] - sig[j_ref] <= slack
