"""Drive the library over a synthetic multi-layer decode batch.

``Layer`` holds one layer's device tensors (KV cache, queries, selection
state, plan, logits, workspace, output).  ``build_histories`` gives every
(request, KV head) the skip list Algorithm 1 would have built before its
current decode position, by running the library's own plan -> decode ->
select pipeline over the phase-2 steps with per-step synthetic queries:
at step ``u`` a request whose position ``t_b`` is still ahead runs at
position ``u``, and the others are marked unused (position -1).

``step`` runs one decode step (all layers) in diagonal or dense mode, or in
one of the sink variants of section 5.1 (``make_variant``: Diagonal+Sink,
StreamingLLM) over the same KV and queries; every launch goes to the current
torch stream and nothing synchronises.
"""

from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional

import torch

from . import binding as B
from . import synth


@dataclass
class Layer:
    kv: synth.LayerKV
    q: torch.Tensor
    bufs: B.Buffers


@dataclass
class Batch:
    w: synth.Workload
    p: B.Params          # diagonal-mode parameters
    pd: B.Params         # the same with dense mode
    s: B.Shape
    pos: torch.Tensor    # int32 [B] on the device
    pos_host: List[int]
    layers: List[Layer]
    dense_bufs: B.Buffers
    scale: float

    def kv_bytes(self, dense: bool, elem_bytes: int = 2) -> int:
        """Algorithmic K+V bytes one step streams over all layers: a K row
        and a V row (4*d bytes in bf16, 2*d in fp8) per attended key per KV
        head."""
        n_att = self.p.n_att
        rows = 0
        for t in self.pos_host:
            if t < 0:
                continue
            rows += self.w.prompt_len + (t + 1 if dense else min(t + 1, n_att))
        return rows * self.s.num_kv_heads * 2 * elem_bytes * self.s.head_dim * len(self.layers)


def make_batch(w: synth.Workload, layers: Optional[int] = None, device="cuda",
               positions: Optional[List[int]] = None) -> Batch:
    nl = w.layers if layers is None else layers
    p = B.params_from_sparsity(w.prompt_len, w.grid_h, w.grid_w, w.window, w.sparsity_permille,
                               B.MODE_DIAGONAL)
    pd = B.make_params(p.prompt_len, p.grid_h, p.grid_w, p.window, p.n_att, B.MODE_DENSE)
    s = B.make_shape(w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim)
    pos_host = list(positions) if positions is not None else synth.positions(w).tolist()
    pos = torch.tensor(pos_host, dtype=torch.int32, device=device)
    rows = max(max(pos_host) + 1, 1)
    out = []
    for layer in range(nl):
        kv = synth.layer_kv(w, layer, device, decode_rows=rows)
        q = synth.layer_query(w, layer, device)
        out.append(Layer(kv, q, B.alloc_buffers(p, s, device)))
    dense_bufs = B.alloc_buffers(pd, s, device)
    return Batch(w, p, pd, s, pos, pos_host, out, dense_bufs, 1.0 / math.sqrt(w.head_dim))


@dataclass
class Variant:
    """Another index-builder mode, another KV element type or a ring-buffer
    cache, over the batch's queries, with its own per-layer buffers (and
    caches, for fp8 and the ring)."""
    name: str
    p: B.Params
    bufs: List[B.Buffers]
    kvs: Optional[List[synth.LayerKV]] = None
    ring_rows: int = 0


def kv_layout_of(kv: synth.LayerKV, ring_rows: int = 0) -> B.KVLayout:
    return B.kv_layout(kv.k, ring_rows=ring_rows, k_scale=kv.k_scale, v_scale=kv.v_scale)


def build_histories(bt: Batch, device="cuda", p: Optional[B.Params] = None,
                    bufs: Optional[List[B.Buffers]] = None,
                    kvs: Optional[List[synth.LayerKV]] = None):
    """Run the phase-2 steps of every layer so that each state holds the skip
    entries appended before its request's decode position (``p``/``bufs``/
    ``kvs``: another variant's parameters, buffers and caches; default the
    batch's own)."""
    p = bt.p if p is None else p
    bufs = [L.bufs for L in bt.layers] if bufs is None else bufs
    kvs = [L.kv for L in bt.layers] if kvs is None else kvs
    s, w = bt.s, bt.w
    if B.state_layout(p, s).cap == 0:
        return  # nothing is ever selected
    last = min(max(bt.pos_host) - 1, p.window + p.sinks - 2)
    for li, (kv, bf) in enumerate(zip(kvs, bufs)):
        B.state_reset(p, s, bf.state)
        lay = kv_layout_of(kv)
        for u in range(p.n_att - 1, last + 1):
            pos = torch.tensor([u if u < t else -1 for t in bt.pos_host], dtype=torch.int32,
                               device=device)
            q = synth.step_query(w, li, u, device)
            B.plan(p, s, pos, bf.state, bf.plan)
            B.decode_attention(p, s, q, kv.k, kv.v, lay, pos, bf.plan, bt.scale, bf.out, bf.logits,
                               bf.workspace)
            B.select(p, s, pos, bf.plan, bf.logits, bf.state)


def make_variant(bt: Batch, name: str, mode: int, sinks: int, device="cuda",
                 fp8: bool = False) -> Variant:
    """The batch's window and N_att in another mode (section 5.1 variants:
    diagonal mode with sinks is Diagonal+Sink, window mode with sinks is
    StreamingLLM), or over an fp8 copy of the caches, with its selection
    histories built."""
    p = B.make_params(bt.p.prompt_len, bt.p.grid_h, bt.p.grid_w, bt.p.window, bt.p.n_att, mode,
                      sinks)
    kvs = [synth.to_fp8(L.kv) for L in bt.layers] if fp8 else None
    v = Variant(name, p, [B.alloc_buffers(p, bt.s, device) for _ in bt.layers], kvs)
    build_histories(bt, device, v.p, v.bufs, v.kvs)
    return v


def ring_cache(kv: synth.LayerKV, prompt_len: int, pos_host: List[int], R: int,
               device="cuda") -> synth.LayerKV:
    """The cache as a ring of ``R`` decode slots per (request, KV head)
    (section 4, "Cost analysis": physical eviction): the prompt rows, then
    decode position ``j`` of the live window ``[t - R + 1, t]`` in slot
    ``j mod R``.  Slots no live position maps to keep a copy of the prompt's
    first row; no step reads them."""
    Bn, H, _, d = kv.k.shape
    t = torch.tensor(pos_host, dtype=torch.int64, device=device).clamp_min(0)[:, None]
    r = torch.arange(R, dtype=torch.int64, device=device)[None, :]
    j = t - torch.remainder(t - r, R)                 # the live position stored in slot r
    src = torch.where(j >= 0, prompt_len + j, torch.zeros_like(j))
    src = src[:, None, :, None].expand(Bn, H, R, d)
    out = []
    for x in (kv.k, kv.v):
        ring = torch.empty((Bn, H, prompt_len + R, d), dtype=x.dtype, device=device)
        ring[:, :, :prompt_len] = x[:, :, :prompt_len]
        ring[:, :, prompt_len:] = torch.gather(x, 2, src)
        out.append(ring)
    return synth.LayerKV(out[0], out[1], prompt_len + R, kv.k_scale, kv.v_scale)


def make_ring_variant(bt: Batch, device="cuda") -> Variant:
    """The batch's diagonal step over ring caches of ``R = N_r`` decode
    slots, the least Algorithm 1 allows, starting from copies of the
    batch's selection states."""
    R = bt.p.window + bt.p.sinks
    kvs = [ring_cache(L.kv, bt.w.prompt_len, bt.pos_host, R, device) for L in bt.layers]
    bufs = [B.alloc_buffers(bt.p, bt.s, device) for _ in bt.layers]
    for bf, L in zip(bufs, bt.layers):
        bf.state.copy_(L.bufs.state)
    return Variant("ring", bt.p, bufs, kvs, ring_rows=R)


def sparse_layer(bt: Batch, L: Layer, timer=None):
    p, s = bt.p, bt.s
    B.plan(p, s, bt.pos, L.bufs.state, L.bufs.plan)
    B.decode_attention(p, s, L.q, L.kv.k, L.kv.v, B.kv_layout(L.kv.k), bt.pos, L.bufs.plan,
                       bt.scale, L.bufs.out, L.bufs.logits, L.bufs.workspace, events=timer)
    B.select(p, s, bt.pos, L.bufs.plan, L.bufs.logits, L.bufs.state)


def fused_layer(bt: Batch, L: Layer, timer=None):
    B.decode_step(bt.p, bt.s, L.q, L.kv.k, L.kv.v, B.kv_layout(L.kv.k), bt.pos, L.bufs.state,
                  L.bufs.plan, bt.scale, L.bufs.out, L.bufs.logits, L.bufs.workspace, events=timer)


def dense_layer(bt: Batch, L: Layer, timer=None):
    db = bt.dense_bufs
    B.decode_attention(bt.pd, bt.s, L.q, L.kv.k, L.kv.v, B.kv_layout(L.kv.k), bt.pos, None,
                       bt.scale, db.out, None, db.workspace, events=timer)


def variant_layer(bt: Batch, v: Variant, i: int, timer=None):
    L, bf = bt.layers[i], v.bufs[i]
    kv = L.kv if v.kvs is None else v.kvs[i]
    B.decode_step(v.p, bt.s, L.q, kv.k, kv.v, kv_layout_of(kv, v.ring_rows), bt.pos, bf.state,
                  bf.plan, bt.scale, bf.out, bf.logits, bf.workspace, events=timer)


def step(bt: Batch, dense: bool = False, timers=None, fused: bool = False,
         variant: Optional[Variant] = None):
    """One decode step over all layers: dense mode, the three separate calls
    (plan, decode, select), the fused step, or the fused step of a variant.
    ``timers[i]`` (a pair from ``binding.timing_events``) receives the start
    and end of layer i's split-K decode kernel when given."""
    for i, L in enumerate(bt.layers):
        tm = None if timers is None else timers[i]
        if variant is not None:
            variant_layer(bt, variant, i, tm)
        else:
            fn = dense_layer if dense else (fused_layer if fused else sparse_layer)
            fn(bt, L, tm)


def with_window(bt: Batch, window: int, device="cuda") -> Batch:
    """The same KV caches, queries and positions under another recent window
    N_r (and the N_att the sparsity rule gives with it), with fresh per-layer
    buffers; the selection states start empty."""
    w = bt.w.with_(window=window, name=f"{bt.w.name}_w{window}")
    p = B.params_from_sparsity(w.prompt_len, w.grid_h, w.grid_w, w.window, w.sparsity_permille,
                               B.MODE_DIAGONAL)
    pd = B.make_params(p.prompt_len, p.grid_h, p.grid_w, p.window, p.n_att, B.MODE_DENSE)
    layers = [Layer(L.kv, L.q, B.alloc_buffers(p, bt.s, device)) for L in bt.layers]
    return Batch(w, p, pd, bt.s, bt.pos, bt.pos_host, layers, bt.dense_bufs, bt.scale)


def build_history_shared(bt: Batch, device="cuda"):
    """Selection histories for a timing run: the library's own phase-2 steps
    build layer 0's skip lists (as ``build_histories``), and every other layer
    starts from a copy of them.  Each layer still reads its own KV cache; the
    kept sets are valid Algorithm 1 histories, shared only to save setup
    time on runs with many layers."""
    first = bt.layers[0]
    build_histories(bt, device, bufs=[first.bufs], kvs=[first.kv])
    for L in bt.layers[1:]:
        L.bufs.state.copy_(first.bufs.state)
