"""Write-side guards: every buffer the library writes (output, plan, window
logits, split workspace, selection state) is placed between two guard
regions of patterned bytes, and after the plan, decode, select, fused-step
and allocation-free calls the guards must be intact.  Run at the three
full-size benchmark shapes (one layer each, the benchmark's launch
configuration) and at the edge cases: unused slots, dense mode, window mode
with sinks, fp8 caches, ring layouts and a single key."""

import math
import random

import pytest
import torch

from oracle import step as ostep
from paper_2609_19702_amd import binding as B
from paper_2609_19702_amd import synth, workload
from tests.gpu_util import DEV, say, states_to_buffer

pytestmark = pytest.mark.gpu

GUARD = 4096  # bytes on each side; a multiple of 256 keeps the buffer aligned


class Guarded:
    """``nbytes`` of device memory between two guard regions."""

    def __init__(self, nbytes, seed):
        self.n = max(int(nbytes), 1)
        g = torch.Generator().manual_seed(seed)
        self.pattern = torch.randint(0, 256, (GUARD * 2,), generator=g, dtype=torch.uint8).to(DEV)
        self.base = torch.empty(self.n + 2 * GUARD, dtype=torch.uint8, device=DEV)
        self.base[:GUARD] = self.pattern[:GUARD]
        self.base[GUARD + self.n:] = self.pattern[GUARD:]
        self.buf = self.base[GUARD:GUARD + self.n]

    def intact(self):
        return (torch.equal(self.base[:GUARD], self.pattern[:GUARD])
                and torch.equal(self.base[GUARD + self.n:], self.pattern[GUARD:]))


class Bufs:
    """The buffers of one layer step, each guarded."""

    def __init__(self, p, s, seed=0):
        self.out = Guarded(s.batch * s.num_q_heads * s.head_dim * 4, seed)
        self.plan = Guarded(B.plan_bytes(p, s), seed + 1)
        self.logits = Guarded(B.window_logits_count(p, s) * 4, seed + 2)
        self.ws = Guarded(B.workspace_bytes(p, s), seed + 3)
        self.state = Guarded(B.state_bytes(p, s), seed + 4)
        self.out_t = self.out.buf.view(torch.float32).view(s.batch, s.num_q_heads, s.head_dim)
        self.plan_t = self.plan.buf[:B.plan_bytes(p, s)]
        self.logits_t = self.logits.buf.view(torch.float32) if B.window_logits_count(p, s) else None
        self.ws_t = self.ws.buf if B.workspace_bytes(p, s) else None
        self.state_t = self.state.buf[:B.state_bytes(p, s)] if B.state_bytes(p, s) else None
        self.plan_t.zero_()

    def check(self, what):
        torch.cuda.synchronize()
        for name in ("out", "plan", "logits", "ws", "state"):
            assert getattr(self, name).intact(), f"{what}: write past the {name} buffer"


def exercise(p, s, q, k, v, lay, pos, st0, tag):
    """Every device call on guarded buffers."""
    scale = 1 / math.sqrt(s.head_dim)
    sparse = p.mode != B.MODE_DENSE
    gb = Bufs(p, s)
    if gb.state_t is not None and st0 is not None:
        gb.state_t.copy_(st0)
    st = gb.state_t
    B.plan(p, s, pos, st if sparse else None, gb.plan_t)
    gb.check(f"{tag} plan")
    B.decode_attention(p, s, q, k, v, lay, pos, gb.plan_t if sparse else None, scale, gb.out_t,
                       gb.logits_t if sparse else None, gb.ws_t)
    gb.check(f"{tag} decode")
    B.select(p, s, pos, gb.plan_t, gb.logits_t, st)
    gb.check(f"{tag} select")
    fb = Bufs(p, s, seed=10)
    if fb.state_t is not None and st0 is not None:
        fb.state_t.copy_(st0)
    B.decode_step(p, s, q, k, v, lay, pos, fb.state_t, fb.plan_t, scale, fb.out_t, fb.logits_t,
                  fb.ws_t)
    fb.check(f"{tag} fused step")
    assert torch.equal(fb.out_t, gb.out_t)
    if B.workspace_bytes(p, s) <= B.NOALLOC_SCRATCH_BYTES:
        nb = Bufs(p, s, seed=20)
        if nb.state_t is not None and st0 is not None:
            nb.state_t.copy_(st0)
        B.decode_step_noalloc(p, s, q, k, v, lay, pos, nb.state_t, nb.plan_t, scale, nb.out_t,
                              nb.logits_t)
        nb.check(f"{tag} allocation-free step")
        assert torch.equal(nb.out_t, gb.out_t)


@pytest.mark.parametrize("name", ["llamagen_xl", "janus_pro_7b", "emu3_8b_gqa"])
@pytest.mark.parametrize("mode", [B.MODE_DIAGONAL, B.MODE_DENSE])
def test_guards_fullsize(name, mode):
    w = synth.WORKLOADS[name]
    say("guards", name, mode)
    bt = workload.make_batch(w, layers=1)
    workload.build_histories(bt)
    L = bt.layers[0]
    p = bt.p if mode == B.MODE_DIAGONAL else bt.pd
    st0 = L.bufs.state if mode == B.MODE_DIAGONAL else None  # dense mode keeps no skip lists
    exercise(p, bt.s, L.q, L.kv.k, L.kv.v, B.kv_layout(L.kv.k), bt.pos, st0, name)


EDGE = [
    # tag, mode, sinks, B, Hq, Hkv, d, L_p, grid, N_r, N_att, fp8, ring
    ("unused+single", B.MODE_DIAGONAL, 0, 3, 4, 4, 64, 0, 4, 8, 3, False, 0),
    ("window+sinks", B.MODE_WINDOW, 4, 5, 8, 2, 128, 20, 12, 40, 12, False, 0),
    ("diag+sinks ring", B.MODE_DIAGONAL, 4, 5, 8, 8, 64, 16, 12, 40, 10, False, 44),
    ("fp8", B.MODE_DIAGONAL, 0, 4, 16, 2, 128, 33, 10, 30, 7, True, 0),
    ("fp8 ring", B.MODE_DIAGONAL, 0, 4, 8, 8, 64, 12, 10, 30, 7, True, 33),
    ("dense gqa", B.MODE_DENSE, 0, 3, 16, 2, 64, 300, 12, 100, 50, False, 0),
]


@pytest.mark.parametrize("case", EDGE, ids=[c[0] for c in EDGE])
def test_guards_edge_cases(case):
    tag, mode, S, Bn, Hq, Hkv, d, Lp, grid, N_r, N_att, fp8, R = case
    say("guards", case)
    L = grid * grid
    rng = random.Random(len(tag))
    ts = [L - 1, -1, 0] + [rng.randrange(L) for _ in range(Bn - 3)]
    w = synth.Workload("guard", 1, Bn, Hq, Hkv, d, Lp, grid, grid, N_r, outlier_frac=0.01)
    kv = synth.layer_kv(w, 0, DEV)
    if fp8:
        kv = synth.to_fp8(kv)
    q = synth.layer_query(w, 0, DEV)
    p = B.make_params(Lp, grid, grid, N_r, N_att, mode, S)
    s = B.make_shape(Bn, Hq, Hkv, d)
    om = {B.MODE_DIAGONAL: "diagonal_sink" if S else "diagonal", B.MODE_WINDOW: "streaming",
          B.MODE_DENSE: "diagonal"}[mode]
    st0 = None
    if mode == B.MODE_DIAGONAL:
        states = [ostep.random_states(Hkv, N_r, N_att, max(t, 0),
                                      [rng.randrange(1 << 30) for _ in range(Hkv * (N_r + S))],
                                      om, S) for t in ts]
        st0 = states_to_buffer(p, s, states, [max(t, 0) for t in ts])
    k, v = kv.k, kv.v
    if R:  # a ring of R slots holding the live rows (the values are irrelevant here)
        k, v = k[:, :, :Lp + R].contiguous(), v[:, :, :Lp + R].contiguous()
    lay = B.kv_layout(k, ring_rows=R, k_scale=kv.k_scale, v_scale=kv.v_scale)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    exercise(p, s, q, k, v, lay, pos, st0, tag)
