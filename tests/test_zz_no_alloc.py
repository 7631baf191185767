"""The allocation-free fused step (``dsa_decode_step_noalloc``) against the
fused step with a caller workspace (``dsa_decode_step``): outputs, plans,
window logits and selection states equal bit for bit, on two calls in a
row through the C ABI, the second with a smaller input, in diagonal and
dense mode; a call that would need more partials than the library's buffer
holds is refused before anything is launched."""

import random

import pytest
import torch

from oracle import step as ostep
from paper_2609_19702_amd import binding as B
from paper_2609_19702_amd import synth
from tests.gpu_util import DEV, say, states_to_buffer

pytestmark = pytest.mark.gpu


def one_call(batch, Hq, Hkv, d, Lp, grid, N_r, permille, mode, seed):
    w = synth.Workload("noalloc", 1, batch, Hq, Hkv, d, Lp, grid, grid, N_r,
                       sparsity_permille=permille, outlier_frac=0.01, seed=seed)
    p = B.params_from_sparsity(Lp, grid, grid, N_r, permille, mode)
    s = B.make_shape(batch, Hq, Hkv, d)
    assert 0 < B.workspace_bytes(p, s) <= B.NOALLOC_SCRATCH_BYTES  # the split partials are used
    kv = synth.layer_kv(w, 0, DEV)
    q = synth.layer_query(w, 0, DEV)
    rng = random.Random(seed)
    L = grid * grid
    ts = [L - 1, p.n_att - 1] + [rng.randrange(L) for _ in range(batch - 2)]
    states = [ostep.random_states(Hkv, p.window, p.n_att, t,
                                  [rng.randrange(1 << 30) for _ in range(Hkv * p.window)])
              for t in ts]
    st0 = states_to_buffer(p, s, states, ts)
    pos = torch.tensor(ts, dtype=torch.int32, device=DEV)
    lay = B.kv_layout(kv.k)
    ref, got = B.alloc_buffers(p, s, DEV), B.alloc_buffers(p, s, DEV)
    ref_st, got_st = st0.clone(), st0.clone()
    B.decode_step(p, s, q, kv.k, kv.v, lay, pos, ref_st, ref.plan, 0.1, ref.out, ref.logits,
                  ref.workspace)
    got.out.fill_(7.0)
    B.decode_step_noalloc(p, s, q, kv.k, kv.v, lay, pos, got_st, got.plan, 0.1, got.out,
                          got.logits)
    torch.cuda.synchronize()
    assert torch.equal(got.out, ref.out)
    assert torch.equal(got_st, ref_st)
    if mode != B.MODE_DENSE:
        assert torch.equal(got.plan, ref.plan)
        assert torch.equal(got.logits, ref.logits)
    say("  noalloc", batch, Hq, Hkv, d, "mode", mode, "workspace bytes", B.workspace_bytes(p, s))


@pytest.mark.parametrize("mode", [B.MODE_DIAGONAL, B.MODE_DENSE])
def test_noalloc_equals_workspace_step(mode):
    # grouped heads (MFMA tile, fused combine and selection), then a smaller
    # call into the same per-GPU buffer
    one_call(6, 32, 8, 128, 256, 16, 128, 900, mode, seed=1)
    one_call(2, 32, 8, 128, 256, 16, 128, 900, mode, seed=2)
    # one query head per KV head (vector-ALU tile), large then small
    one_call(5, 8, 8, 64, 300, 12, 72, 950, mode, seed=3)
    one_call(2, 8, 8, 64, 100, 12, 72, 950, mode, seed=4)


def test_noalloc_refuses_oversized_workspace():
    """Refused on the host, before any pointer is used (the raw C entry
    point is called with no buffers at all)."""
    import ctypes
    p = B.make_params(256, 24, 24, 256, 29, B.MODE_DENSE)
    s = B.make_shape(512, 32, 32, 128)
    assert B.workspace_bytes(p, s) > B.NOALLOC_SCRATCH_BYTES
    lay = B.KVLayout(None, 0, 0, 128, 0)
    st = B.lib().dsa_decode_step_noalloc(ctypes.byref(p), ctypes.byref(s), None, None, None,
                                         ctypes.byref(lay), None, None, None, 0, 0.1, None, None,
                                         None)
    assert st == B.ERR_WORKSPACE
