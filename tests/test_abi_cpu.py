"""Host-side checks of libdsa.so that need no GPU: the library loads, exports
every entry point ``include/dsa.h`` declares, and its host logic (parameter
rule, validation, buffer layouts, split configuration) is right.  No device
work is launched here."""

import ctypes
import os
import re

import pytest

from oracle import params as oparams
from paper_2609_19702_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "dsa.h")).read()
    return sorted(set(re.findall(r"DSA_API\s+[\w\s\*]+?\b(dsa_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_symbols()
    assert len(names) >= 15
    lib = ctypes.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(B.SIGNATURES), "binding and header disagree"
    assert B.abi_version() == 4


def test_status_strings():
    for st in (0, -1, -2, -3, -4):
        assert B.status_str(st) and "unknown" not in B.status_str(st)
    assert "unknown" in B.status_str(7)


@pytest.mark.parametrize("h,w,window,permille", [
    (24, 24, 128, 950), (24, 24, 256, 900), (64, 64, 512, 950), (16, 16, 64, 950),
    (16, 16, 64, 900), (96, 96, 64, 950), (2, 2, 4, 875), (4, 4, 8, 0), (3, 5, 15, 1000),
    (48, 48, 1024, 950), (7, 11, 33, 333),
])
def test_params_from_sparsity_matches_oracle(h, w, window, permille):
    p = B.params_from_sparsity(10, h, w, window, permille)
    assert p.n_att == oparams.n_att_from_sparsity(h, w, window, permille)
    assert p.window == window


def test_default_window():
    p = B.params_from_sparsity(0, 24, 24, 0, 950)
    assert p.window == oparams.default_window(24, 24)


def test_params_from_sparsity_sink_modes():
    # window mode: the recent window is not bounded by N_r
    p = B.params_from_sparsity(0, 24, 24, 0, 200, mode=B.MODE_WINDOW, sinks=4)
    assert (p.n_att, p.sinks, p.mode) == (oparams.n_att_from_sparsity(24, 24, 576, 200), 4, 2)
    p = B.params_from_sparsity(0, 24, 24, 0, 200, mode=B.MODE_DIAGONAL, sinks=4)
    assert p.n_att == 288 and p.window == 288
    # at least one window token after the sinks
    p = B.params_from_sparsity(0, 4, 4, 8, 1000, mode=B.MODE_DIAGONAL, sinks=4)
    assert p.n_att == 5
    with pytest.raises(B.DSAError):
        B.params_from_sparsity(0, 4, 4, 4, 950, mode=B.MODE_DIAGONAL, sinks=4)
    with pytest.raises(B.DSAError):
        B.params_from_sparsity(0, 4, 4, 4, 950, mode=B.MODE_WINDOW, sinks=-1)


@pytest.mark.parametrize("bad", [
    dict(prompt_len=-1), dict(grid_h=0), dict(window=0), dict(window=70000), dict(n_att=0),
    dict(n_att=200), dict(mode=3), dict(sinks=-1), dict(sinks=8), dict(mode=2, sinks=9),
    dict(mode=2, n_att=(1 << 24) + 1),
])
def test_validate_rejects_bad_params(bad):
    kw = dict(prompt_len=8, grid_h=8, grid_w=8, window=32, n_att=8, mode=1)
    kw.update(bad)
    p = B.make_params(**kw)
    assert B.validate(p, B.make_shape(2, 4, 4, 64)) == B.ERR_INVALID_ARG
    assert B.plan_bytes(p, B.make_shape(2, 4, 4, 64)) == 0


def test_validate_sink_modes():
    s = B.make_shape(2, 4, 4, 64)
    assert B.validate(B.make_params(8, 8, 8, 32, 8, 1, sinks=7), s) == B.OK
    assert B.validate(B.make_params(8, 8, 8, 32, 200, 2, sinks=4), s) == B.OK  # n_att > N_r
    assert B.validate(B.make_params(8, 8, 8, 32, 8, 0, sinks=50), s) == B.OK   # dense ignores it


def test_validate_shapes():
    p = B.make_params(8, 8, 8, 32, 8)
    assert B.validate(p, B.make_shape(2, 4, 4, 64)) == B.OK
    assert B.validate(p, B.make_shape(2, 32, 8, 128)) == B.OK
    assert B.validate(p, B.make_shape(2, 6, 4, 64)) == B.ERR_INVALID_ARG   # 6 % 4
    assert B.validate(p, B.make_shape(0, 4, 4, 64)) == B.ERR_INVALID_ARG
    assert B.validate(p, B.make_shape(2, 4, 4, 96)) == B.ERR_UNSUPPORTED
    assert B.validate(p, B.make_shape(2, 12, 4, 64)) == B.ERR_UNSUPPORTED  # group 3


@pytest.mark.parametrize("mode,sinks", [(0, 0), (1, 0), (1, 4), (2, 4), (2, 0)])
@pytest.mark.parametrize("shape,par", [
    ((64, 20, 20, 64), (120, 24, 24, 128, 950)),
    ((128, 32, 32, 128), (256, 24, 24, 256, 950)),
    ((32, 32, 8, 128), (256, 64, 64, 512, 950)),
    ((1, 8, 8, 64), (32, 16, 16, 64, 950)),
    ((256, 32, 32, 128), (256, 96, 96, 1024, 950)),
    ((3, 8, 1, 64), (0, 5, 7, 9, 500)),
])
def test_layouts_and_split_config(mode, sinks, shape, par):
    p = B.params_from_sparsity(*par, mode=mode, sinks=sinks)
    s = B.make_shape(*shape)
    pairs = s.batch * s.num_kv_heads
    pl, sl, li = B.plan_layout(p, s), B.state_layout(p, s), B.launch_info(p, s)
    L_dec = p.grid_h * p.grid_w
    assert pl.cap == (min(p.n_att, L_dec) if mode else 0)
    assert sl.cap == (p.window - (p.n_att - sinks) if mode == 1 else 0)
    for off in (pl.count_offset, pl.flags_offset, pl.indices_offset,
                sl.count_offset, sl.flags_offset, sl.offsets_offset):
        assert off % 256 == 0
    assert pl.flags_offset >= pl.count_offset + 4 * pairs
    assert pl.indices_offset >= pl.flags_offset + 4 * pairs
    assert pl.bytes == B.plan_bytes(p, s) and pl.bytes >= pl.indices_offset + 4 * pairs * pl.cap
    assert sl.bytes == B.state_bytes(p, s) and sl.bytes >= sl.offsets_offset + 2 * pairs * sl.cap
    rows_max = p.prompt_len + (pl.cap if mode else L_dec)
    block = 32 if li.kernel_variant == 100 else (512 // s.head_dim) * li.kernel_variant
    assert (li.kernel_variant == 100) == (s.num_q_heads > s.num_kv_heads)
    assert 1 <= li.waves_per_group <= (8 if li.kernel_variant == 100 else 4)
    assert li.rows_per_split % block == 0
    assert li.rows_per_split * li.max_splits >= rows_max
    assert li.rows_per_split * (li.max_splits - 1) < max(rows_max, 1)
    assert li.workgroups == pairs * li.max_splits
    g = s.num_q_heads // s.num_kv_heads
    want_ws = pairs * li.max_splits * g * (s.head_dim + 2) * 4 if li.max_splits > 1 else 0
    assert li.workspace_bytes == want_ws == B.workspace_bytes(p, s)
    assert B.window_logits_count(p, s) == s.batch * s.num_q_heads * pl.cap


STRUCTS = {
    "dsa_params": "Params", "dsa_shape": "Shape", "dsa_kv_layout": "KVLayout",
    "dsa_plan_layout": "PlanLayout", "dsa_state_layout": "StateLayout",
    "dsa_launch_info": "LaunchInfo",
}


def test_struct_layouts_match_the_header(tmp_path):
    """The binding's ctypes structures have the C compiler's size and field
    offsets for every structure the header declares."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no host C compiler")
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "dsa.h"', "int main(void) {"]
    for cname, pyname in STRUCTS.items():
        st = getattr(B, pyname)
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in st._fields_:
            lines.append(f'  printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    subprocess.run([gcc, "-D__HIP_PLATFORM_AMD__", "-I", inc, "-I", "/opt/rocm/include",
                    str(src), "-o", str(exe)], check=True)
    got = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    for line in filter(None, got):
        cname, field, value = line.split()
        st = getattr(B, STRUCTS[cname])
        want = ctypes.sizeof(st) if field == "size" else getattr(st, field).offset
        assert int(value) == want, (cname, field, value, want)


# The launch configurations the committed profiles and measurements were
# taken with: (rows per split, splits, workgroups, waves per workgroup,
# kernel variant) for the three model-shaped workloads at 95% sparsity, in
# diagonal and dense mode.  A change to the split rule shows up here first.
BENCH_CONFIGS = {
    ("llamagen_xl", 1): (192, 1, 1280, 3, 8),
    ("llamagen_xl", 0): (128, 6, 7680, 3, 8),
    ("janus_pro_7b", 1): (288, 1, 4096, 4, 8),
    ("janus_pro_7b", 0): (192, 5, 20480, 4, 8),
    ("emu3_8b_gqa", 1): (480, 1, 256, 8, 100),
    ("emu3_8b_gqa", 0): (256, 17, 4352, 2, 100),
}


@pytest.mark.parametrize("name,mode", sorted(BENCH_CONFIGS))
def test_benchmark_launch_configs(name, mode):
    from paper_2609_19702_amd import synth
    w = synth.WORKLOADS[name]
    p = B.params_from_sparsity(w.prompt_len, w.grid_h, w.grid_w, w.window, w.sparsity_permille,
                               mode=mode, sinks=0)
    s = B.make_shape(w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim)
    li = B.launch_info(p, s)
    got = (li.rows_per_split, li.max_splits, li.workgroups, li.waves_per_group, li.kernel_variant)
    assert got == BENCH_CONFIGS[(name, mode)]


def test_binding_rejects_bad_tensors_before_the_call():
    """The binding checks device, element type, density and size of every
    tensor it passes; a mismatch raises before any pointer reaches the
    library (so this needs no GPU)."""
    import torch
    p = B.make_params(8, 4, 4, 8, 3)
    s = B.make_shape(2, 4, 2, 64)
    q = torch.zeros((2, 4, 64), dtype=torch.bfloat16)
    k = torch.zeros((2, 2, 24, 64), dtype=torch.bfloat16)
    out = torch.zeros((2, 4, 64), dtype=torch.float32)
    pos = torch.zeros(2, dtype=torch.int32)
    lay = B.kv_layout(k)
    with pytest.raises(ValueError, match="GPU tensor"):
        B.decode_attention(p, s, q, k, k, lay, pos, None, 0.1, out)
    with pytest.raises(ValueError, match="GPU tensor"):
        B.decode_step(p, s, q, k, k, lay, pos, None, None, 0.1, out, None)
    with pytest.raises(ValueError, match="GPU tensor"):
        B.plan(p, s, pos, None, torch.zeros(B.plan_bytes(p, s), dtype=torch.uint8))
