"""Seeded synthetic inputs shaped like the paper's workloads.

This module is shared by the tests, the benchmark and the CPU oracle's
callers.  It holds no arithmetic of the method itself: it only names the
workload shapes and draws seeded random tensors (queries, KV caches, decode
positions, outlier masks, and the random integers that stand in for a
selection history).

Workloads (synthetic stand-ins for the paper's models; no weights, prompts or
benchmark items are used):

* ``tiny``          1 request, 8 heads (MHA), d=64, prompt 32, 16x16 grid,
                    window 64 -- small enough for the fp64 oracle to replay
                    every one of the 256 decode steps.
* ``llamagen_xl``   36 layers x 20 heads, d=64 (MHA), prompt 120, 24x24 grid
                    (576 visual tokens), batch 64, window 128.
* ``janus_pro_7b``  30 layers x 32 heads, d=128 (MHA), prompt 256, 24x24,
                    batch 128, window 256.
* ``emu3_8b_gqa``   32 query / 8 KV heads, d=128, prompt 256, 64x64 grid
                    (4096 visual tokens), batch 32, window 512, 1% of key
                    rows scaled by 8 (outlier keys); 32 layers.
* ``sweep_*``       the Janus head shape over grid, batch and window.

Values are N(0, 1) in fp32, rounded to bf16 (round to nearest even) before
either side sees them.  Decode positions are "ragged": each request's newest
decode position is drawn uniformly from ``[0, H*W)``.

fp8 caches (``to_fp8``) are the bf16 cache stored as OCP E4M3 bytes with
one fp32 scale per (request, KV head) for K and one for V: the largest
magnitude of that head's rows maps to 448, and every value is rounded to
the nearest E4M3 value by torch's float8_e4m3fn conversion.  That is how
the test inputs are made; the library and the oracle only read the bytes
and the scales.
"""

from __future__ import annotations

import dataclasses
from dataclasses import dataclass
from typing import Dict, Optional

import torch

# tensor ids used in the seed of every generated tensor
T_KP, T_VP, T_K, T_V, T_Q, T_OUTLIER, T_POS, T_CHOICE, T_STEPQ = range(9)


@dataclass(frozen=True)
class Workload:
    name: str
    layers: int
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    prompt_len: int
    grid_h: int
    grid_w: int
    window: int
    sparsity_permille: int = 950
    positions: str = "ragged"       # "ragged" | "last" | "first"
    outlier_frac: float = 0.0
    outlier_scale: float = 8.0
    seed: int = 0

    @property
    def decode_len(self) -> int:
        return self.grid_h * self.grid_w

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 1, 1, 8, 8, 64, 32, 16, 16, 64, positions="last"),
    "llamagen_xl": Workload("llamagen_xl", 36, 64, 20, 20, 64, 120, 24, 24, 128),
    "janus_pro_7b": Workload("janus_pro_7b", 30, 128, 32, 32, 128, 256, 24, 24, 256),
    "emu3_8b_gqa": Workload("emu3_8b_gqa", 32, 32, 32, 8, 128, 256, 64, 64, 512,
                            outlier_frac=0.01),
}


def sweep_workloads():
    """The Janus-shaped sweep: grid x batch x window (diagonal and dense are
    the two modes run on each cell)."""
    out = []
    for g in (24, 48, 96):
        for b in (1, 16, 64, 256):
            for w in (64, 256, 1024):
                out.append(Workload(f"sweep_g{g}_b{b}_w{w}", 4, b, 32, 32, 128, 256, g, g, w))
    return out


def seed_of(w: Workload, layer: int, tensor_id: int, sub: int = 0) -> int:
    base = (w.seed * 1_000_003 + layer * 16 + tensor_id)
    return base * 100_003 + sub


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def randn_bf16(shape, seed: int, device="cpu") -> torch.Tensor:
    """N(0, 1) fp32 from a seeded generator on ``device``, rounded to bf16."""
    x = torch.randn(shape, generator=_gen(device, seed), device=device, dtype=torch.float32)
    return x.to(torch.bfloat16)


def positions(w: Workload, layer: int = 0) -> torch.Tensor:
    """Newest decode position of each request (int32, CPU)."""
    if w.positions == "last":
        return torch.full((w.batch,), w.decode_len - 1, dtype=torch.int32)
    if w.positions == "first":
        return torch.zeros((w.batch,), dtype=torch.int32)
    g = _gen("cpu", seed_of(w, 0, T_POS))
    return torch.randint(0, w.decode_len, (w.batch,), generator=g, dtype=torch.int64).to(torch.int32)


def random_ints(w: Workload, layer: int, n: int, sub: int = 0) -> torch.Tensor:
    """``n`` non-negative random integers (CPU), e.g. to drive a random
    selection history."""
    g = _gen("cpu", seed_of(w, layer, T_CHOICE, sub))
    return torch.randint(0, 2**31 - 1, (n,), generator=g, dtype=torch.int64)


@dataclass
class LayerKV:
    """A head-major KV cache of one layer: ``k``/``v`` are
    ``[B, Hkv, rows, d]`` bf16 (or E4M3 bytes as uint8, with fp32 scales
    ``k_scale``/``v_scale`` of ``B * Hkv`` values) with the ``prompt_len``
    prompt rows first and decode position ``j`` at row ``prompt_len + j``."""
    k: torch.Tensor
    v: torch.Tensor
    rows: int
    k_scale: Optional[torch.Tensor] = None
    v_scale: Optional[torch.Tensor] = None

    @property
    def strides(self):
        """(batch, head, row) strides in elements."""
        s = self.k.stride()
        return s[0], s[1], s[2]


def layer_kv(w: Workload, layer: int, device="cpu", decode_rows: Optional[int] = None) -> LayerKV:
    """Seeded KV cache of one layer with ``decode_rows`` decode rows (default:
    the whole grid)."""
    n_dec = w.decode_len if decode_rows is None else int(decode_rows)
    B, H, d, Lp = w.batch, w.num_kv_heads, w.head_dim, w.prompt_len
    rows = Lp + n_dec
    out = []
    for tp, td in ((T_KP, T_K), (T_VP, T_V)):
        x = torch.empty((B, H, rows, d), dtype=torch.float32, device=device)
        if Lp:
            x[:, :, :Lp] = torch.randn((B, H, Lp, d), generator=_gen(device, seed_of(w, layer, tp)),
                                       device=device, dtype=torch.float32)
        x[:, :, Lp:] = torch.randn((B, H, n_dec, d), generator=_gen(device, seed_of(w, layer, td)),
                                   device=device, dtype=torch.float32)
        if td == T_K and w.outlier_frac > 0:
            u = torch.rand((B, H, rows), generator=_gen(device, seed_of(w, layer, T_OUTLIER)),
                           device=device, dtype=torch.float32)
            x *= torch.where(u < w.outlier_frac, w.outlier_scale, 1.0).unsqueeze(-1)
        out.append(x.to(torch.bfloat16))
        del x
    return LayerKV(out[0], out[1], rows)


E4M3_MAX = 448.0


def _fp8_one(x: torch.Tensor):
    """E4M3 bytes and per-(request, head) scales of a ``[B, H, rows, d]``
    bf16 tensor, one request at a time (bounded temporary memory)."""
    B, H = x.shape[:2]
    codes = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    scale = torch.empty((B, H), dtype=torch.float32, device=x.device)
    for b in range(B):
        xb = x[b].float()
        amax = xb.abs().amax(dim=(1, 2)).clamp_min(1e-30)
        sc = amax / E4M3_MAX
        codes[b] = (xb / sc[:, None, None]).clamp(-E4M3_MAX, E4M3_MAX).to(
            torch.float8_e4m3fn).view(torch.uint8)
        scale[b] = sc
        del xb
    return codes, scale.reshape(-1).contiguous()


def to_fp8(kv: LayerKV) -> LayerKV:
    """The same cache as E4M3 bytes plus per-(request, KV head) scales."""
    kc, ks = _fp8_one(kv.k)
    vc, vs = _fp8_one(kv.v)
    return LayerKV(kc, vc, kv.rows, ks, vs)


def layer_query(w: Workload, layer: int, device="cpu") -> torch.Tensor:
    """Queries ``[B, Hq, d]`` bf16 of the timed step of one layer."""
    return randn_bf16((w.batch, w.num_q_heads, w.head_dim), seed_of(w, layer, T_Q), device)


def step_query(w: Workload, layer: int, step: int, device="cpu") -> torch.Tensor:
    """Queries ``[B, Hq, d]`` bf16 used at decode step ``step`` while a
    selection history is built."""
    return randn_bf16((w.batch, w.num_q_heads, w.head_dim), seed_of(w, layer, T_STEPQ, step), device)


def tiny_tensors() -> Dict[str, torch.Tensor]:
    """The tiny workload's full trajectory inputs, drawn on the CPU from one
    generator seeded with 0 in this order: Kp, Vp ``[L_p, H, d]``, then K, V
    ``[L_dec, H, d]``, then Q ``[L_dec, H, d]`` (fp32 N(0,1) -> bf16)."""
    w = WORKLOADS["tiny"]
    g = _gen("cpu", 0)
    H, d, Lp, L = w.num_kv_heads, w.head_dim, w.prompt_len, w.decode_len
    Kp = torch.randn((Lp, H, d), generator=g)
    Vp = torch.randn((Lp, H, d), generator=g)
    K = torch.randn((L, H, d), generator=g)
    V = torch.randn((L, H, d), generator=g)
    Q = torch.randn((L, H, d), generator=g)
    return {n: x.to(torch.bfloat16) for n, x in
            (("Kp", Kp), ("Vp", Vp), ("K", K), ("V", V), ("Q", Q))}
