"""ctypes binding of ``libdsa.so`` (declared in ``include/dsa.h``).

Argument marshalling only: every step of the decode path runs in the HIP
kernels of the library.  PyTorch supplies device memory (tensors) and the
stream (``torch.cuda.current_stream()``); this module passes their raw
pointers through the C ABI and turns non-zero status codes into
``DSAError``.  There is no fallback: if the library is missing the import
of the entry points fails.
"""

from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional

import torch  # loads the HIP runtime that libdsa.so binds to (same soname)

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdsa.so")

MODE_DENSE = 0
MODE_DIAGONAL = 1
MODE_WINDOW = 2
KV_BF16 = 0
KV_FP8_E4M3 = 1

FLAG_INACTIVE = 1
FLAG_POS_CLAMPED = 2
FLAG_STATE_BEHIND = 4
FLAG_BAD_OFFSET = 8
FLAG_COUNT = 16

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = 0, -1, -2, -3, -4


class DSAError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {status_str(status)} (status {status})")
        self.status = status


class Params(C.Structure):
    _fields_ = [("prompt_len", C.c_int32), ("grid_h", C.c_int32), ("grid_w", C.c_int32),
                ("window", C.c_int32), ("n_att", C.c_int32), ("mode", C.c_int32),
                ("sinks", C.c_int32)]

    def __repr__(self):
        return (f"Params(prompt_len={self.prompt_len}, grid={self.grid_h}x{self.grid_w}, "
                f"window={self.window}, n_att={self.n_att}, mode={self.mode}, sinks={self.sinks})")


class Shape(C.Structure):
    _fields_ = [("batch", C.c_int32), ("num_q_heads", C.c_int32),
                ("num_kv_heads", C.c_int32), ("head_dim", C.c_int32)]


class KVLayout(C.Structure):
    _fields_ = [("d_row_base", C.c_void_p), ("stride_batch", C.c_int64),
                ("stride_head", C.c_int64), ("stride_row", C.c_int64),
                ("ring_rows", C.c_int64), ("d_k_scale", C.c_void_p), ("d_v_scale", C.c_void_p),
                ("dtype", C.c_int32)]


class PlanLayout(C.Structure):
    _fields_ = [("count_offset", C.c_size_t), ("flags_offset", C.c_size_t),
                ("indices_offset", C.c_size_t), ("cap", C.c_int32), ("bytes", C.c_size_t)]


class StateLayout(C.Structure):
    _fields_ = [("count_offset", C.c_size_t), ("flags_offset", C.c_size_t),
                ("offsets_offset", C.c_size_t), ("cap", C.c_int32), ("bytes", C.c_size_t),
                ("kept_count_offset", C.c_size_t), ("kept_offset", C.c_size_t),
                ("kept_cap", C.c_int32), ("kept_stride", C.c_int32)]


class LaunchInfo(C.Structure):
    _fields_ = [("rows_per_split", C.c_int32), ("max_splits", C.c_int32),
                ("workgroups", C.c_int32), ("kernel_variant", C.c_int32),
                ("waves_per_group", C.c_int32), ("workspace_bytes", C.c_size_t),
                ("kept_read", C.c_int32)]


# name -> (restype, argtypes); mirrors include/dsa.h
_P, _S = C.POINTER(Params), C.POINTER(Shape)
_VP = C.c_void_p
SIGNATURES = {
    "dsa_abi_version": (C.c_int32, []),
    "dsa_status_str": (C.c_char_p, [C.c_int32]),
    "dsa_params_from_sparsity": (C.c_int32, [C.c_int32] * 7 + [_P]),
    "dsa_validate": (C.c_int32, [_P, _S]),
    "dsa_get_state_layout": (C.c_int32, [_P, _S, C.POINTER(StateLayout)]),
    "dsa_get_plan_layout": (C.c_int32, [_P, _S, C.POINTER(PlanLayout)]),
    "dsa_get_launch_info": (C.c_int32, [_P, _S, C.POINTER(LaunchInfo)]),
    "dsa_state_bytes": (C.c_size_t, [_P, _S]),
    "dsa_plan_bytes": (C.c_size_t, [_P, _S]),
    "dsa_workspace_bytes": (C.c_size_t, [_P, _S]),
    "dsa_window_logits_count": (C.c_size_t, [_P, _S]),
    "dsa_state_reset": (C.c_int32, [_P, _S, _VP, _VP, _VP]),
    "dsa_plan": (C.c_int32, [_P, _S, _VP, _VP, _VP, C.c_size_t, _VP]),
    "dsa_decode_attention": (C.c_int32, [_P, _S, _VP, _VP, _VP, C.POINTER(KVLayout), _VP, _VP,
                                         C.c_float, _VP, _VP, _VP, C.c_size_t, _VP]),
    "dsa_decode_attention_timed": (C.c_int32, [_P, _S, _VP, _VP, _VP, C.POINTER(KVLayout), _VP,
                                               _VP, C.c_float, _VP, _VP, _VP, C.c_size_t, _VP,
                                               _VP, _VP]),
    "dsa_decode_step": (C.c_int32, [_P, _S, _VP, _VP, _VP, C.POINTER(KVLayout), _VP, _VP, _VP,
                                    C.c_size_t, C.c_float, _VP, _VP, _VP, C.c_size_t, _VP]),
    "dsa_decode_step_timed": (C.c_int32, [_P, _S, _VP, _VP, _VP, C.POINTER(KVLayout), _VP, _VP,
                                          _VP, C.c_size_t, C.c_float, _VP, _VP, _VP, C.c_size_t,
                                          _VP, _VP, _VP]),
    "dsa_decode_step_noalloc": (C.c_int32, [_P, _S, _VP, _VP, _VP, C.POINTER(KVLayout), _VP, _VP,
                                            _VP, C.c_size_t, C.c_float, _VP, _VP, _VP]),
    "dsa_select": (C.c_int32, [_P, _S, _VP, _VP, _VP, _VP, _VP]),
}

NOALLOC_SCRATCH_BYTES = 16 << 20  # DSA_NOALLOC_SCRATCH_BYTES

_lib = None


def lib() -> C.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_19702_amd.build` (there is no fallback)")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _lib = L
    return _lib


def status_str(status: int) -> str:
    return lib().dsa_status_str(int(status)).decode()


def _check(status: int, where: str):
    if status != OK:
        raise DSAError(status, where)


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _nbytes(x) -> int:
    return x.numel() * x.element_size()


def _need(x, name, dtype=None, min_bytes=0, contiguous=True):
    """Argument checks before a device call (tensors only; raw integer
    pointers pass through unchecked): on the GPU, of the expected element
    type, dense where the library assumes it, and at least ``min_bytes``
    long.  A mismatch raises ``ValueError`` instead of letting the kernels
    read or write outside the tensor."""
    if x is None or isinstance(x, int):
        return
    if not x.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if dtype is not None and x.dtype not in (dtype if isinstance(dtype, tuple) else (dtype,)):
        raise ValueError(f"{name} must be {dtype}, got {x.dtype}")
    if contiguous and not x.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if _nbytes(x) < min_bytes:
        raise ValueError(f"{name} holds {_nbytes(x)} bytes, needs {min_bytes}")


_KV_DTYPES = (torch.bfloat16, torch.uint8, torch.float8_e4m3fn)


def _check_decode_args(p, s, q, k, v, layout, decode_pos, out, window_logits):
    B_, Hq, Hkv, d = s.batch, s.num_q_heads, s.num_kv_heads, s.head_dim
    _need(q, "q", torch.bfloat16, B_ * Hq * d * 2)
    _need(out, "out", torch.float32, B_ * Hq * d * 4)
    _need(decode_pos, "decode_pos", torch.int32, B_ * 4)
    _need(window_logits, "window_logits", torch.float32, window_logits_count(p, s) * 4)
    for x, name in ((k, "k"), (v, "v")):
        _need(x, name, _KV_DTYPES, contiguous=False)
    if isinstance(k, torch.Tensor) and isinstance(v, torch.Tensor):
        if k.dtype != v.dtype or k.shape != v.shape or k.stride() != v.stride():
            raise ValueError("k and v must share element type, shape and strides")
        if k.dim() == 4 and layout.d_row_base is None:
            rows_needed = p.prompt_len + (layout.ring_rows if layout.ring_rows else 1)
            if k.shape[0] < B_ or k.shape[1] < Hkv or k.shape[3] != d or k.shape[2] < rows_needed:
                raise ValueError(f"cache of shape {tuple(k.shape)} does not hold {B_} requests x "
                                 f"{Hkv} KV heads x {rows_needed}+ rows of {d} elements")


# ---- host-only helpers ------------------------------------------------------

def abi_version() -> int:
    return lib().dsa_abi_version()


def make_params(prompt_len, grid_h, grid_w, window, n_att, mode=MODE_DIAGONAL, sinks=0) -> Params:
    return Params(prompt_len, grid_h, grid_w, window, n_att, mode, sinks)


def params_from_sparsity(prompt_len, grid_h, grid_w, window, sparsity_permille,
                         mode=MODE_DIAGONAL, sinks=0) -> Params:
    p = Params()
    _check(lib().dsa_params_from_sparsity(prompt_len, grid_h, grid_w, window,
                                          sparsity_permille, mode, sinks, C.byref(p)),
           "dsa_params_from_sparsity")
    return p


def make_shape(batch, num_q_heads, num_kv_heads, head_dim) -> Shape:
    return Shape(batch, num_q_heads, num_kv_heads, head_dim)


def validate(p: Params, s: Shape) -> int:
    return lib().dsa_validate(C.byref(p), C.byref(s))


def state_layout(p: Params, s: Shape) -> StateLayout:
    out = StateLayout()
    _check(lib().dsa_get_state_layout(C.byref(p), C.byref(s), C.byref(out)), "dsa_get_state_layout")
    return out


def plan_layout(p: Params, s: Shape) -> PlanLayout:
    out = PlanLayout()
    _check(lib().dsa_get_plan_layout(C.byref(p), C.byref(s), C.byref(out)), "dsa_get_plan_layout")
    return out


def launch_info(p: Params, s: Shape) -> LaunchInfo:
    out = LaunchInfo()
    _check(lib().dsa_get_launch_info(C.byref(p), C.byref(s), C.byref(out)), "dsa_get_launch_info")
    return out


def state_bytes(p, s) -> int:
    return lib().dsa_state_bytes(C.byref(p), C.byref(s))


def plan_bytes(p, s) -> int:
    return lib().dsa_plan_bytes(C.byref(p), C.byref(s))


def workspace_bytes(p, s) -> int:
    return lib().dsa_workspace_bytes(C.byref(p), C.byref(s))


def window_logits_count(p, s) -> int:
    return lib().dsa_window_logits_count(C.byref(p), C.byref(s))


# ---- device calls -------------------------------------------------------------

def state_reset(p, s, state, req_mask=None, stream=None):
    _check(lib().dsa_state_reset(C.byref(p), C.byref(s), _ptr(state), _ptr(req_mask),
                                 _stream(stream)), "dsa_state_reset")


def plan(p, s, decode_pos, state, plan_buf, stream=None):
    _need(decode_pos, "decode_pos", torch.int32, s.batch * 4)
    _need(state, "state", None, state_bytes(p, s) if state_layout(p, s).cap else 0)
    _check(lib().dsa_plan(C.byref(p), C.byref(s), _ptr(decode_pos), _ptr(state), _ptr(plan_buf),
                          plan_buf.numel() * plan_buf.element_size(), _stream(stream)), "dsa_plan")


def kv_layout(k: torch.Tensor, row_base: Optional[torch.Tensor] = None,
              ring_rows: int = 0, k_scale: Optional[torch.Tensor] = None,
              v_scale: Optional[torch.Tensor] = None) -> KVLayout:
    """Layout of a ``[B, Hkv, rows, d]`` cache (any strides with unit stride
    along d); ``row_base`` optionally gives per-request base offsets;
    ``ring_rows = R > 0`` stores decode position ``j`` at row ``L_p + j``
    for the ``S`` sinks and at ``L_p + S + (j - S) % (R - S)`` after them.
    A bf16 cache is ``torch.bfloat16``; an fp8 (OCP E4M3) cache is
    ``torch.float8_e4m3fn`` or its bytes as ``torch.uint8``, with optional
    fp32 ``k_scale``/``v_scale`` of ``B * Hkv`` values."""
    sb, sh, sr, sd = k.stride()
    if sd != 1:
        raise ValueError("head_dim must be contiguous")
    if k.dtype == torch.bfloat16:
        dtype = KV_BF16
    elif k.dtype in (torch.uint8, torch.float8_e4m3fn):
        dtype = KV_FP8_E4M3
    else:
        raise ValueError(f"unsupported KV dtype {k.dtype}")
    return KVLayout(_ptr(row_base), sb, sh, sr, int(ring_rows), _ptr(k_scale), _ptr(v_scale),
                    dtype)


def decode_attention(p, s, q, k, v, layout: KVLayout, decode_pos, plan_buf, sm_scale, out,
                     window_logits=None, workspace=None, stream=None, events=None):
    """``events``: optional (start, stop) pair from ``timing_events()``; they
    then receive the start of the split-K kernel and the end of the call's
    last kernel."""
    _check_decode_args(p, s, q, k, v, layout, decode_pos, out, window_logits)
    if p.mode != MODE_DENSE:
        _need(plan_buf, "plan", None, plan_bytes(p, s))
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    args = (C.byref(p), C.byref(s), _ptr(q), _ptr(k), _ptr(v), C.byref(layout), _ptr(decode_pos),
            _ptr(plan_buf), float(sm_scale), _ptr(out), _ptr(window_logits), _ptr(workspace),
            ws_bytes)
    if events is None:
        _check(lib().dsa_decode_attention(*args, _stream(stream)), "dsa_decode_attention")
    else:
        _check(lib().dsa_decode_attention_timed(*args, events[0].cuda_event, events[1].cuda_event,
                                                _stream(stream)), "dsa_decode_attention_timed")


def decode_step(p, s, q, k, v, layout: KVLayout, decode_pos, state, plan_buf, sm_scale, out,
                window_logits, workspace=None, stream=None, events=None):
    """One fused decode step: plan + attention + selection in one pass."""
    _check_decode_args(p, s, q, k, v, layout, decode_pos, out, window_logits)
    _need(state, "state", None, state_bytes(p, s) if state_layout(p, s).cap else 0)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    pb = 0 if plan_buf is None else plan_buf.numel() * plan_buf.element_size()
    args = (C.byref(p), C.byref(s), _ptr(q), _ptr(k), _ptr(v), C.byref(layout), _ptr(decode_pos),
            _ptr(state), _ptr(plan_buf), pb, float(sm_scale), _ptr(out), _ptr(window_logits),
            _ptr(workspace), ws_bytes)
    if events is None:
        _check(lib().dsa_decode_step(*args, _stream(stream)), "dsa_decode_step")
    else:
        _check(lib().dsa_decode_step_timed(*args, events[0].cuda_event, events[1].cuda_event,
                                           _stream(stream)), "dsa_decode_step_timed")


def decode_step_noalloc(p, s, q, k, v, layout: KVLayout, decode_pos, state, plan_buf, sm_scale,
                        out, window_logits, stream=None):
    """``decode_step`` without a workspace: the split partials live in the
    library's own per-GPU buffer (for callers that cannot allocate)."""
    _check_decode_args(p, s, q, k, v, layout, decode_pos, out, window_logits)
    _need(state, "state", None, state_bytes(p, s) if state_layout(p, s).cap else 0)
    pb = 0 if plan_buf is None else plan_buf.numel() * plan_buf.element_size()
    _check(lib().dsa_decode_step_noalloc(C.byref(p), C.byref(s), _ptr(q), _ptr(k), _ptr(v),
                                         C.byref(layout), _ptr(decode_pos), _ptr(state),
                                         _ptr(plan_buf), pb, float(sm_scale), _ptr(out),
                                         _ptr(window_logits), _stream(stream)),
           "dsa_decode_step_noalloc")


def timing_events():
    """A (start, stop) pair of timing events that exist on the device (torch
    creates its events lazily, at the first record)."""
    pair = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    for e in pair:
        e.record()
    return pair


def select(p, s, decode_pos, plan_buf, window_logits, state, stream=None):
    if state_layout(p, s).cap:
        _need(decode_pos, "decode_pos", torch.int32, s.batch * 4)
        _need(plan_buf, "plan", None, plan_bytes(p, s))
        _need(window_logits, "window_logits", torch.float32, window_logits_count(p, s) * 4)
        _need(state, "state", None, state_bytes(p, s))
    _check(lib().dsa_select(C.byref(p), C.byref(s), _ptr(decode_pos), _ptr(plan_buf),
                            _ptr(window_logits), _ptr(state), _stream(stream)), "dsa_select")


# ---- buffers (torch allocations) and views --------------------------------------

@dataclass
class Buffers:
    """Device buffers of one layer: selection state, plan, window logits,
    split workspace and output."""
    state: torch.Tensor
    plan: torch.Tensor
    logits: torch.Tensor
    workspace: Optional[torch.Tensor]
    out: torch.Tensor


def alloc_buffers(p: Params, s: Shape, device="cuda") -> Buffers:
    nb = lambda n: torch.zeros(max(int(n), 1), dtype=torch.uint8, device=device)
    ws = workspace_bytes(p, s)
    return Buffers(
        state=nb(state_bytes(p, s)),
        plan=nb(plan_bytes(p, s)),
        logits=torch.zeros(max(window_logits_count(p, s), 1), dtype=torch.float32, device=device),
        workspace=nb(ws) if ws else None,
        out=torch.zeros((s.batch, s.num_q_heads, s.head_dim), dtype=torch.float32, device=device),
    )


def plan_views(p: Params, s: Shape, plan_buf: torch.Tensor):
    """(count [B*Hkv], flags [B*Hkv], indices [B*Hkv, cap]) int32 views."""
    L = plan_layout(p, s)
    pairs = s.batch * s.num_kv_heads
    i32 = lambda off, n: plan_buf[off:off + 4 * n].view(torch.int32)
    idx = i32(L.indices_offset, pairs * L.cap).view(pairs, L.cap)
    return i32(L.count_offset, pairs), i32(L.flags_offset, pairs), idx


def state_views(p: Params, s: Shape, state_buf: torch.Tensor):
    """(count [B*Hkv] int32, flags [B*Hkv] int32, offsets [B*Hkv, cap] as
    int16 bit patterns of the stored uint16 values)."""
    L = state_layout(p, s)
    pairs = s.batch * s.num_kv_heads
    cnt = state_buf[L.count_offset:L.count_offset + 4 * pairs].view(torch.int32)
    flg = state_buf[L.flags_offset:L.flags_offset + 4 * pairs].view(torch.int32)
    off = state_buf[L.offsets_offset:L.offsets_offset + 2 * pairs * L.cap].view(torch.int16)
    return cnt, flg, off.view(pairs, L.cap)


def kept_views(p: Params, s: Shape, state_buf: torch.Tensor):
    """(tags [B*Hkv, 2] int32: k + 1 for the list of slot s after k skip
    entries, 0 for none; lists [B*Hkv, 2, kept_stride] as int16 bit patterns
    of the stored uint16 kept offsets, largest first)."""
    L = state_layout(p, s)
    pairs = s.batch * s.num_kv_heads
    tags = state_buf[L.kept_count_offset:L.kept_count_offset + 8 * pairs].view(torch.int32)
    n = 2 * pairs * L.kept_stride
    lists = state_buf[L.kept_offset:L.kept_offset + 2 * n].view(torch.int16)
    return tags.view(pairs, 2), lists.view(pairs, 2, L.kept_stride)
