"""MI355X-native mixture-of-experts FFN block (forward + backward).

Python binding of the C ABI in include/moe.h, with the same entry-point names.
Torch supplies device memory and streams; the block itself runs entirely in
the gfx950 HIP kernels of libmoe.so.  The functions here only turn tensors into
pointers (and, in MoEBlock / MoEExperts, allocate the caller-owned buffers).
"""
from __future__ import annotations

import ctypes

import torch

from . import _lib
from ._lib import (MOE_F_DW_FP32, MOE_F_MASK, MOE_F_RECOMPUTE, MOE_MAX_EXPERTS, MOE_MAX_TOPK,
                   MOE_NOALLOC_SCRATCH_BYTES, MoeDims,
                   MoeError, MoeExpertsDims, MoeExpertsSavedView, MoeLora, MoeSavedView, check, lib)

__all__ = [
    "dims", "experts_dims", "moe_saved_bytes", "moe_fwd_workspace_bytes",
    "moe_bwd_workspace_bytes", "moe_saved_views", "moe_fwd", "moe_fwd_noalloc", "moe_bwd",
    "moe_infer_workspace_bytes", "moe_infer", "MoEInfer",
    "moe_lora_saved_bytes", "moe_lora_workspace_bytes", "moe_lora_fwd", "moe_lora_bwd", "lora_args", "MoELoRA",
    "moe_experts_saved_bytes", "moe_experts_workspace_bytes", "moe_experts_saved_views",
    "moe_experts_fwd", "moe_experts_bwd", "moe_last_error", "moe_version",
    "moe_trace_enable", "moe_trace_read", "MoEBlock", "MoEExperts", "MoeError", "MOE_F_MASK", "MOE_F_DW_FP32",
    "MOE_F_RECOMPUTE",
    "MOE_MAX_EXPERTS", "MOE_MAX_TOPK",
]


def dims(T, H, E, F, top_k, mask=False, dw_fp32=False, recompute=False, aux_loss_coef=0.0,
         z_loss_coef=0.0) -> MoeDims:
    flags = ((MOE_F_MASK if mask else 0) | (MOE_F_DW_FP32 if dw_fp32 else 0)
             | (MOE_F_RECOMPUTE if recompute else 0))
    return MoeDims(T, H, E, F, top_k, flags, aux_loss_coef, z_loss_coef)


def experts_dims(rows, H, E, F, dw_fp32=False, recompute=False) -> MoeExpertsDims:
    return MoeExpertsDims(rows, H, E, F, (MOE_F_DW_FP32 if dw_fp32 else 0)
                          | (MOE_F_RECOMPUTE if recompute else 0))


def _p(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("tensor must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _s(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def moe_last_error() -> str:
    return lib().moe_last_error().decode()


def moe_version() -> int:
    return lib().moe_version()


def moe_trace_enable(on: bool) -> None:
    check(lib().moe_trace_enable(1 if on else 0))


def moe_trace_read() -> dict:
    """{kernel name: (total ms, launches)} since the last read (waits for the
    recorded events)."""
    n = 64
    ms = (ctypes.c_double * n)()
    cnt = (ctypes.c_int32 * n)()
    m = lib().moe_trace_read(ms, cnt, n)
    if m < 0:
        check(m)
    return {lib().moe_trace_name(i).decode(): (ms[i], cnt[i]) for i in range(m) if cnt[i]}


# ------------------------------------------------------------------ full block
def moe_saved_bytes(d: MoeDims) -> int:
    return lib().moe_saved_bytes(ctypes.byref(d))


def moe_fwd_workspace_bytes(d: MoeDims) -> int:
    return lib().moe_fwd_workspace_bytes(ctypes.byref(d))


def moe_bwd_workspace_bytes(d: MoeDims) -> int:
    return lib().moe_bwd_workspace_bytes(ctypes.byref(d))


def _view(base: torch.Tensor, ptr: int, dtype, shape):
    if ptr is None:  # a region the flags leave out
        return None
    off = ptr - base.data_ptr()
    n = 1
    for s in shape:
        n *= s
    nbytes = n * torch.empty((), dtype=dtype).element_size()
    return base[off:off + nbytes].view(dtype).view(shape)


def moe_saved_views(d: MoeDims, saved: torch.Tensor) -> dict:
    """Tensors viewing the routing and activations inside a `saved` buffer."""
    v = MoeSavedView()
    check(lib().moe_saved_views(ctypes.byref(d), _p(saved), ctypes.byref(v)))
    T, H, E, F, k = d.T, d.H, d.E, d.F, d.top_k
    R = T * k
    i32, f32, bf = torch.int32, torch.float32, torch.bfloat16
    return dict(
        logits=_view(saved, v.logits, f32, (T, E)),
        topk_idx=_view(saved, v.topk_idx, i32, (T, k)),
        gates=_view(saved, v.gates, f32, (T, k)),
        counts=_view(saved, v.counts, i32, (E,)),
        offsets=_view(saved, v.offsets, i32, (E + 1,)),
        row_token=_view(saved, v.row_token, i32, (R,)),
        row_of=_view(saved, v.row_of, i32, (T, k)),
        xp=_view(saved, v.xp, bf, (R, H)),
        g=_view(saved, v.g, bf, (R, F)),
        u=_view(saved, v.u, bf, (R, F)),
        a=_view(saved, v.a, bf, (R, F)),
        o=_view(saved, v.o, bf, (R, H)),
        router_loss=_view(saved, v.router_loss, f32, (2,)),
    )


def moe_fwd(d, x, w_r, w_gate, w_up, w_down, token_mask, y, saved, ws, stream=None):
    check(lib().moe_fwd(ctypes.byref(d), _p(x), _p(w_r), _p(w_gate), _p(w_up), _p(w_down),
                        _p(token_mask), _p(y), _p(saved), _p(ws),
                        0 if ws is None else ws.numel() * ws.element_size(), _s(stream)))


def moe_fwd_noalloc(d, x, w_r, w_gate, w_up, w_down, token_mask, y, saved, stream=None):
    """moe_fwd with the library's static scratch instead of a workspace."""
    check(lib().moe_fwd_noalloc(ctypes.byref(d), _p(x), _p(w_r), _p(w_gate), _p(w_up), _p(w_down),
                                _p(token_mask), _p(y), _p(saved), _s(stream)))


def moe_bwd(d, x, w_r, w_gate, w_up, w_down, dy, saved, dx, dw_r, dw_gate, dw_up, dw_down, ws,
            stream=None):
    check(lib().moe_bwd(ctypes.byref(d), _p(x), _p(w_r), _p(w_gate), _p(w_up), _p(w_down), _p(dy),
                        _p(saved), _p(dx), _p(dw_r), _p(dw_gate), _p(dw_up), _p(dw_down), _p(ws),
                        0 if ws is None else ws.numel() * ws.element_size(), _s(stream)))


# ------------------------------------------------------------------ forward only
def moe_infer_workspace_bytes(d: MoeDims) -> int:
    return lib().moe_infer_workspace_bytes(ctypes.byref(d))


def moe_infer(d, x, w_r, w_gate, w_up, w_down, token_mask, y, ws, stream=None):
    check(lib().moe_infer(ctypes.byref(d), _p(x), _p(w_r), _p(w_gate), _p(w_up), _p(w_down),
                          _p(token_mask), _p(y), _p(ws),
                          0 if ws is None else ws.numel() * ws.element_size(), _s(stream)))


# ------------------------------------------------------------------ expert LoRA
def lora_args(rank, scale, a1, b1_gate, b1_up, a2, b2) -> MoeLora:
    """The adapter descriptor (device tensors stay owned by the caller)."""
    return MoeLora(rank, scale, _p(a1), _p(b1_gate), _p(b1_up), _p(a2), _p(b2))


def moe_lora_saved_bytes(d: MoeDims, rank: int) -> int:
    return lib().moe_lora_saved_bytes(ctypes.byref(d), rank)


def moe_lora_workspace_bytes(d: MoeDims, rank: int) -> int:
    return lib().moe_lora_workspace_bytes(ctypes.byref(d), rank)


def moe_lora_fwd(d, x, w_r, w_gate, w_up, w_down, lora: MoeLora, token_mask, y, saved, ws, stream=None):
    check(lib().moe_lora_fwd(ctypes.byref(d), _p(x), _p(w_r), _p(w_gate), _p(w_up), _p(w_down),
                             ctypes.byref(lora), _p(token_mask), _p(y), _p(saved), _p(ws),
                             0 if ws is None else ws.numel() * ws.element_size(), _s(stream)))


def moe_lora_bwd(d, x, w_r, w_gate, w_up, w_down, lora: MoeLora, dy, saved, dx, da1, db1_gate, db1_up, da2, db2,
                 ws, stream=None):
    check(lib().moe_lora_bwd(ctypes.byref(d), _p(x), _p(w_r), _p(w_gate), _p(w_up), _p(w_down),
                             ctypes.byref(lora), _p(dy), _p(saved), _p(dx), _p(da1), _p(db1_gate), _p(db1_up),
                             _p(da2), _p(db2), _p(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                             _s(stream)))


# ------------------------------------------------------------------ experts only
def moe_experts_saved_bytes(d: MoeExpertsDims) -> int:
    return lib().moe_experts_saved_bytes(ctypes.byref(d))


def moe_experts_workspace_bytes(d: MoeExpertsDims) -> int:
    return lib().moe_experts_workspace_bytes(ctypes.byref(d))


def moe_experts_saved_views(d: MoeExpertsDims, saved: torch.Tensor) -> dict:
    v = MoeExpertsSavedView()
    check(lib().moe_experts_saved_views(ctypes.byref(d), _p(saved), ctypes.byref(v)))
    bf = torch.bfloat16
    return dict(offsets=_view(saved, v.offsets, torch.int32, (d.E + 1,)),
                g=_view(saved, v.g, bf, (d.rows, d.F)), u=_view(saved, v.u, bf, (d.rows, d.F)),
                a=_view(saved, v.a, bf, (d.rows, d.F)))


def moe_experts_fwd(d, xp, counts, w_gate, w_up, w_down, o, saved, ws, stream=None):
    check(lib().moe_experts_fwd(ctypes.byref(d), _p(xp), _p(counts), _p(w_gate), _p(w_up),
                                _p(w_down), _p(o), _p(saved), _p(ws),
                                0 if ws is None else ws.numel() * ws.element_size(), _s(stream)))


def moe_experts_bwd(d, xp, w_gate, w_up, w_down, d_o, saved, dxp, dw_gate, dw_up, dw_down, ws,
                    stream=None):
    check(lib().moe_experts_bwd(ctypes.byref(d), _p(xp), _p(w_gate), _p(w_up), _p(w_down),
                                _p(d_o), _p(saved), _p(dxp), _p(dw_gate), _p(dw_up), _p(dw_down),
                                _p(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                                _s(stream)))


# ------------------------------------------------------------------ owners of buffers
class MoEBlock:
    """Caller-side buffers for one block shape: saved activations, workspaces
    and outputs, allocated once with torch on `device`."""

    def __init__(self, T, H, E, F, top_k, mask=False, dw_fp32=False, recompute=False, aux_loss_coef=0.0,
                 z_loss_coef=0.0, device="cuda"):
        self.d = dims(T, H, E, F, top_k, mask, dw_fp32, recompute, aux_loss_coef, z_loss_coef)
        nb = moe_saved_bytes(self.d)
        if nb == 0:
            raise MoeError(_lib.MOE_ERR_ARG, moe_last_error())
        dev = torch.device(device)
        self.saved = torch.empty(nb, dtype=torch.uint8, device=dev)
        ws = max(moe_fwd_workspace_bytes(self.d), moe_bwd_workspace_bytes(self.d))
        self.ws = torch.empty(ws, dtype=torch.uint8, device=dev)
        wdt = torch.float32 if dw_fp32 else torch.bfloat16
        self.y = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
        self.dx = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
        self.dw_r = torch.empty((H, E), dtype=wdt, device=dev)
        self.dw_gate = torch.empty((E, H, F), dtype=wdt, device=dev)
        self.dw_up = torch.empty((E, H, F), dtype=wdt, device=dev)
        self.dw_down = torch.empty((E, F, H), dtype=wdt, device=dev)
        self.views = moe_saved_views(self.d, self.saved)

    def forward(self, x, w_r, w_gate, w_up, w_down, token_mask=None, stream=None):
        moe_fwd(self.d, x, w_r, w_gate, w_up, w_down, token_mask, self.y, self.saved, self.ws, stream)
        return self.y

    def backward(self, x, w_r, w_gate, w_up, w_down, dy, stream=None):
        moe_bwd(self.d, x, w_r, w_gate, w_up, w_down, dy, self.saved, self.dx, self.dw_r,
                self.dw_gate, self.dw_up, self.dw_down, self.ws, stream)
        return self.dx, self.dw_r, self.dw_gate, self.dw_up, self.dw_down


class MoEExperts:
    """Caller-side buffers for one expert-parallel rank's local experts."""

    def __init__(self, rows, H, E, F, dw_fp32=False, recompute=False, device="cuda"):
        self.d = experts_dims(rows, H, E, F, dw_fp32, recompute)
        dev = torch.device(device)
        self.saved = torch.empty(moe_experts_saved_bytes(self.d), dtype=torch.uint8, device=dev)
        self.ws = torch.empty(moe_experts_workspace_bytes(self.d), dtype=torch.uint8, device=dev)
        wdt = torch.float32 if dw_fp32 else torch.bfloat16
        self.o = torch.empty((rows, H), dtype=torch.bfloat16, device=dev)
        self.dxp = torch.empty((rows, H), dtype=torch.bfloat16, device=dev)
        self.dw_gate = torch.empty((E, H, F), dtype=wdt, device=dev)
        self.dw_up = torch.empty((E, H, F), dtype=wdt, device=dev)
        self.dw_down = torch.empty((E, F, H), dtype=wdt, device=dev)
        self.views = moe_experts_saved_views(self.d, self.saved)

    def forward(self, xp, counts, w_gate, w_up, w_down, stream=None):
        moe_experts_fwd(self.d, xp, counts, w_gate, w_up, w_down, self.o, self.saved, self.ws, stream)
        return self.o

    def backward(self, xp, w_gate, w_up, w_down, d_o, stream=None):
        moe_experts_bwd(self.d, xp, w_gate, w_up, w_down, d_o, self.saved, self.dxp, self.dw_gate,
                        self.dw_up, self.dw_down, self.ws, stream)
        return self.dxp, self.dw_gate, self.dw_up, self.dw_down


class MoEInfer:
    """Caller-side buffers of the forward-only (serving) pass: workspace and
    output for one block shape."""

    def __init__(self, T, H, E, F, top_k, mask=False, device="cuda"):
        self.d = dims(T, H, E, F, top_k, mask)
        nb = moe_infer_workspace_bytes(self.d)
        if nb == 0:
            raise MoeError(_lib.MOE_ERR_ARG, moe_last_error())
        dev = torch.device(device)
        self.ws = torch.empty(nb, dtype=torch.uint8, device=dev)
        self.y = torch.empty((T, H), dtype=torch.bfloat16, device=dev)

    def forward(self, x, w_r, w_gate, w_up, w_down, token_mask=None, stream=None):
        moe_infer(self.d, x, w_r, w_gate, w_up, w_down, token_mask, self.y, self.ws, stream)
        return self.y


class MoELoRA:
    """Caller-side buffers of the block with rank-r expert adapters: saved
    activations, workspace, dX and the adapter gradients."""

    def __init__(self, T, H, E, F, top_k, rank, mask=False, dw_fp32=False, recompute=False, aux_loss_coef=0.0,
                 z_loss_coef=0.0, device="cuda"):
        self.d = dims(T, H, E, F, top_k, mask, dw_fp32, recompute, aux_loss_coef, z_loss_coef)
        self.rank = rank
        nb = moe_lora_saved_bytes(self.d, rank)
        if nb == 0:
            raise MoeError(_lib.MOE_ERR_ARG, "invalid dims or LoRA rank")
        dev = torch.device(device)
        self.saved = torch.empty(nb, dtype=torch.uint8, device=dev)
        self.ws = torch.empty(moe_lora_workspace_bytes(self.d, rank), dtype=torch.uint8, device=dev)
        wdt = torch.float32 if dw_fp32 else torch.bfloat16
        self.y = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
        self.dx = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
        self.da1 = torch.empty((E, H, rank), dtype=wdt, device=dev)
        self.db1_gate = torch.empty((E, rank, F), dtype=wdt, device=dev)
        self.db1_up = torch.empty((E, rank, F), dtype=wdt, device=dev)
        self.da2 = torch.empty((E, F, rank), dtype=wdt, device=dev)
        self.db2 = torch.empty((E, rank, H), dtype=wdt, device=dev)
        self.views = moe_saved_views(self.d, self.saved)

    def forward(self, x, w_r, w_gate, w_up, w_down, lora: MoeLora, token_mask=None, stream=None):
        moe_lora_fwd(self.d, x, w_r, w_gate, w_up, w_down, lora, token_mask, self.y, self.saved, self.ws, stream)
        return self.y

    def backward(self, x, w_r, w_gate, w_up, w_down, lora: MoeLora, dy, stream=None):
        moe_lora_bwd(self.d, x, w_r, w_gate, w_up, w_down, lora, dy, self.saved, self.dx, self.da1, self.db1_gate,
                     self.db1_up, self.da2, self.db2, self.ws, stream)
        return self.dx, self.da1, self.db1_gate, self.db1_up, self.da2, self.db2
