"""ctypes binding of libmoe.so (the C ABI of include/moe.h).

Argument marshalling only: every step of the block runs in the library's HIP
kernels.  Loading fails loudly if the library has not been built; there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmoe.so")

MOE_OK = 0
MOE_ERR_ARG = -1
MOE_ERR_SHAPE = -2
MOE_ERR_ALIGN = -3
MOE_ERR_WORKSPACE = -4
MOE_ERR_HIP = -5
MOE_MAX_EXPERTS = 256
MOE_MAX_TOPK = 32
MOE_F_MASK = 1
MOE_F_DW_FP32 = 2
MOE_F_RECOMPUTE = 4
MOE_NOALLOC_SCRATCH_BYTES = 64 << 20

EXPORTS = (
    "moe_saved_bytes", "moe_fwd_workspace_bytes", "moe_bwd_workspace_bytes",
    "moe_saved_views", "moe_fwd", "moe_fwd_noalloc", "moe_bwd", "moe_infer_workspace_bytes", "moe_infer",
    "moe_lora_saved_bytes", "moe_lora_workspace_bytes", "moe_lora_fwd", "moe_lora_bwd",
    "moe_experts_saved_bytes", "moe_experts_workspace_bytes",
    "moe_experts_saved_views", "moe_experts_fwd", "moe_experts_bwd",
    "moe_trace_enable", "moe_trace_read", "moe_trace_name",
    "moe_last_error", "moe_version",
)


class MoeDims(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("H", ctypes.c_int32), ("E", ctypes.c_int32),
                ("F", ctypes.c_int32), ("top_k", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("aux_loss_coef", ctypes.c_float), ("z_loss_coef", ctypes.c_float)]


class MoeSavedView(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "logits", "topk_idx", "gates", "counts", "offsets", "row_token", "row_of",
        "xp", "g", "u", "a", "o", "router_loss")]


class MoeLora(ctypes.Structure):
    _fields_ = [("rank", ctypes.c_int32), ("scale", ctypes.c_float),
                ("a1", ctypes.c_void_p), ("b1_gate", ctypes.c_void_p), ("b1_up", ctypes.c_void_p),
                ("a2", ctypes.c_void_p), ("b2", ctypes.c_void_p)]


class MoeExpertsDims(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int32), ("H", ctypes.c_int32), ("E", ctypes.c_int32),
                ("F", ctypes.c_int32), ("flags", ctypes.c_uint32)]


class MoeExpertsSavedView(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("offsets", "g", "u", "a")]


class MoeError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{msg} (code {code})")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2608_00916_amd.build` "
            "(there is no fallback implementation)")
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    S = ctypes.c_size_t
    D = ctypes.POINTER(MoeDims)
    ED = ctypes.POINTER(MoeExpertsDims)
    sig = {
        "moe_saved_bytes": (S, [D]),
        "moe_fwd_workspace_bytes": (S, [D]),
        "moe_bwd_workspace_bytes": (S, [D]),
        "moe_saved_views": (ctypes.c_int, [D, P, ctypes.POINTER(MoeSavedView)]),
        "moe_fwd": (ctypes.c_int, [D, P, P, P, P, P, P, P, P, P, S, P]),
        "moe_fwd_noalloc": (ctypes.c_int, [D, P, P, P, P, P, P, P, P, P]),
        "moe_bwd": (ctypes.c_int, [D, P, P, P, P, P, P, P, P, P, P, P, P, P, S, P]),
        "moe_infer_workspace_bytes": (S, [D]),
        "moe_lora_saved_bytes": (S, [D, ctypes.c_int32]),
        "moe_lora_workspace_bytes": (S, [D, ctypes.c_int32]),
        "moe_lora_fwd": (ctypes.c_int, [D, P, P, P, P, P, ctypes.POINTER(MoeLora), P, P, P, P, S, P]),
        "moe_lora_bwd": (ctypes.c_int, [D, P, P, P, P, P, ctypes.POINTER(MoeLora), P, P, P, P, P, P, P, P, P, S,
                                        P]),
        "moe_infer": (ctypes.c_int, [D, P, P, P, P, P, P, P, P, S, P]),
        "moe_experts_saved_bytes": (S, [ED]),
        "moe_experts_workspace_bytes": (S, [ED]),
        "moe_experts_saved_views": (ctypes.c_int, [ED, P, ctypes.POINTER(MoeExpertsSavedView)]),
        "moe_experts_fwd": (ctypes.c_int, [ED, P, P, P, P, P, P, P, P, S, P]),
        "moe_experts_bwd": (ctypes.c_int, [ED, P, P, P, P, P, P, P, P, P, P, P, S, P]),
        "moe_trace_enable": (ctypes.c_int, [ctypes.c_int]),
        "moe_trace_read": (ctypes.c_int, [ctypes.POINTER(ctypes.c_double),
                                          ctypes.POINTER(ctypes.c_int32), ctypes.c_int]),
        "moe_trace_name": (ctypes.c_char_p, [ctypes.c_int]),
        "moe_last_error": (ctypes.c_char_p, []),
        "moe_version": (ctypes.c_int, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def check(rc: int) -> None:
    if rc != MOE_OK:
        raise MoeError(rc, lib().moe_last_error().decode())
