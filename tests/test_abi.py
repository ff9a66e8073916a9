"""The C ABI without a GPU: the header compiles as C, the library loads and
exports every function the header declares, size queries are consistent, and
every argument error is reported before any device work is launched."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2608_00916_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_\w+)\s*\(", text)))


def test_header_compiles_as_c():
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-fsyntax-only", "-x", "c", HEADER],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_library_exports_every_declared_function():
    L = _lib.lib()
    names = declared_functions()
    assert len(names) >= 16
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(_lib.EXPORTS)


def D(T=256, H=128, E=8, F=256, k=2, flags=0, aux=0.0, zl=0.0):
    return _lib.MoeDims(T, H, E, F, k, flags, aux, zl)


def test_size_queries():
    L = _lib.lib()
    d = D()
    saved = L.moe_saved_bytes(ctypes.byref(d))
    R = 256 * 2
    # at least Xp, G, U, A, O and the routing tables
    assert saved >= R * (128 * 2 * 2 + 256 * 2 * 3) + 256 * 8 * 4
    assert L.moe_fwd_workspace_bytes(ctypes.byref(d)) > 0
    assert L.moe_bwd_workspace_bytes(ctypes.byref(d)) >= R * 128 * 2 + 2 * R * 256 * 2
    # sizes grow with T and are 0 for invalid dims
    assert L.moe_saved_bytes(ctypes.byref(D(T=512))) > saved
    assert L.moe_saved_bytes(ctypes.byref(D(H=100))) == 0
    ed = _lib.MoeExpertsDims(1000, 256, 4, 128, 0)
    assert L.moe_experts_saved_bytes(ctypes.byref(ed)) >= 3 * 1000 * 128 * 2
    assert L.moe_experts_workspace_bytes(ctypes.byref(ed)) >= 2 * 1000 * 128 * 2
    assert L.moe_version() >= 100


def test_saved_views_are_disjoint_and_aligned():
    L = _lib.lib()
    d = D()
    base = 1 << 20
    v = _lib.MoeSavedView()
    assert L.moe_saved_views(ctypes.byref(d), base, ctypes.byref(v)) == 0
    ptrs = [getattr(v, n) for n, _ in _lib.MoeSavedView._fields_]
    assert all(p % 256 == 0 for p in ptrs)
    assert len(set(ptrs)) == len(ptrs) and sorted(ptrs) == ptrs
    assert ptrs[-1] < base + L.moe_saved_bytes(ctypes.byref(d))


FAKE = 1 << 24  # aligned, never dereferenced: every call below fails its checks first


def fwd(d, **over):
    a = dict(x=FAKE, w_r=FAKE, w_gate=FAKE, w_up=FAKE, w_down=FAKE, mask=None, y=FAKE, saved=FAKE,
             ws=FAKE, ws_bytes=1 << 40)
    a.update(over)
    L = _lib.lib()
    return L.moe_fwd(ctypes.byref(d), a["x"], a["w_r"], a["w_gate"], a["w_up"], a["w_down"], a["mask"],
                     a["y"], a["saved"], a["ws"], a["ws_bytes"], None)


def bwd(d, **over):
    a = dict(x=FAKE, w_r=FAKE, w_gate=FAKE, w_up=FAKE, w_down=FAKE, dy=FAKE, saved=FAKE, dx=FAKE,
             dw_r=FAKE, dw_gate=FAKE, dw_up=FAKE, dw_down=FAKE, ws=FAKE, ws_bytes=1 << 40)
    a.update(over)
    L = _lib.lib()
    return L.moe_bwd(ctypes.byref(d), a["x"], a["w_r"], a["w_gate"], a["w_up"], a["w_down"], a["dy"],
                     a["saved"], a["dx"], a["dw_r"], a["dw_gate"], a["dw_up"], a["dw_down"], a["ws"],
                     a["ws_bytes"], None)


@pytest.mark.parametrize("dims,code", [
    (D(T=0), _lib.MOE_ERR_ARG),
    (D(k=0), _lib.MOE_ERR_ARG),
    (D(k=9), _lib.MOE_ERR_ARG),                 # k > E
    (D(E=264, k=2), _lib.MOE_ERR_ARG),          # E above the limit
    (D(E=64, k=33), _lib.MOE_ERR_ARG),          # k above the limit
    (D(H=100), _lib.MOE_ERR_SHAPE),
    (D(F=200), _lib.MOE_ERR_SHAPE),
    (D(E=12), _lib.MOE_ERR_SHAPE),
    (D(flags=8), _lib.MOE_ERR_ARG),
    (D(aux=-0.01), _lib.MOE_ERR_ARG),           # router-loss coefficients >= 0
    (D(zl=float("nan")), _lib.MOE_ERR_ARG),
    (D(aux=float("inf")), _lib.MOE_ERR_ARG),
])
def test_bad_dims(dims, code):
    assert fwd(dims) == code
    assert bwd(dims) == code
    assert _lib.lib().moe_last_error().decode() != ""


def test_bad_pointers_and_workspace():
    d = D()
    assert fwd(d, x=None) == _lib.MOE_ERR_ARG
    assert "x is NULL" in _lib.lib().moe_last_error().decode()
    assert fwd(d, w_down=FAKE + 8) == _lib.MOE_ERR_ALIGN
    assert fwd(D(flags=_lib.MOE_F_MASK)) == _lib.MOE_ERR_ARG  # mask flag without mask
    assert fwd(d, ws_bytes=0) == _lib.MOE_ERR_WORKSPACE
    assert bwd(d, dy=None) == _lib.MOE_ERR_ARG
    assert bwd(d, dw_r=FAKE + 4) == _lib.MOE_ERR_ALIGN
    assert bwd(d, ws_bytes=1024) == _lib.MOE_ERR_WORKSPACE
    L = _lib.lib()
    ed = _lib.MoeExpertsDims(100, 128, 4, 128, 0)
    assert L.moe_experts_fwd(ctypes.byref(ed), FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, None, 0,
                             None) == _lib.MOE_ERR_ARG
    bad = _lib.MoeExpertsDims(100, 128, 4, 100, 0)
    assert L.moe_experts_fwd(ctypes.byref(bad), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, 0,
                             None) == _lib.MOE_ERR_SHAPE
    assert L.moe_experts_bwd(ctypes.byref(ed), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                             FAKE, FAKE, 16, None) == _lib.MOE_ERR_WORKSPACE


def test_trace_api_without_launches():
    L = _lib.lib()
    assert L.moe_trace_enable(0) == 0
    n = L.moe_trace_read(None, None, 0)
    assert n >= 17
    names = {L.moe_trace_name(i).decode() for i in range(n)}
    assert {"router_logits", "topk", "gateup_fwd", "gateup_wgrad", "combine", "router_dx"} <= names
    assert L.moe_trace_name(-1).decode() == ""


def test_recompute_flag_layout():
    """MOE_F_RECOMPUTE drops G and U from the saved buffer (views NULL)."""
    L = _lib.lib()
    d, dr = D(), D(flags=_lib.MOE_F_RECOMPUTE)
    R, F = 256 * 2, 256
    assert L.moe_saved_bytes(ctypes.byref(d)) - L.moe_saved_bytes(ctypes.byref(dr)) == 2 * R * F * 2
    v = _lib.MoeSavedView()
    assert L.moe_saved_views(ctypes.byref(dr), 1 << 20, ctypes.byref(v)) == 0
    assert v.g is None and v.u is None and v.a is not None and v.o is not None
    ed = _lib.MoeExpertsDims(1000, 256, 4, 128, _lib.MOE_F_RECOMPUTE)
    ev = _lib.MoeExpertsSavedView()
    assert L.moe_experts_saved_views(ctypes.byref(ed), 1 << 20, ctypes.byref(ev)) == 0
    assert ev.g is None and ev.u is None and ev.a is not None
    full = _lib.MoeExpertsDims(1000, 256, 4, 128, 0)
    assert (L.moe_experts_saved_bytes(ctypes.byref(full)) - L.moe_experts_saved_bytes(ctypes.byref(ed))
            == 2 * 1000 * 128 * 2)


def test_router_loss_workspaces():
    """Router losses on: the forward workspace holds their partial sums and the
    backward workspace the dense dz W_r^T term; the saved buffer is unchanged."""
    L = _lib.lib()
    d, da = D(), D(aux=0.01, zl=0.001)
    assert L.moe_saved_bytes(ctypes.byref(d)) == L.moe_saved_bytes(ctypes.byref(da))
    assert L.moe_fwd_workspace_bytes(ctypes.byref(da)) >= L.moe_fwd_workspace_bytes(ctypes.byref(d)) + 64 * 9 * 4
    assert L.moe_bwd_workspace_bytes(ctypes.byref(da)) >= L.moe_bwd_workspace_bytes(ctypes.byref(d)) + 256 * 128 * 4
    v = _lib.MoeSavedView()
    assert L.moe_saved_views(ctypes.byref(da), 1 << 20, ctypes.byref(v)) == 0
    assert v.router_loss is not None and v.router_loss % 256 == 0


def test_lora_sizes_and_errors():
    L = _lib.lib()
    d = D()
    base = L.moe_saved_bytes(ctypes.byref(d))
    assert L.moe_lora_saved_bytes(ctypes.byref(d), 16) >= base + 2 * 256 * 2 * 16 * 2
    assert L.moe_lora_workspace_bytes(ctypes.byref(d), 32) >= L.moe_bwd_workspace_bytes(ctypes.byref(d))
    for bad in (0, 8, 24, 80):
        assert L.moe_lora_saved_bytes(ctypes.byref(d), bad) == 0
    lo = _lib.MoeLora(16, 2.0, FAKE, FAKE, FAKE, FAKE, FAKE)
    ws = 1 << 40

    def fwd_l(lora, dims=d):
        return L.moe_lora_fwd(ctypes.byref(dims), FAKE, FAKE, FAKE, FAKE, FAKE, lora, None, FAKE, FAKE, FAKE, ws,
                              None)
    assert fwd_l(None) == _lib.MOE_ERR_ARG
    assert fwd_l(ctypes.byref(_lib.MoeLora(24, 2.0, FAKE, FAKE, FAKE, FAKE, FAKE))) == _lib.MOE_ERR_SHAPE
    assert fwd_l(ctypes.byref(_lib.MoeLora(16, float("nan"), FAKE, FAKE, FAKE, FAKE, FAKE))) == _lib.MOE_ERR_ARG
    assert fwd_l(ctypes.byref(_lib.MoeLora(16, 2.0, FAKE, None, FAKE, FAKE, FAKE))) == _lib.MOE_ERR_ARG
    assert fwd_l(ctypes.byref(_lib.MoeLora(16, 2.0, FAKE, FAKE, FAKE, FAKE + 2, FAKE))) == _lib.MOE_ERR_ALIGN
    assert L.moe_lora_bwd(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, ctypes.byref(lo), FAKE, FAKE, FAKE, FAKE,
                          FAKE, FAKE, FAKE, FAKE, FAKE, 16, None) == _lib.MOE_ERR_WORKSPACE
    assert L.moe_lora_bwd(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, ctypes.byref(lo), FAKE, FAKE, FAKE, None,
                          FAKE, FAKE, FAKE, FAKE, FAKE, ws, None) == _lib.MOE_ERR_ARG


@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="a GPU is present: this test would launch on fake pointers")
def test_launch_failure_maps_to_moe_err_hip():
    """A launch the HIP runtime refuses (here: no GPU in the machine) comes
    back as MOE_ERR_HIP with the runtime's message, after every argument check
    has passed (valid sizes, non-null 16-byte aligned pointers that are never
    dereferenced on the host)."""
    L = _lib.lib()
    d = D()
    fake = 1 << 20
    rc = L.moe_fwd(ctypes.byref(d), fake, fake, fake, fake, fake, None, fake, fake, fake, 1 << 30, None)
    assert rc == _lib.MOE_ERR_HIP, rc
    msg = L.moe_last_error().decode()
    assert msg.startswith("router:") and len(msg) > len("router: ")


def test_noalloc_forward_rejects_sizes_beyond_its_scratch():
    """moe_fwd_noalloc refuses a batch whose forward scratch exceeds the
    static array, with MOE_ERR_WORKSPACE, before any device call (the
    pointers here are never dereferenced), and accepts the workspace query's
    own limit arithmetic: T = 65536 at E = 128 needs more, T = 8192 less."""
    L = _lib.lib()
    big = D(T=65536, H=2048, E=128, F=768, k=8)
    small = D(T=8192, H=2048, E=128, F=768, k=8)
    assert L.moe_fwd_workspace_bytes(ctypes.byref(big)) > _lib.MOE_NOALLOC_SCRATCH_BYTES
    assert L.moe_fwd_workspace_bytes(ctypes.byref(small)) <= _lib.MOE_NOALLOC_SCRATCH_BYTES
    fake = 1 << 20
    rc = L.moe_fwd_noalloc(ctypes.byref(big), fake, fake, fake, fake, fake, None, fake, fake, None)
    assert rc == _lib.MOE_ERR_WORKSPACE
    assert "static array" in L.moe_last_error().decode()
    # invalid dims are reported first, as by moe_fwd
    assert L.moe_fwd_noalloc(ctypes.byref(D(H=100)), fake, fake, fake, fake, fake, None, fake, fake,
                             None) == _lib.MOE_ERR_SHAPE
