"""The allocation-free forward (moe_fwd_noalloc) against moe_fwd through the
C ABI: the same kernels with the scratch in the library's static array, so
every output and every routing table and activation it saves must match
moe_fwd's bit for bit.  Two calls in a row share the array, the second with a
smaller batch (and a mask); the backward from the allocation-free forward's
saved buffer matches the one from moe_fwd's."""
import numpy as np
import pytest

import workloads
from tests.parity import dev_bf16, host

pytestmark = pytest.mark.gpu

NAMES = ("logits", "topk_idx", "gates", "counts", "offsets", "row_token", "row_of", "xp", "g", "u", "a", "o")


def run_pair(shape, mask_every=0):
    import torch
    import paper_2608_00916_amd as moe
    inp = workloads.block_inputs(**shape)
    d = inp["dims"]
    T = d["T"]
    print(f"GPU no-alloc T={T} H={d['H']} E={d['E']} k={d['k']} F={d['F']} mask_every={mask_every}", flush=True)
    t = {n: dev_bf16(inp[n]) for n in ("x", "w_r", "w_gate", "w_up", "w_down", "dy")}
    tm = None
    if mask_every:
        tm = torch.from_numpy((np.arange(T) % mask_every != 1).astype(np.uint8)).cuda()
    ref = moe.MoEBlock(T, d["H"], d["E"], d["F"], d["k"], mask=tm is not None)
    nal = moe.MoEBlock(T, d["H"], d["E"], d["F"], d["k"], mask=tm is not None)
    assert moe.moe_fwd_workspace_bytes(nal.d) <= moe.MOE_NOALLOC_SCRATCH_BYTES
    nal.saved.fill_(0x5A)
    nal.y.fill_(7.0)
    ref.forward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], tm)
    moe.moe_fwd_noalloc(nal.d, t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], tm, nal.y, nal.saved)
    torch.cuda.synchronize()
    assert torch.equal(nal.y, ref.y)
    R = int(ref.views["offsets"][-1].item())
    for n in NAMES:
        a, b = ref.views[n], nal.views[n]
        if n in ("xp", "g", "u", "a", "o"):
            a, b = a[:R], b[:R]
        assert np.array_equal(host(a), host(b)), n
    for blk in (ref, nal):
        blk.backward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], t["dy"])
    torch.cuda.synchronize()
    for n in ("dx", "dw_r", "dw_gate", "dw_up", "dw_down"):
        assert torch.equal(getattr(nal, n), getattr(ref, n)), n


def test_noalloc_forward_matches_moe_fwd_twice():
    # a larger batch first (several 128-row tiles per expert, ragged), then a
    # smaller masked one through the same static array
    run_pair(dict(T=3000, H=512, E=32, k=4, F=384, seed=71))
    run_pair(dict(T=300, H=256, E=16, k=2, F=256, seed=72), mask_every=5)
