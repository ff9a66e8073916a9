"""GPU parity of the expert-LoRA entry points (moe_lora_fwd / moe_lora_bwd)
against the oracle's lora_forward / lora_backward: Y, dX and the five adapter
gradients element by element, over ragged tiles, empty experts, masked tokens,
every supported rank, fp32 gradients, the recompute flag (bit-identical) and
the router losses."""
import numpy as np
import pytest

import workloads
from oracle import moe_oracle as O
from tests.parity import assert_close, check_routing, dev_bf16, host, touched_experts

pytestmark = pytest.mark.gpu

ADAPTERS = ("a1", "b1_gate", "b1_up", "a2", "b2")


def lora_inputs(inp, rank, seed, std=0.05, scale=2.0):
    d = inp["dims"]
    E, H, F = d["E"], d["H"], d["F"]
    s = np.random.SeedSequence(seed).spawn(5)
    shapes = dict(a1=(E, H, rank), b1_gate=(E, rank, F), b1_up=(E, rank, F), a2=(E, F, rank), b2=(E, rank, H))
    return {n: workloads.normal_bf16(q, shapes[n], std) for n, q in zip(ADAPTERS, s)}, scale


def run(inp, rank, lo_bits, scale, dw_fp32=False, recompute=False, coefs=(0.0, 0.0)):
    import torch
    import paper_2608_00916_amd as moe
    d = inp["dims"]
    mask = inp["mask"]
    print(f"GPU lora T={d['T']} H={d['H']} E={d['E']} k={d['k']} F={d['F']} rank={rank} "
          f"mask={mask is not None} fp32={dw_fp32} recompute={recompute} coefs={coefs}", flush=True)
    t = {n: dev_bf16(inp[n]) for n in ("x", "w_r", "w_gate", "w_up", "w_down", "dy")}
    lt = {n: dev_bf16(lo_bits[n]) for n in ADAPTERS}
    lora = moe.lora_args(rank, scale, *(lt[n] for n in ADAPTERS))
    tm = None if mask is None else torch.from_numpy(mask.astype(np.uint8)).cuda()
    blk = moe.MoELoRA(d["T"], d["H"], d["E"], d["F"], d["k"], rank, mask=tm is not None, dw_fp32=dw_fp32,
                      recompute=recompute, aux_loss_coef=coefs[0], z_loss_coef=coefs[1])
    blk.forward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], lora, tm)
    blk.backward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], lora, t["dy"])
    torch.cuda.synchronize()
    v = blk.views
    out = dict(y=host(blk.y), dx=host(blk.dx), logits=host(v["logits"]), idx=host(v["topk_idx"]),
               gates=host(v["gates"]))
    out.update({"d" + n: host(getattr(blk, "d" + n)) for n in ADAPTERS})
    return out


def oracle(inp, lo_bits, scale, coefs=(0.0, 0.0)):
    d = inp["dims"]
    w = {n: O.widen_bf16(inp[n]) for n in ("x", "w_r", "w_gate", "w_up", "w_down", "dy")}
    lo = {n: O.widen_bf16(lo_bits[n]) for n in ADAPTERS}
    lo["scale"] = scale
    mask = None if inp["mask"] is None else inp["mask"].astype(bool)
    f = O.lora_forward(w["x"], w["w_r"], w["w_gate"], w["w_up"], w["w_down"], lo, d["k"], mask)
    b = O.lora_backward(w["x"], w["w_r"], w["w_gate"], w["w_up"], w["w_down"], lo, f, w["dy"])
    if coefs != (0.0, 0.0):  # the router losses' gradient reaches dX through dz W_r^T
        dz_aux = O.router_aux_dz(f["z"], f["idx"], coefs[0], coefs[1], mask)
        b["dx"] = b["dx"] + dz_aux @ w["w_r"].T
    return f, b, mask


def compare(inp, g, f, b, mask, tol=2e-2, case=None):
    """Y and dX on every token whose expert set matches the oracle's, and the
    adapter gradients of every expert no near-tie flip reaches (see the block
    tests); flips are recorded."""
    d = inp["dims"]
    _, _, flipped = check_routing(f["z"], f["idx"], f["gates"], g["logits"], g["idx"], g["gates"], d["k"], mask,
                                  case=case)
    keep = ~flipped
    assert_close("y", g["y"][keep], f["Y"][keep], case=case)
    assert_close("dx", g["dx"][keep], b["dx"][keep], case=case)
    cols = ~touched_experts(flipped, g["idx"], f["idx"], d["E"])
    empty = np.nonzero(f["counts"] == 0)[0]
    for n in ADAPTERS:
        assert_close("d" + n, g["d" + n][cols], b["d" + n][cols], tol, case=case)
        assert np.all(g["d" + n][empty] == 0), n


CASES = {
    "tiny_r16": (dict(T=256, H=128, E=8, k=2, F=256, seed=61), 16),
    "ragged_multi_tile_r32": (dict(T=1000, H=512, E=8, k=2, F=384, seed=62), 32),
    "empty_experts_r16": (dict(T=257, H=256, E=32, k=3, F=128, seed=63, zipf_s=1.2, n_cold=6), 16),
    "rank64": (dict(T=300, H=256, E=16, k=4, F=256, seed=64), 64),
    "rank48_narrow": (dict(T=200, H=384, E=8, k=2, F=128, seed=65), 48),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_lora_matches_oracle(case):
    shape, rank = CASES[case]
    inp = workloads.block_inputs(**shape)
    lo, scale = lora_inputs(inp, rank, seed=shape["seed"] + 100)
    f, b, mask = oracle(inp, lo, scale)
    compare(inp, run(inp, rank, lo, scale), f, b, mask, case="lora_" + case)


def test_lora_masked_fp32_grads():
    """fp32 adapter gradients: tighter than the bf16 bar, though not as tight
    as the base weight gradients' (the rank-r intermediates P1, P2, Q1, Q2 are
    stored bf16, one more rounding in each product), and really unrounded."""
    inp = workloads.block_inputs(T=333, H=256, E=16, k=2, F=128, seed=66)
    inp["mask"] = (np.arange(333) % 5 != 1).astype(np.uint8)
    lo, scale = lora_inputs(inp, 16, seed=166)
    f, b, mask = oracle(inp, lo, scale)
    g = run(inp, 16, lo, scale, dw_fp32=True)
    compare(inp, g, f, b, mask, tol=1e-2, case="lora_masked_fp32")
    v = g["da1"].astype(np.float32)
    assert np.any(v.view(np.uint32) & 0xFFFF), "fp32 gradients hold only bf16 values"


def test_lora_recompute_is_bit_identical():
    inp = workloads.block_inputs(T=500, H=256, E=8, k=2, F=256, seed=67)
    lo, scale = lora_inputs(inp, 16, seed=167)
    a = run(inp, 16, lo, scale)
    r = run(inp, 16, lo, scale, recompute=True)
    for n in a:
        assert np.array_equal(a[n], r[n]), n


def test_lora_with_router_losses():
    """The frozen router still passes its input gradient, including the
    router losses' part, into dX."""
    inp = workloads.block_inputs(T=256, H=128, E=8, k=2, F=256, seed=68)
    inp["dy"] = workloads.bf16_bits(O.widen_bf16(inp["dy"]) * 1e-2)
    lo, scale = lora_inputs(inp, 16, seed=168)
    coefs = (0.5, 0.05)
    f, b, mask = oracle(inp, lo, scale, coefs)
    g = run(inp, 16, lo, scale, coefs=coefs)
    # the routing counts enter every token's loss gradient: no flip allowed
    _, _, flipped = check_routing(f["z"], f["idx"], f["gates"], g["logits"], g["idx"], g["gates"],
                                  inp["dims"]["k"], mask)
    assert not flipped.any(), "a near tie flipped an expert set on the fixed seed"
    compare(inp, g, f, b, mask, case="lora_router_losses")
