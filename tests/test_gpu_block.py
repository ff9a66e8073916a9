"""GPU parity of the whole MoE block (forward + backward) against the fp64
oracle, element by element, at sizes the oracle finishes in seconds: the tiny
workload, ragged token counts spanning several 128-row tiles, empty experts,
k = 1, k = E, the largest E and k, masked and all-masked batches, T = 1, both
weight-gradient dtypes, and bitwise determinism.  Calls go through the C ABI
(libmoe.so via its ctypes binding)."""
import numpy as np
import pytest

import workloads
from oracle import moe_oracle as O
from tests.parity import (Guards, assert_close, check_permutation_valid, check_routing, dev_bf16, host,
                          row_pairs, touched_experts)

pytestmark = pytest.mark.gpu


def oracle_run(inp):
    d = inp["dims"]
    w = {n: O.widen_bf16(inp[n]) for n in ("x", "w_r", "w_gate", "w_up", "w_down", "dy")}
    mask = None if inp["mask"] is None else inp["mask"].astype(bool)
    f = O.moe_forward(w["x"], w["w_r"], w["w_gate"], w["w_up"], w["w_down"], d["k"], mask)
    b = O.moe_backward(w["x"], w["w_r"], w["w_gate"], w["w_up"], w["w_down"], f, w["dy"])
    return f, b


def gpu_run(inp, dw_fp32=False, repeat=1, recompute=False):
    import torch
    import paper_2608_00916_amd as moe
    d = inp["dims"]
    mask = inp["mask"]
    print(f"GPU block T={d['T']} H={d['H']} E={d['E']} k={d['k']} F={d['F']} "
          f"mask={mask is not None} dw_fp32={dw_fp32} recompute={recompute}", flush=True)
    blk = moe.MoEBlock(d["T"], d["H"], d["E"], d["F"], d["k"], mask=mask is not None,
                       dw_fp32=dw_fp32, recompute=recompute)
    # every buffer the library writes sits between sentinel bands
    guards = Guards()
    for n in ("saved", "ws", "y", "dx", "dw_r", "dw_gate", "dw_up", "dw_down"):
        setattr(blk, n, guards.like(getattr(blk, n)))
    blk.views = moe.moe_saved_views(blk.d, blk.saved)
    t = {n: dev_bf16(inp[n]) for n in ("x", "w_r", "w_gate", "w_up", "w_down", "dy")}
    tm = None if mask is None else torch.from_numpy(mask.astype(np.uint8)).cuda()
    outs = []
    for _ in range(repeat):
        blk.forward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], tm)
        blk.backward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], t["dy"])
        torch.cuda.synchronize()
        guards.check()
        v = blk.views
        R = int(v["offsets"][-1].item())
        out = {n: host(v[n]) for n in ("logits", "topk_idx", "gates", "counts", "offsets",
                                      "row_token", "row_of")}
        for n in ("xp", "g", "u", "a", "o"):
            out[n] = None if v[n] is None else host(v[n][:R])
        out.update(y=host(blk.y), dx=host(blk.dx), dw_r=host(blk.dw_r), dw_gate=host(blk.dw_gate),
                   dw_up=host(blk.dw_up), dw_down=host(blk.dw_down))
        outs.append(out)
    return outs if repeat > 1 else outs[0]


def compare(inp, g, f, b, case=None):
    """Every GPU output against the oracle's.  Without near-tie flips the
    routing tables are bit-exact and every tensor is compared whole.  A token
    whose near tie made the GPU pick another expert set is left out of the
    token-wise comparisons (Y, dX, its rows of Xp, G, U, A, O), and the experts
    it reaches under either routing are left out of the weight-gradient and
    dW_r comparisons; everything else is still compared, and the flip is
    recorded."""
    d = inp["dims"]
    mask = inp["mask"]
    E = d["E"]
    n_set, n_order, flipped = check_routing(f["z"], f["idx"], f["gates"], g["logits"],
                                            g["topk_idx"], g["gates"], d["k"], mask, case=case)
    check_permutation_valid(g["topk_idx"], g["counts"], g["offsets"], g["row_token"], g["row_of"], E)
    if not flipped.any():
        if n_order == 0:
            assert np.array_equal(g["row_of"], f["row_of"])
        assert np.array_equal(g["counts"], f["counts"])
        assert np.array_equal(g["offsets"], f["offsets"])
        assert np.array_equal(g["row_token"], f["row_token"])
    keep = ~flipped
    valid = np.ones(d["T"], dtype=bool) if mask is None else mask.astype(bool)
    gr, rr = row_pairs(g["topk_idx"], g["row_of"], f["idx"], f["row_of"], np.nonzero(keep & valid)[0])
    if len(gr):
        # the gather is a byte copy
        assert np.array_equal(g["xp"][gr], f["xp"][rr])
        for n, ref in (("g", f["G"]), ("u", f["U"]), ("a", f["A"]), ("o", f["O"])):
            if g[n] is not None:
                assert_close(n, g[n][gr], ref[rr], case=case)
    assert_close("y", g["y"][keep], f["Y"][keep], case=case)
    assert_close("dx", g["dx"][keep], b["dx"][keep], case=case)
    cols = ~touched_experts(flipped, g["topk_idx"], f["idx"], E)
    for n in ("dw_gate", "dw_up", "dw_down"):
        assert_close(n, g[n][cols], b[n][cols], case=case)
    assert_close("dw_r", g["dw_r"][:, cols], b["dw_r"][:, cols], case=case)
    if mask is not None:
        m = ~valid
        assert np.all(g["y"][m] == 0) and np.all(g["dx"][m] == 0)
    # experts without rows have exactly zero weight gradients
    empty = np.nonzero(g["counts"] == 0)[0]
    for n in ("dw_gate", "dw_up", "dw_down"):
        assert np.all(g[n][empty] == 0)


def test_tiny_workload_fwd_bwd():
    """T=256, H=128, E=8, top-2, F=256 (the tiny workload), element-wise."""
    inp = workloads.make("tiny")
    f, b = oracle_run(inp)
    compare(inp, gpu_run(inp), f, b, case="tiny")


def test_tiny_workload_fp32_weight_grads():
    """fp32 weight gradients skip the output rounding, so they are held to
    1e-2 rather than 2e-2.  Their inputs are still bf16: A = silu(G) U is
    formed from the bf16-rounded G and U (the stored activations, which the
    backward also reads) and rounded again, up to 3 x 2^-9 relative per
    element of A, and dO carries its own bf16 rounding."""
    inp = workloads.make("tiny")
    f, b = oracle_run(inp)
    g = gpu_run(inp, dw_fp32=True)
    _, _, flipped = check_routing(f["z"], f["idx"], f["gates"], g["logits"], g["topk_idx"], g["gates"],
                                  inp["dims"]["k"])
    assert not flipped.any(), "a near tie flipped an expert set on the fixed tiny seed"
    for n in ("dw_r", "dw_gate", "dw_up", "dw_down"):
        assert_close(n, g[n], b[n], tol=1e-2, case="tiny_fp32_dw")


EDGE = {
    # ragged T over several 128-row tiles per expert, deeper K loops
    "ragged_multi_tile": dict(T=1000, H=512, E=8, k=2, F=384, seed=21),
    "ragged_T": dict(T=300, H=256, E=16, k=4, F=128, seed=22),
    # one token: dW_r is rank one, x dz^T with dz = g1 g2 (dg1 - dg2) (-1, 1),
    # so its relative error is that of dg1 - dg2.  bf16-stored O bounds each
    # dg to ~2^-9 relative; the seed is one whose two gate gradients do not
    # nearly cancel (asserted from the oracle in the test)
    "single_token": dict(T=1, H=128, E=8, k=2, F=128, seed=24),
    "top1": dict(T=200, H=128, E=8, k=1, F=128, seed=24),
    "k_equals_E": dict(T=130, H=128, E=8, k=8, F=256, seed=25),
    "max_E_max_k": dict(T=100, H=128, E=256, k=32, F=128, seed=26),
    # 16-slot kernels with k < 16, and H = 640: a row pass of 1024 columns
    # whose second chunk is masked past H
    "k12_H640": dict(T=150, H=640, E=32, k=12, F=128, seed=28),
    # biased router: several experts receive no rows
    "empty_experts": dict(T=257, H=256, E=32, k=3, F=128, seed=27, zipf_s=1.2, n_cold=6),
    # more than 128 chunks of 256 tokens: the permutation scans the chunk
    # counts per expert before scattering
    "scanned_chunks": dict(T=40000, H=128, E=8, k=2, F=128, seed=29),
    # twice the Qwen widths: 64-step K loops over H, six 256-column tiles of
    # F, eight of H, and ragged two-tile experts
    "wide_H4096_F1536": dict(T=600, H=4096, E=8, k=2, F=1536, seed=30),
}


@pytest.mark.parametrize("case", sorted(EDGE))
def test_edge_shapes(case):
    inp = workloads.block_inputs(**EDGE[case])
    f, b = oracle_run(inp)
    if case == "empty_experts":
        assert (f["counts"] == 0).sum() >= 6
    if case == "single_token":
        dg = b["dg"][0]
        assert abs(dg[0] - dg[1]) >= 0.25 * np.abs(dg).max(), "single-token case must not nearly cancel"
    compare(inp, gpu_run(inp), f, b, case="edge_" + case)


def test_nan_token():
    """One token's hidden row is NaN, so all its logits are NaN.  The top-k
    works on integer order keys: the token still gets k distinct experts in
    [0, E), and the permutation stays the valid stable one of that selection.
    No other token changes: their routing and outputs match the oracle run
    with that row zeroed (rows never mix in the forward)."""
    inp = workloads.block_inputs(T=300, H=256, E=16, k=4, F=128, seed=61)
    d = inp["dims"]
    bad = 7
    x = inp["x"].copy()
    x[bad] = 0x7FC0  # bf16 quiet NaN
    g = gpu_run(dict(inp, x=x))
    idx = g["topk_idx"]
    assert np.all((idx >= 0) & (idx < d["E"]))
    assert len(set(idx[bad].tolist())) == d["k"]
    check_permutation_valid(idx, g["counts"], g["offsets"], g["row_token"], g["row_of"], d["E"])
    x0 = inp["x"].copy()
    x0[bad] = 0
    f, _ = oracle_run(dict(inp, x=x0))
    o = np.arange(d["T"]) != bad
    _, _, flipped = check_routing(f["z"][o], f["idx"][o], f["gates"][o], g["logits"][o], idx[o],
                                  g["gates"][o], d["k"], case="nan_token")
    assert np.all(np.isfinite(g["y"][o]))
    assert_close("y", g["y"][o][~flipped], f["Y"][o][~flipped], case="nan_token")


def test_underflowing_gates():
    """Router logits far apart (W_r scaled up 1000x): many second gates are
    exactly 0 in fp32.  The gate gradient then takes its g = 0 branch
    (dg = 0, so dz = g (dg - sum g dg) stays 0, as the fp64 oracle's tiny g
    makes it) instead of dividing by zero."""
    inp = workloads.block_inputs(T=200, H=128, E=8, k=2, F=128, seed=41)
    inp["w_r"] = workloads.bf16_bits((O.widen_bf16(inp["w_r"]) * 1000.0).astype(np.float32))
    f, b = oracle_run(inp)
    g = gpu_run(inp)
    assert (g["gates"][:, 1] == 0).sum() >= 20, "the case needs gates that underflow"
    for n in ("dx", "dw_r"):
        assert np.all(np.isfinite(g[n]))
    compare(inp, g, f, b, case="underflowing_gates")


@pytest.mark.parametrize("frac", [0.3, 1.0])
def test_masked_tokens(frac):
    inp = workloads.block_inputs(T=333, H=256, E=16, k=2, F=128, seed=31)
    g = np.random.default_rng(5)
    mask = np.ones(333, dtype=np.uint8)
    mask[g.choice(333, int(round(frac * 333)), replace=False)] = 0
    inp["mask"] = mask
    f, b = oracle_run(inp)
    out = gpu_run(inp)
    if frac == 1.0:
        assert f["R"] == 0 and out["offsets"][-1] == 0
        for n in ("y", "dx", "dw_r", "dw_gate", "dw_up", "dw_down"):
            assert np.all(out[n] == 0), n
        assert np.all(out["row_token"] == -1) and np.all(out["topk_idx"] == -1)
        return
    compare(inp, out, f, b, case=f"masked_{frac}")


def test_bitwise_deterministic():
    inp = workloads.block_inputs(T=777, H=256, E=16, k=4, F=256, seed=41)
    a, c = gpu_run(inp, repeat=2)
    for n in a:
        assert np.array_equal(a[n], c[n]), n


def test_recompute_is_bit_identical():
    """MOE_F_RECOMPUTE: the forward keeps no G and U and the backward
    recomputes them with the same kernel, so every output and gradient is
    bit-identical to the run that kept them (which is checked against the
    oracle here too)."""
    inp = workloads.block_inputs(T=777, H=256, E=16, k=4, F=384, seed=43)
    inp["mask"] = (np.arange(777) % 5 != 3).astype(np.uint8)
    f, b = oracle_run(inp)
    a = gpu_run(inp)
    compare(inp, a, f, b, case="recompute")
    r = gpu_run(inp, recompute=True)
    assert r["g"] is None and r["u"] is None
    for n in a:
        if n not in ("g", "u"):
            assert np.array_equal(a[n], r[n]), n


@pytest.mark.parametrize("case", ["tiny_masked", "max_E"])
def test_router_losses(case):
    """Load-balancing loss and z-loss on: the loss values against the oracle's
    definition (fp32 on the GPU), dX and dW_r against the oracle's backward with
    the losses' gradient, and the forward outputs unchanged bit for bit.  The
    coefficients are large enough that the losses' gradient dominates dW_r."""
    import torch
    import paper_2608_00916_amd as moe
    if case == "tiny_masked":
        inp = workloads.block_inputs(T=333, H=256, E=16, k=2, F=128, seed=51)
        inp["mask"] = (np.arange(333) % 7 != 2).astype(np.uint8)
    else:
        inp = workloads.block_inputs(T=200, H=128, E=256, k=8, F=128, seed=52)
    # a small upstream gradient, so that the losses' gradient dominates dz
    inp["dy"] = workloads.bf16_bits(O.widen_bf16(inp["dy"]) * 1e-3)
    coefs = (0.5, 0.05)
    d = inp["dims"]
    mask = inp["mask"]
    print(f"GPU block router losses {case} T={d['T']} E={d['E']} k={d['k']}", flush=True)
    t = {n: dev_bf16(inp[n]) for n in ("x", "w_r", "w_gate", "w_up", "w_down", "dy")}
    tm = None if mask is None else torch.from_numpy(mask.astype(np.uint8)).cuda()
    outs = []
    for c in ((0.0, 0.0), coefs):
        blk = moe.MoEBlock(d["T"], d["H"], d["E"], d["F"], d["k"], mask=tm is not None, aux_loss_coef=c[0],
                           z_loss_coef=c[1])
        blk.forward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], tm)
        blk.backward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], t["dy"])
        torch.cuda.synchronize()
        outs.append(dict(y=host(blk.y), dx=host(blk.dx), dw_r=host(blk.dw_r), dw_gate=host(blk.dw_gate),
                         loss=host(blk.views["router_loss"]), idx=host(blk.views["topk_idx"]),
                         logits=host(blk.views["logits"]), gates=host(blk.views["gates"])))
    base, g = outs
    for n in ("y", "dw_gate"):
        assert np.array_equal(base[n], g[n]), n
    w = {n: O.widen_bf16(inp[n]) for n in ("x", "w_r", "w_gate", "w_up", "w_down", "dy")}
    mb = None if mask is None else mask.astype(bool)
    f = O.moe_forward(w["x"], w["w_r"], w["w_gate"], w["w_up"], w["w_down"], d["k"], mb)
    _, _, flipped = check_routing(f["z"], f["idx"], f["gates"], g["logits"], g["idx"], g["gates"], d["k"], mb,
                                  case="router_losses_" + case)
    # the routing counts enter every token's loss gradient, so a flip anywhere
    # changes dz everywhere: the fixed seeds must route exactly as the oracle
    assert not flipped.any(), "a near tie flipped an expert set on the fixed seed"
    l_aux, l_z = O.router_aux_loss(f["z"], f["idx"], coefs[0], coefs[1], mb)
    assert abs(g["loss"][0] - l_aux) <= 1e-4 * abs(l_aux), (g["loss"], l_aux)
    assert abs(g["loss"][1] - l_z) <= 1e-4 * abs(l_z), (g["loss"], l_z)
    b = O.moe_backward(w["x"], w["w_r"], w["w_gate"], w["w_up"], w["w_down"], f, w["dy"], aux=coefs, mask=mb)
    b0 = O.moe_backward(w["x"], w["w_r"], w["w_gate"], w["w_up"], w["w_down"], f, w["dy"])
    # the losses' gradient is the larger part of dW_r here
    assert np.abs(b["dw_r"] - b0["dw_r"]).max() > 0.5 * np.abs(b0["dw_r"]).max()
    assert_close("dx", g["dx"], b["dx"], case="router_losses_" + case)
    assert_close("dw_r", g["dw_r"], b["dw_r"], case="router_losses_" + case)
