"""GPU parity at the workloads' full sizes, in the launch configuration the
bench times (MoEBlock / MoEExperts over the C ABI).

Routing, counts, offsets and the permutation are compared for every token.
Values are compared on samples the oracle computes exactly: the block is
separable over tokens except for the weight gradients, so the oracle run on a
token subset S gives Y[S] and dX[S] exactly, and also the full-batch dW of
every expert all of whose tokens are in S and the matching columns of dW_r
(dz vanishes outside an expert's tokens)."""
import numpy as np
import pytest

import workloads
from oracle import moe_oracle as O
from tests.parity import (assert_close, assert_router_grad, check_permutation_valid,
                          check_routing, dev_bf16, host, router_grad_bound)

pytestmark = pytest.mark.gpu


def run_block(inp):
    import torch
    import paper_2608_00916_amd as moe
    d = inp["dims"]
    mask = inp["mask"]
    print(f"GPU block full size T={d['T']} H={d['H']} E={d['E']} k={d['k']} F={d['F']} "
          f"mask={mask is not None}", flush=True)
    blk = moe.MoEBlock(d["T"], d["H"], d["E"], d["F"], d["k"], mask=mask is not None)
    t = {n: dev_bf16(inp[n]) for n in ("x", "w_r", "w_gate", "w_up", "w_down", "dy")}
    tm = None if mask is None else torch.from_numpy(mask.astype(np.uint8)).cuda()
    blk.forward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], tm)
    blk.backward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], t["dy"])
    torch.cuda.synchronize()
    v = blk.views
    out = {n: host(v[n]) for n in ("logits", "topk_idx", "gates", "counts", "offsets", "row_token",
                                  "row_of")}
    out.update(y=host(blk.y), dx=host(blk.dx), dw_r=host(blk.dw_r))
    out["dw"] = (blk.dw_gate, blk.dw_up, blk.dw_down)  # stay on the GPU; sampled below
    return out


def check_full(name, check_experts, extra_tokens=256, seed=0):
    inp = workloads.make(name)
    d = inp["dims"]
    T, E, k = d["T"], d["E"], d["k"]
    mask = None if inp["mask"] is None else inp["mask"].astype(bool)
    g = run_block(inp)

    # routing and permutation, every token
    x = O.widen_bf16(inp["x"])
    w_r = O.widen_bf16(inp["w_r"])
    z = O.router_logits(x, w_r)
    idx = O.select_topk(z, k, mask)
    gates = O.topk_gates(z, idx)
    n_set, n_order, flipped = check_routing(z, idx, gates, g["logits"], g["topk_idx"], g["gates"], k,
                                            mask)
    print(f"{name}: near ties set={n_set} order={n_order} flipped={int(flipped.sum())}", flush=True)
    check_permutation_valid(g["topk_idx"], g["counts"], g["offsets"], g["row_token"], g["row_of"], E)
    counts, offsets, row_token, row_of = O.permutation(idx, E)
    if not flipped.any():
        assert np.array_equal(g["counts"], counts)
        assert np.array_equal(g["offsets"], offsets)
        assert np.array_equal(g["row_token"], row_token)
    if n_order == 0 and not flipped.any():
        assert np.array_equal(g["row_of"], row_of)

    # experts whose full dW is checked: all their tokens go into the sample
    experts = check_experts(counts)
    rng = np.random.default_rng(seed)
    S = set(rng.choice(T, extra_tokens, replace=False).tolist()) | {0, T - 1}
    for e in experts:
        S |= set(np.nonzero((idx == e).any(axis=1))[0].tolist())
    S = np.array(sorted(S))
    assert not flipped[S].any(), "a sampled token sits on a near tie; pick another sample"
    w = {n: O.widen_bf16(inp[n]) for n in ("w_gate", "w_up", "w_down")}
    dy = O.widen_bf16(inp["dy"][S])
    mS = None if mask is None else mask[S]
    f = O.moe_forward(x[S], w_r, w["w_gate"], w["w_up"], w["w_down"], k, mS)
    b = O.moe_backward(x[S], w_r, w["w_gate"], w["w_up"], w["w_down"], f, dy)
    assert_close("y[S]", g["y"][S], f["Y"])
    assert_close("dx[S]", g["dx"][S], b["dx"])
    if mask is not None:
        assert np.all(g["y"][~mask] == 0) and np.all(g["dx"][~mask] == 0)
    bound = router_grad_bound(f, dy, x[S])
    for e in experts:
        assert_router_grad(g["dw_r"][:, e], b["dw_r"][:, e], bound[:, e])
        for gt, n in zip(g["dw"], ("dw_gate", "dw_up", "dw_down")):
            got = host(gt[e])
            if counts[e] == 0:
                assert np.all(got == 0), f"{n}[{e}] of an empty expert"
            else:
                assert_close(f"{n}[{e}]", got, b[n][e])
    return counts


def test_qwen3_30b_a3b_fullsize():
    """T=8192, H=2048, E=128, top-8, F=768: the bench workload."""
    def pick(c):
        return [int(np.argmin(c)), int(np.argmax(c)), 0]
    check_full("qwen3_30b_a3b", pick)


def test_zipf_fullsize():
    """T=32768 with Zipf expert popularity: empty experts write zero weight
    gradients; a mid-popularity and a cold expert are checked in full."""
    def pick(c):
        nz = np.nonzero(c)[0]
        mid = int(nz[np.argsort(c[nz])[len(nz) // 2]])
        cold = int(nz[np.argmin(c[nz])])
        empty = [int(e) for e in np.nonzero(c == 0)[0]]
        assert len(empty) == 4 and c.max() > 8 * c.mean()
        return empty + [cold, mid]
    check_full("zipf", pick)


def test_long_passage_fullsize():
    """T=65536 = 16 x 4096 with padding masked out of routing."""
    def pick(c):
        return [int(np.argmin(c))]
    check_full("long_passage", pick, extra_tokens=128)


def test_ep_share_fullsize():
    """One expert-parallel rank: 16 local experts, 8192 dispatched rows;
    every output and gradient compared element-wise."""
    import torch
    import paper_2608_00916_amd as moe
    inp = workloads.make("ep_share")
    d = inp["dims"]
    print(f"GPU experts rows={d['R']} E={d['E']} H={d['H']} F={d['F']}", flush=True)
    ex = moe.MoEExperts(d["R"], d["H"], d["E"], d["F"])
    t = {n: dev_bf16(inp[n]) for n in ("xp", "w_gate", "w_up", "w_down", "d_o")}
    counts = torch.from_numpy(inp["counts"]).cuda()
    ex.forward(t["xp"], counts, t["w_gate"], t["w_up"], t["w_down"])
    ex.backward(t["xp"], t["w_gate"], t["w_up"], t["w_down"], t["d_o"])
    torch.cuda.synchronize()
    w = {n: O.widen_bf16(inp[n]) for n in ("xp", "w_gate", "w_up", "w_down", "d_o")}
    f = O.experts_share_forward(w["xp"], inp["counts"], w["w_gate"], w["w_up"], w["w_down"])
    b = O.experts_share_backward(w["xp"], inp["counts"], w["w_gate"], w["w_up"], w["w_down"], f,
                                 w["d_o"])
    assert np.array_equal(host(ex.views["offsets"]), f["offsets"])
    assert_close("o", host(ex.o), f["O"])
    for n, ref in (("g", f["G"]), ("u", f["U"]), ("a", f["A"])):
        assert_close(n, host(ex.views[n]), ref)
    assert_close("dxp", host(ex.dxp), b["dxp"])
    assert_close("dw_gate", host(ex.dw_gate), b["dw_gate"])
    assert_close("dw_up", host(ex.dw_up), b["dw_up"])
    assert_close("dw_down", host(ex.dw_down), b["dw_down"])
