"""GPU parity at the workloads' full sizes, in the launch configuration the
bench times (MoEBlock / MoEExperts / MoELoRA over the C ABI).

Routing, counts, offsets and the permutation are compared for every token.
Values are compared on samples the oracle computes exactly: the block is
separable over tokens except for the weight gradients, so the oracle run on a
token subset S gives Y[S] and dX[S] exactly, and also the full-batch dW of
every expert all of whose tokens are in S and the matching columns of dW_r
(dz vanishes outside an expert's tokens).  Every measured error and the
near-tie counts (set ties, order ties, flipped expert sets) are recorded."""
import numpy as np
import pytest

import workloads
from oracle import moe_oracle as O
from tests.parity import (assert_close, check_permutation_valid, check_routing, dev_bf16, host, record,
                          touched_experts)

pytestmark = pytest.mark.gpu

ADAPTERS = ("a1", "b1_gate", "b1_up", "a2", "b2")


def lora_bits(d, rank, seed, std=0.05):
    E, H, F = d["E"], d["H"], d["F"]
    s = np.random.SeedSequence(seed).spawn(5)
    shapes = dict(a1=(E, H, rank), b1_gate=(E, rank, F), b1_up=(E, rank, F), a2=(E, F, rank), b2=(E, rank, H))
    return {n: workloads.normal_bf16(q, shapes[n], std) for n, q in zip(ADAPTERS, s)}


def run_block(inp, lora=None, coefs=(0.0, 0.0)):
    """lora = (rank, scale, adapter bits) runs moe_lora_fwd / moe_lora_bwd."""
    import torch
    import paper_2608_00916_amd as moe
    d = inp["dims"]
    mask = inp["mask"]
    print(f"GPU block full size T={d['T']} H={d['H']} E={d['E']} k={d['k']} F={d['F']} "
          f"mask={mask is not None} lora={None if lora is None else lora[0]} coefs={coefs}", flush=True)
    t = {n: dev_bf16(inp[n]) for n in ("x", "w_r", "w_gate", "w_up", "w_down", "dy")}
    tm = None if mask is None else torch.from_numpy(mask.astype(np.uint8)).cuda()
    if lora is None:
        blk = moe.MoEBlock(d["T"], d["H"], d["E"], d["F"], d["k"], mask=mask is not None, aux_loss_coef=coefs[0],
                           z_loss_coef=coefs[1])
        blk.forward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], tm)
        blk.backward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], t["dy"])
        grads = {"dw_gate": blk.dw_gate, "dw_up": blk.dw_up, "dw_down": blk.dw_down}
    else:
        rank, scale, bits = lora
        lt = {n: dev_bf16(bits[n]) for n in ADAPTERS}
        la = moe.lora_args(rank, scale, *(lt[n] for n in ADAPTERS))
        blk = moe.MoELoRA(d["T"], d["H"], d["E"], d["F"], d["k"], rank, mask=mask is not None)
        blk.forward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], la, tm)
        blk.backward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], la, t["dy"])
        grads = {"d" + n: getattr(blk, "d" + n) for n in ADAPTERS}
    torch.cuda.synchronize()
    v = blk.views
    out = {n: host(v[n]) for n in ("logits", "topk_idx", "gates", "counts", "offsets", "row_token",
                                  "row_of")}
    out.update(y=host(blk.y), dx=host(blk.dx))
    out["dw_r"] = host(blk.dw_r) if lora is None else None
    out["loss"] = host(v["router_loss"])
    out["grads"] = grads  # stay on the GPU; sampled below
    return out


def check_full(name, check_experts, extra_tokens=256, seed=0, lora=None, coefs=(0.0, 0.0), overrides=None):
    case = name + ("" if lora is None else f"_lora_r{lora[0]}") + ("" if coefs == (0.0, 0.0) else "_router_losses")
    case += "".join(f"_{k}{v}" for k, v in (overrides or {}).items())
    inp = workloads.make(name, **(overrides or {}))
    d = inp["dims"]
    T, E, k = d["T"], d["E"], d["k"]
    mask = None if inp["mask"] is None else inp["mask"].astype(bool)
    g = run_block(inp, lora, coefs)

    # routing and permutation, every token
    x = O.widen_bf16(inp["x"])
    w_r = O.widen_bf16(inp["w_r"])
    z = O.router_logits(x, w_r)
    idx = O.select_topk(z, k, mask)
    gates = O.topk_gates(z, idx)
    n_set, n_order, flipped = check_routing(z, idx, gates, g["logits"], g["topk_idx"], g["gates"], k, mask,
                                            case=case)
    print(f"{case}: near ties set={n_set} order={n_order} flipped={int(flipped.sum())}", flush=True)
    check_permutation_valid(g["topk_idx"], g["counts"], g["offsets"], g["row_token"], g["row_of"], E)
    counts, offsets, row_token, row_of = O.permutation(idx, E)
    exact = not flipped.any()
    if exact:
        assert np.array_equal(g["counts"], counts)
        assert np.array_equal(g["offsets"], offsets)
        assert np.array_equal(g["row_token"], row_token)
        if n_order == 0:
            assert np.array_equal(g["row_of"], row_of)
    record(case, routing_bit_exact=bool(exact and n_order == 0), counts_bit_exact=bool(exact))
    if coefs != (0.0, 0.0):
        # the routing counts enter every token's loss gradient: no flip allowed
        assert exact, "a near tie flipped an expert set on the fixed seed"
        l_aux, l_z = O.router_aux_loss(z, idx, coefs[0], coefs[1], mask)
        la, lz = g["loss"]
        record(case, l_aux_rel=abs(la - l_aux) / abs(l_aux), l_z_rel=abs(lz - l_z) / abs(l_z))
        assert abs(la - l_aux) <= 1e-4 * abs(l_aux) and abs(lz - l_z) <= 1e-4 * abs(l_z), (g["loss"], l_aux, l_z)

    # experts whose full gradients are checked: all their tokens go into the
    # sample; experts a flipped token reaches are not among them
    touched = touched_experts(flipped, g["topk_idx"], idx, E)
    experts = [e for e in check_experts(counts) if not touched[e]]
    rng = np.random.default_rng(seed)
    S = set(rng.choice(np.nonzero(~flipped)[0], extra_tokens, replace=False).tolist())
    S |= {t for t in (0, T - 1) if not flipped[t]}
    for e in experts:
        S |= set(np.nonzero((idx == e).any(axis=1))[0].tolist())
    S = np.array(sorted(S))
    assert not flipped[S].any()
    w = {n: O.widen_bf16(inp[n]) for n in ("w_gate", "w_up", "w_down")}
    dy = O.widen_bf16(inp["dy"][S])
    mS = None if mask is None else mask[S]
    if lora is None:
        f = O.moe_forward(x[S], w_r, w["w_gate"], w["w_up"], w["w_down"], k, mS)
        b = O.moe_backward(x[S], w_r, w["w_gate"], w["w_up"], w["w_down"], f, dy)
    else:
        lo = {n: O.widen_bf16(lora[2][n]) for n in ADAPTERS}
        lo["scale"] = lora[1]
        f = O.lora_forward(x[S], w_r, w["w_gate"], w["w_up"], w["w_down"], lo, k, mS)
        b = O.lora_backward(x[S], w_r, w["w_gate"], w["w_up"], w["w_down"], lo, f, dy)
    dz_aux = None
    if coefs != (0.0, 0.0):  # the losses' dz over the whole batch (global routing fractions)
        dz_aux = O.router_aux_dz(z, idx, coefs[0], coefs[1], mask)
        b["dx"] = b["dx"] + dz_aux[S] @ w_r.T
    assert_close("y[S]", g["y"][S], f["Y"], case=case)
    assert_close("dx[S]", g["dx"][S], b["dx"], case=case)
    if mask is not None:
        assert np.all(g["y"][~mask] == 0) and np.all(g["dx"][~mask] == 0)
    names = ("dw_gate", "dw_up", "dw_down") if lora is None else tuple("d" + n for n in ADAPTERS)
    for e in experts:
        if lora is None:
            ref = b["dw_r"][:, e]
            if dz_aux is not None:  # the losses' dense part reaches column e from every token
                ref = ref + x.T @ dz_aux[:, e]
            assert_close("dw_r[:, e]", g["dw_r"][:, e], ref, case=case)
        for n in names:
            got = host(g["grads"][n][e])
            if counts[e] == 0:
                assert np.all(got == 0), f"{n}[{e}] of an empty expert"
            else:
                assert_close(f"{n}[e]", got, b[n][e], case=case)
    record(case, experts_checked=len(experts), sample_tokens=int(len(S)))
    return counts


def pick_qwen(c):
    return [int(np.argmin(c)), int(np.argmax(c)), 0]


def test_qwen3_30b_a3b_fullsize():
    """T=8192, H=2048, E=128, top-8, F=768: the bench workload."""
    check_full("qwen3_30b_a3b", pick_qwen)


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


def test_qwen3_30b_a3b_lora_fullsize():
    """Rank-16 expert LoRA at the bench shape (moe_lora_fwd / moe_lora_bwd):
    Y and dX on sampled tokens, the five adapter gradients of whole experts."""
    inp_dims = workloads.CONFIGS["qwen3_30b_a3b"]
    bits = lora_bits(inp_dims, 16, seed=316)
    check_full("qwen3_30b_a3b", pick_qwen, lora=(16, 2.0, bits))


def test_qwen3_30b_a3b_router_losses_fullsize():
    """Load-balancing loss and z-loss on at the bench shape: the loss values,
    dX on sampled tokens, and the dW_r columns of whole experts (their gate
    part from the sample, the losses' dense part from the whole batch)."""
    check_full("qwen3_30b_a3b", pick_qwen, coefs=(0.01, 0.001))


def test_rows_beyond_2gib_fullsize():
    """The Qwen shape at T=131072: 2^20 routed rows, so Xp, O, dO and dXp
    hold 4 GiB each and every row-indexed byte offset passes 2^31 (they are
    formed in 64 bits).  Routing for every token; Y, dX, dW_r and the weight
    gradients of the least-routed expert on the oracle's token sample."""
    check_full("qwen3_30b_a3b", lambda c: [int(np.argmin(c))], extra_tokens=128,
               overrides=dict(T=131072, seed=5))


def test_bitwise_deterministic_fullsize():
    """Two fwd+bwd calls on the Zipf batch (T=32768: hot experts, empty
    experts, the device-built weight-gradient schedule, 64 dW_r splits) give
    the same bits in every output, routing table and gradient."""
    import torch
    import paper_2608_00916_amd as moe
    inp = workloads.make("zipf")
    d = inp["dims"]
    print(f"GPU determinism T={d['T']} H={d['H']} E={d['E']} k={d['k']} F={d['F']}", flush=True)
    t = {n: dev_bf16(inp[n]) for n in ("x", "w_r", "w_gate", "w_up", "w_down", "dy")}
    blk = moe.MoEBlock(d["T"], d["H"], d["E"], d["F"], d["k"])
    names = ("y", "dx", "dw_r", "dw_gate", "dw_up", "dw_down")
    views = ("logits", "topk_idx", "gates", "counts", "offsets", "row_token", "row_of", "xp", "g", "u", "a", "o")
    runs = []
    for _ in range(2):
        blk.forward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"])
        blk.backward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], t["dy"])
        torch.cuda.synchronize()
        R = int(blk.views["offsets"][-1])
        snap = {n: getattr(blk, n).clone() for n in names}
        for n in views:
            v = blk.views[n]
            snap[n] = (v[:R] if n in ("xp", "g", "u", "a", "o", "row_token") else v).clone()
        runs.append(snap)
    for n in runs[0]:  # bytes, so that floats compare bit for bit
        assert torch.equal(runs[0][n].contiguous().view(torch.uint8), runs[1][n].contiguous().view(torch.uint8)), n
    record("zipf_two_runs", bitwise_equal=True)


def test_ep_share_fullsize():
    """One expert-parallel rank: 16 local experts and the 8359 rows a top-8
    router sends them from a T=8192 batch; every output and gradient compared
    element-wise."""
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
    c = "ep_share"
    assert_close("o", host(ex.o), f["O"], case=c)
    for n, ref in (("g", f["G"]), ("u", f["U"]), ("a", f["A"])):
        assert_close(n, host(ex.views[n]), ref, case=c)
    assert_close("dxp", host(ex.dxp), b["dxp"], case=c)
    assert_close("dw_gate", host(ex.dw_gate), b["dw_gate"], case=c)
    assert_close("dw_up", host(ex.dw_up), b["dw_up"], case=c)
    assert_close("dw_down", host(ex.dw_down), b["dw_down"], case=c)
