"""Pins of the fp64 oracle against what mathematics fixes (no GPU).

Each test fails on a plausible mistake in one oracle step: wrong tie-break or
slot order (brute-force stable sort, hand-worked fixtures), un-normalised gates
(sum to one, full softmax at k = E, closed form), a broken permutation
(hand-worked fixture, brute-force sort of (expert, token) pairs, bijection), a
transposed or missing operand in the experts (dense SwiGLU reduction at E = k = 1,
identical experts), and any error in the hand-derived backward (central finite
differences in fp64 and an independent PyTorch autograd re-implementation)."""
import json
import math
import os

import numpy as np
import pytest
import scipy.special

import workloads
from oracle import moe_oracle as O
from tests.parity import touched_experts

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def rand_block(T, H, E, k, F, seed, n_masked=0, wstd=0.3):
    g = np.random.default_rng(seed)
    x = g.standard_normal((T, H))
    w_r = g.standard_normal((H, E)) * wstd
    w_g = g.standard_normal((E, H, F)) * wstd
    w_u = g.standard_normal((E, H, F)) * wstd
    w_d = g.standard_normal((E, F, H)) * wstd
    dy = g.standard_normal((T, H))
    mask = None
    if n_masked:
        mask = np.ones(T, dtype=bool)
        mask[g.choice(T, n_masked, replace=False)] = False
    return x, w_r, w_g, w_u, w_d, dy, mask


# ------------------------------------------------------------ selection + gates
def test_gates_golden():
    fx = json.load(open(os.path.join(GOLD, "gates_small.json")))
    for c in fx["cases"]:
        z = np.array([c["z"]])
        idx = O.select_topk(z, c["k"])
        g = O.topk_gates(z, idx)
        assert idx[0].tolist() == c["idx"]
        np.testing.assert_allclose(g[0], c["gates"], rtol=1e-15, atol=0)
    # the closed form of case a, independent of the stored numbers
    e = math.e
    np.testing.assert_allclose(fx["cases"][0]["gates"], [3 / (3 + e), e / (3 + e)], rtol=1e-15)


@pytest.mark.parametrize("k", [1, 2, 3, 8])
def test_topk_matches_brute_force_stable_sort(k):
    g = np.random.default_rng(11)
    T, E = 500, 16
    # quantised logits so that exact ties are frequent
    z = np.round(g.standard_normal((T, E)) * 4) / 4
    idx = O.select_topk(z, k)
    ref = np.argsort(-z.astype(np.float32), axis=1, kind="stable")[:, :k]
    assert np.array_equal(idx, ref)
    # k distinct experts per token
    assert all(len(set(r)) == k for r in idx.tolist())


def test_selection_decided_in_fp32():
    # two logits distinct in fp64 but equal once rounded to fp32: lower index wins
    z = np.array([[1.0 + 1e-12, 1.0, 0.0]])
    assert O.select_topk(z[:, ::-1].copy(), 1)[0, 0] == 1  # [0, 1, 1+1e-12] -> tie at fp32 -> index 1
    assert O.select_topk(z, 1)[0, 0] == 0


def test_gates_sum_to_one_and_equal_renormalised_softmax():
    g = np.random.default_rng(3)
    z = g.standard_normal((300, 12)) * 2
    for k in (1, 3, 5):
        idx = O.select_topk(z, k)
        gates = O.topk_gates(z, idx)
        np.testing.assert_allclose(gates.sum(1), 1.0, atol=1e-14)
        p = scipy.special.softmax(z, axis=1)
        ps = np.take_along_axis(p, idx, axis=1)
        np.testing.assert_allclose(gates, ps / ps.sum(1, keepdims=True), rtol=1e-12)
        # slots in descending logit order
        zs = np.take_along_axis(z, idx, axis=1)
        assert np.all(np.diff(zs, axis=1) <= 0)


def test_k_equals_E_gives_full_softmax():
    g = np.random.default_rng(4)
    z = g.standard_normal((64, 7))
    idx = O.select_topk(z, 7)
    gates = O.topk_gates(z, idx)
    full = np.take_along_axis(scipy.special.softmax(z, axis=1), idx, axis=1)
    np.testing.assert_allclose(gates, full, rtol=1e-13)


def test_masked_tokens_not_routed():
    g = np.random.default_rng(5)
    z = g.standard_normal((10, 4))
    mask = np.array([1, 0, 1, 1, 0, 1, 1, 1, 1, 0], dtype=bool)
    idx = O.select_topk(z, 2, mask)
    gates = O.topk_gates(z, idx)
    assert np.all(idx[~mask] == -1) and np.all(gates[~mask] == 0)
    assert np.all(idx[mask] >= 0)


# ------------------------------------------------------------ permutation
def test_permutation_golden():
    fx = json.load(open(os.path.join(GOLD, "permutation_small.json")))
    counts, offsets, row_token, row_of = O.permutation(np.array(fx["idx"]), fx["E"])
    assert counts.tolist() == fx["counts"]
    assert offsets.tolist() == fx["offsets"]
    assert row_token.tolist() == fx["row_token"]
    assert row_of.tolist() == fx["row_of"]


def test_permutation_brute_force_and_invariants():
    g = np.random.default_rng(6)
    T, E, k = 333, 9, 3
    z = g.standard_normal((T, E))
    mask = g.random(T) > 0.2
    idx = O.select_topk(z, k, mask)
    counts, offsets, row_token, row_of = O.permutation(idx, E)
    Tv = int(mask.sum())
    assert counts.sum() == Tv * k and offsets[E] == Tv * k
    assert np.all(np.diff(offsets) >= 0) and offsets[0] == 0
    # brute force: sort all (expert, token, slot) triples lexicographically
    pairs = sorted((int(idx[t, j]), t, j) for t in range(T) for j in range(k) if mask[t])
    assert [t for _, t, _ in pairs] == row_token[:Tv * k].tolist()
    for r, (e, t, j) in enumerate(pairs):
        assert row_of[t, j] == r
        assert offsets[e] <= r < offsets[e + 1]
    assert np.all(row_token[Tv * k:] == -1)
    assert np.all(row_of[~mask] == -1)


# ------------------------------------------------------------ forward reductions
def dense_swiglu_torch(x, w_g, w_u, w_d):
    import torch
    xt = torch.from_numpy(x)
    a = torch.nn.functional.silu(xt @ torch.from_numpy(w_g)) * (xt @ torch.from_numpy(w_u))
    return (a @ torch.from_numpy(w_d)).numpy()


def test_single_expert_top1_is_dense_swiglu():
    x, w_r, w_g, w_u, w_d, dy, _ = rand_block(40, 12, 1, 1, 10, seed=7)
    f = O.moe_forward(x, w_r, w_g, w_u, w_d, 1)
    np.testing.assert_allclose(f["gates"], 1.0)
    np.testing.assert_allclose(f["Y"], dense_swiglu_torch(x, w_g[0], w_u[0], w_d[0]), rtol=1e-12, atol=1e-12)
    b = O.moe_backward(x, w_r, w_g, w_u, w_d, f, dy)
    assert np.abs(b["dw_r"]).max() < 1e-12


def test_identical_experts_reduce_to_dense_ffn():
    x, w_r, w_g, w_u, w_d, dy, mask = rand_block(50, 10, 5, 3, 8, seed=8, n_masked=5)
    w_g[:] = w_g[0]
    w_u[:] = w_u[0]
    w_d[:] = w_d[0]
    f = O.moe_forward(x, w_r, w_g, w_u, w_d, 3, mask)
    ref = dense_swiglu_torch(x, w_g[0], w_u[0], w_d[0])
    ref[~mask] = 0
    np.testing.assert_allclose(f["Y"], ref, rtol=1e-12, atol=1e-12)
    b = O.moe_backward(x, w_r, w_g, w_u, w_d, f, dy)
    assert np.abs(b["dw_r"]).max() < 1e-10 * np.abs(b["dw_gate"]).max()
    assert np.all(b["dx"][~mask] == 0)


def test_linearity_in_w_down_and_dy():
    x, w_r, w_g, w_u, w_d, dy, mask = rand_block(30, 8, 4, 2, 6, seed=9, n_masked=3)
    f1 = O.moe_forward(x, w_r, w_g, w_u, w_d, 2, mask)
    f2 = O.moe_forward(x, w_r, w_g, w_u, 2.5 * w_d, 2, mask)
    np.testing.assert_allclose(f2["Y"], 2.5 * f1["Y"], rtol=1e-12, atol=1e-13)
    b1 = O.moe_backward(x, w_r, w_g, w_u, w_d, f1, dy)
    b2 = O.moe_backward(x, w_r, w_g, w_u, w_d, f1, -3.0 * dy)
    for n in ("dx", "dw_r", "dw_gate", "dw_up", "dw_down"):
        np.testing.assert_allclose(b2[n], -3.0 * b1[n], rtol=1e-12, atol=1e-13)


def test_token_forward_matches_block():
    x, w_r, w_g, w_u, w_d, _, _ = rand_block(20, 8, 5, 2, 6, seed=10)
    f = O.moe_forward(x, w_r, w_g, w_u, w_d, 2)
    tf = O.token_forward(x[[3, 17]], w_r, w_g, w_u, w_d, 2)
    np.testing.assert_allclose(tf["Y"], f["Y"][[3, 17]], rtol=1e-12)
    assert np.array_equal(tf["idx"], f["idx"][[3, 17]])


def test_experts_share_matches_block_internals():
    x, w_r, w_g, w_u, w_d, dy, _ = rand_block(40, 8, 6, 2, 6, seed=12)
    f = O.moe_forward(x, w_r, w_g, w_u, w_d, 2)
    b = O.moe_backward(x, w_r, w_g, w_u, w_d, f, dy)
    s = O.experts_share_forward(f["xp"], f["counts"], w_g, w_u, w_d)
    np.testing.assert_array_equal(s["O"], f["O"])
    sb = O.experts_share_backward(f["xp"], f["counts"], w_g, w_u, w_d, s, b["dO"])
    for n in ("dxp", "dw_gate", "dw_up", "dw_down"):
        np.testing.assert_array_equal(sb[n], b[n])


# ------------------------------------------------------------ backward
FD_SHAPE = dict(T=24, H=7, E=6, k=2, F=5)


def _fd_setup():
    # seed chosen so that no selection is within 1e-3 of a tie, far above the
    # logit perturbation of the finite differences
    for seed in range(100, 200):
        x, w_r, w_g, w_u, w_d, dy, mask = rand_block(**FD_SHAPE, seed=seed, n_masked=4)
        z = O.router_logits(x, w_r)
        st, ot = O.near_ties(z, FD_SHAPE["k"], gap=1e-3)
        if not st.any() and not ot.any():
            return x, w_r, w_g, w_u, w_d, dy, mask
    raise RuntimeError("no tie-free seed")


def test_gradients_match_central_finite_differences():
    x, w_r, w_g, w_u, w_d, dy, mask = _fd_setup()
    k = FD_SHAPE["k"]
    params = dict(x=x, w_r=w_r, w_gate=w_g, w_up=w_u, w_down=w_d)

    def loss(p):
        f = O.moe_forward(p["x"], p["w_r"], p["w_gate"], p["w_up"], p["w_down"], k, mask)
        return float(np.sum(dy * f["Y"]))

    f = O.moe_forward(x, w_r, w_g, w_u, w_d, k, mask)
    b = O.moe_backward(x, w_r, w_g, w_u, w_d, f, dy)
    grads = dict(x=b["dx"], w_r=b["dw_r"], w_gate=b["dw_gate"], w_up=b["dw_up"], w_down=b["dw_down"])
    g = np.random.default_rng(0)
    eps = 1e-6
    for name in params:
        for _ in range(3):
            v = g.standard_normal(params[name].shape)
            pp = dict(params)
            pm = dict(params)
            pp[name] = params[name] + eps * v
            pm[name] = params[name] - eps * v
            fd = (loss(pp) - loss(pm)) / (2 * eps)
            an = float(np.sum(grads[name] * v))
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)


def test_gradients_match_torch_autograd():
    import torch
    x, w_r, w_g, w_u, w_d, dy, mask = rand_block(60, 9, 7, 3, 6, seed=13, n_masked=6)
    k = 3
    f = O.moe_forward(x, w_r, w_g, w_u, w_d, k, mask)
    b = O.moe_backward(x, w_r, w_g, w_u, w_d, f, dy)

    t = {n: torch.tensor(a, requires_grad=True) for n, a in
         dict(x=x, w_r=w_r, w_g=w_g, w_u=w_u, w_d=w_d).items()}
    valid = torch.from_numpy(mask)
    idx = torch.from_numpy(np.where(f["idx"] < 0, 0, f["idx"]))
    z = t["x"] @ t["w_r"]
    gates = torch.softmax(torch.gather(z, 1, idx), dim=1) * valid[:, None]
    y = torch.zeros_like(t["x"])
    for j in range(k):
        for e in range(w_r.shape[1]):
            sel = (idx[:, j] == e) & valid
            if sel.any():
                xs = t["x"][sel]
                a = torch.nn.functional.silu(xs @ t["w_g"][e]) * (xs @ t["w_u"][e])
                y = y.index_add(0, sel.nonzero()[:, 0], gates[sel, j:j + 1] * (a @ t["w_d"][e]))
    np.testing.assert_allclose(y.detach().numpy(), f["Y"], rtol=1e-12, atol=1e-12)
    (y * torch.from_numpy(dy)).sum().backward()
    for n, on in (("x", "dx"), ("w_r", "dw_r"), ("w_g", "dw_gate"), ("w_u", "dw_up"), ("w_d", "dw_down")):
        np.testing.assert_allclose(b[on], t[n].grad.numpy(), rtol=1e-10, atol=1e-11, err_msg=n)


# ------------------------------------------------------------ router losses
def test_aux_loss_closed_forms():
    """Equal logits: every P_e = 1/E, so L_aux = aux_coef * sum_e f_e = aux_coef
    whatever the routing, and lse = ln E, so L_z = z_coef (ln E)^2.  Balanced
    routing (f_e = 1/E): L_aux = aux_coef * sum_e P_e = aux_coef for any
    logits."""
    T, E, k = 24, 6, 2
    z = np.zeros((T, E))
    idx = O.select_topk(z, k)
    l_aux, l_z = O.router_aux_loss(z, idx, 0.01, 0.001)
    assert math.isclose(l_aux, 0.01, rel_tol=1e-14)
    assert math.isclose(l_z, 0.001 * math.log(E) ** 2, rel_tol=1e-14)
    # balanced: token t prefers experts 2t, 2t+1 (mod E): 24 tokens x 2 slots = 8 per expert
    g = np.random.default_rng(3)
    z = g.standard_normal((T, E)) * 0.1
    for t in range(T):
        z[t, (2 * t) % E] += 10.0
        z[t, (2 * t + 1) % E] += 9.0
    idx = O.select_topk(z, k)
    counts = np.bincount(idx.ravel(), minlength=E)
    assert np.all(counts == T * k // E)
    l_aux, _ = O.router_aux_loss(z, idx, 0.3, 0.0)
    assert math.isclose(l_aux, 0.3, rel_tol=1e-13)
    # masked tokens count nowhere: masking half the tokens equals dropping them
    mask = np.arange(T) % 2 == 0
    a = O.router_aux_loss(z, idx, 0.3, 0.2, mask)
    b = O.router_aux_loss(z[mask], idx[mask], 0.3, 0.2)
    assert np.allclose(a, b, rtol=1e-14)


def test_aux_dz_matches_finite_differences():
    """The analytic gradient of L_aux + L_z against central differences of
    the loss definition in z, routing held fixed (f is piecewise constant)."""
    g = np.random.default_rng(21)
    T, E, k = 40, 8, 3
    z = g.standard_normal((T, E))
    mask = g.random(T) > 0.2
    idx = O.select_topk(z, k, mask)
    dz = O.router_aux_dz(z, idx, 0.05, 0.02, mask)
    assert np.all(dz[~mask] == 0)

    def total(zz):
        a, b = O.router_aux_loss(zz, idx, 0.05, 0.02, mask)
        return a + b
    eps = 1e-6
    for _ in range(4):
        v = g.standard_normal(z.shape)
        fd = (total(z + eps * v) - total(z - eps * v)) / (2 * eps)
        an = float(np.sum(dz * v))
        assert abs(fd - an) <= 1e-8 * max(1.0, abs(an)), (fd, an)


def test_aux_dz_matches_torch_autograd():
    import torch
    g = np.random.default_rng(22)
    T, E, k = 50, 16, 4
    z = g.standard_normal((T, E)) * 2.0
    mask = g.random(T) > 0.3
    idx = O.select_topk(z, k, mask)
    Tv = int(mask.sum())
    f = torch.zeros(E, dtype=torch.float64)
    for e in range(E):
        f[e] = float(np.count_nonzero(idx[mask] == e)) / (Tv * k)
    zt = torch.tensor(z, requires_grad=True)
    m = torch.from_numpy(mask)
    p = torch.softmax(zt, dim=1)[m]
    lse = torch.logsumexp(zt, dim=1)[m]
    loss = 0.07 * E * torch.sum(f * p.mean(dim=0)) + 0.03 * torch.mean(lse ** 2)
    loss.backward()
    np.testing.assert_allclose(O.router_aux_dz(z, idx, 0.07, 0.03, mask), zt.grad.numpy(), rtol=1e-10,
                               atol=1e-13)
    a, b = O.router_aux_loss(z, idx, 0.07, 0.03, mask)
    assert math.isclose(a + b, float(loss.detach()), rel_tol=1e-12)


def test_block_gradients_with_aux_match_finite_differences():
    """The block objective <Y, dY> + L_aux + L_z: its dW_r and dX from
    moe_backward(aux=...) against central differences (routing tie-free)."""
    x, w_r, w_g, w_u, w_d, dy, mask = _fd_setup()
    k = FD_SHAPE["k"]
    aux = (0.05, 0.01)
    f0 = O.moe_forward(x, w_r, w_g, w_u, w_d, k, mask)

    def loss(xx, wr):
        f = O.moe_forward(xx, wr, w_g, w_u, w_d, k, mask)
        assert np.array_equal(f["idx"], f0["idx"])
        a, b = O.router_aux_loss(f["z"], f["idx"], aux[0], aux[1], mask)
        return float(np.sum(dy * f["Y"])) + a + b

    b = O.moe_backward(x, w_r, w_g, w_u, w_d, f0, dy, aux=aux, mask=mask)
    g = np.random.default_rng(4)
    eps = 1e-6
    for _ in range(3):
        v = g.standard_normal(w_r.shape)
        fd = (loss(x, w_r + eps * v) - loss(x, w_r - eps * v)) / (2 * eps)
        an = float(np.sum(b["dw_r"] * v))
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), ("w_r", fd, an)
        v = g.standard_normal(x.shape)
        fd = (loss(x + eps * v, w_r) - loss(x - eps * v, w_r)) / (2 * eps)
        an = float(np.sum(b["dx"] * v))
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), ("x", fd, an)


# ------------------------------------------------------------ expert LoRA
def rand_lora(E, H, F, r, seed, scale=2.0, std=0.3):
    g = np.random.default_rng(seed)
    return dict(scale=scale, a1=g.standard_normal((E, H, r)) * std, b1_gate=g.standard_normal((E, r, F)) * std,
                b1_up=g.standard_normal((E, r, F)) * std, a2=g.standard_normal((E, F, r)) * std,
                b2=g.standard_normal((E, r, H)) * std)


def test_lora_equals_merged_weights():
    """LoRA is a low-rank update of the weights: the adapted forward equals
    the plain forward with W + scale a b merged into every expert, and with
    b1 = b2 = 0 (the usual initialisation) it equals the base forward."""
    x, w_r, w_g, w_u, w_d, dy, mask = rand_block(70, 10, 6, 2, 7, seed=31, n_masked=5)
    lo = rand_lora(6, 10, 7, 3, seed=32)
    f = O.lora_forward(x, w_r, w_g, w_u, w_d, lo, 2, mask)
    s = lo["scale"]
    merged = O.moe_forward(x, w_r, w_g + s * lo["a1"] @ lo["b1_gate"], w_u + s * lo["a1"] @ lo["b1_up"],
                           w_d + s * lo["a2"] @ lo["b2"], 2, mask)
    for n in ("G", "U", "A", "O", "Y"):
        np.testing.assert_allclose(f[n], merged[n], rtol=1e-12, atol=1e-12, err_msg=n)
    zero = dict(lo, b1_gate=0 * lo["b1_gate"], b1_up=0 * lo["b1_up"], b2=0 * lo["b2"])
    f0 = O.lora_forward(x, w_r, w_g, w_u, w_d, zero, 2, mask)
    base = O.moe_forward(x, w_r, w_g, w_u, w_d, 2, mask)
    np.testing.assert_array_equal(f0["Y"], base["Y"])


def test_lora_gradients_match_finite_differences():
    """Adapter gradients and dX of <Y, dY> against central differences
    (routing tie-free), and dX equal to the merged-weight block's dX."""
    x, w_r, w_g, w_u, w_d, dy, mask = _fd_setup()
    k = FD_SHAPE["k"]
    E, H, F = w_r.shape[1], x.shape[1], w_g.shape[2]
    lo = rand_lora(E, H, F, 2, seed=33, scale=0.7)
    f = O.lora_forward(x, w_r, w_g, w_u, w_d, lo, k, mask)
    b = O.lora_backward(x, w_r, w_g, w_u, w_d, lo, f, dy)

    def loss(xx, ll):
        ff = O.lora_forward(xx, w_r, w_g, w_u, w_d, ll, k, mask)
        assert np.array_equal(ff["idx"], f["idx"])
        return float(np.sum(dy * ff["Y"]))
    g = np.random.default_rng(5)
    eps = 1e-6
    for n in ("a1", "b1_gate", "b1_up", "a2", "b2"):
        for _ in range(2):
            v = g.standard_normal(lo[n].shape)
            fd = (loss(x, dict(lo, **{n: lo[n] + eps * v})) - loss(x, dict(lo, **{n: lo[n] - eps * v}))) / (2 * eps)
            an = float(np.sum(b["d" + n] * v))
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (n, fd, an)
    v = g.standard_normal(x.shape)
    fd = (loss(x + eps * v, lo) - loss(x - eps * v, lo)) / (2 * eps)
    assert abs(fd - float(np.sum(b["dx"] * v))) <= 1e-6 * max(1.0, abs(fd))
    s = lo["scale"]
    wm = (w_g + s * lo["a1"] @ lo["b1_gate"], w_u + s * lo["a1"] @ lo["b1_up"], w_d + s * lo["a2"] @ lo["b2"])
    fm = O.moe_forward(x, w_r, *wm, k, mask)
    bm = O.moe_backward(x, w_r, *wm, fm, dy)
    np.testing.assert_allclose(b["dx"], bm["dx"], rtol=1e-10, atol=1e-12)


def test_lora_gradients_match_torch_autograd():
    import torch
    x, w_r, w_g, w_u, w_d, dy, mask = rand_block(50, 8, 5, 2, 6, seed=34, n_masked=4)
    lo = rand_lora(5, 8, 6, 3, seed=35, scale=1.5)
    k = 2
    f = O.lora_forward(x, w_r, w_g, w_u, w_d, lo, k, mask)
    b = O.lora_backward(x, w_r, w_g, w_u, w_d, lo, f, dy)
    t = {n: torch.tensor(lo[n], requires_grad=True) for n in ("a1", "b1_gate", "b1_up", "a2", "b2")}
    xt = torch.tensor(x, requires_grad=True)
    valid = torch.from_numpy(mask)
    idx = torch.from_numpy(np.where(f["idx"] < 0, 0, f["idx"]))
    z = xt @ torch.from_numpy(w_r)
    gates = torch.softmax(torch.gather(z, 1, idx), dim=1) * valid[:, None]
    s = lo["scale"]
    y = torch.zeros_like(xt)
    for j in range(k):
        for e in range(5):
            sel = (idx[:, j] == e) & valid
            if sel.any():
                xs = xt[sel]
                wg = torch.from_numpy(w_g[e]) + s * t["a1"][e] @ t["b1_gate"][e]
                wu = torch.from_numpy(w_u[e]) + s * t["a1"][e] @ t["b1_up"][e]
                wd = torch.from_numpy(w_d[e]) + s * t["a2"][e] @ t["b2"][e]
                a = torch.nn.functional.silu(xs @ wg) * (xs @ wu)
                y = y.index_add(0, sel.nonzero()[:, 0], gates[sel, j:j + 1] * (a @ wd))
    np.testing.assert_allclose(y.detach().numpy(), f["Y"], rtol=1e-11, atol=1e-12)
    (y * torch.from_numpy(dy)).sum().backward()
    for n in t:
        np.testing.assert_allclose(b["d" + n], t[n].grad.numpy(), rtol=1e-10, atol=1e-11, err_msg=n)
    np.testing.assert_allclose(b["dx"], xt.grad.numpy(), rtol=1e-10, atol=1e-11)


# ------------------------------------------------------------ workloads
def test_workload_routing_statistics():
    """The Zipf workload: hottest expert about ten times the mean, four experts
    with no rows (router and selection only, at full size)."""
    d = workloads.make("zipf", only=set())
    x = O.widen_bf16(d["x"])
    w_r = O.widen_bf16(d["w_r"])
    idx = O.select_topk(O.router_logits(x, w_r), 8)
    c = np.bincount(idx.ravel(), minlength=128)
    assert (c == 0).sum() == 4
    assert 8.0 < c.max() / c.mean() < 12.0


def test_ep_share_rows_are_the_oracle_routing():
    """The stored rows of the expert-parallel share are what the oracle router
    sends to experts 0..15 on the seed-2 Qwen-shape batch (re-derived here),
    and the workload gathers exactly those token rows of that batch."""
    import importlib.util
    path = os.path.join(os.path.dirname(__file__), "golden", "make_ep_share_rows.py")
    spec = importlib.util.spec_from_file_location("make_ep_share_rows", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    counts, row_token = mod.compute()
    stored_tokens, stored_counts = workloads.ep_rows(8192, 2048, 128, 8, 2, 16)
    assert list(stored_counts) == counts and list(stored_tokens) == row_token
    # expert-major, tokens ascending within each expert, each token at most once per expert
    off = np.concatenate([[0], np.cumsum(counts)])
    for e in range(16):
        seg = np.asarray(row_token[off[e]:off[e + 1]])
        assert np.all(np.diff(seg) > 0)
    d = workloads.make("ep_share")
    x = workloads.make("qwen3_30b_a3b", seed=2, only=set())["x"]
    assert d["dims"]["R"] == sum(counts) == d["xp"].shape[0]
    assert np.array_equal(d["xp"], x[np.asarray(row_token)])


def test_long_passage_mask():
    d = workloads.make("long_passage", only=set())
    m = d["mask"].reshape(16, 4096)
    lens = m.sum(1)
    assert np.all(lens >= 2048) and np.all(lens <= 4096)
    assert np.all(m[:, :2048] == 1)
    assert np.array_equal(m, (np.arange(4096)[None] < lens[:, None]).astype(np.uint8))


def test_bf16_encoding_round_trip():
    v = np.array([1.0, -2.5, 3.14159, 1e-3, 65504.0, 1.00390625, 1.01171875], dtype=np.float32)
    b = workloads.bf16_bits(v)
    back = O.widen_bf16(b)
    # exactly representable values survive; others within half an ulp (2^-8 relative)
    assert back[0] == 1.0 and back[1] == -2.5
    assert np.all(np.abs(back - v) <= np.abs(v) * 2.0 ** -8)
    # ties go to the even mantissa: 1 + 2^-8 -> 1; 1 + 3*2^-8 -> 1 + 2^-6
    assert back[5] == 1.0 and back[6] == 1.015625


def test_fp32_instance_matches_fp64():
    """The oracle's single-precision instance (inputs widened to float32; the
    CPU baseline times it) is the same code in fp32: it routes every token
    away from near ties exactly as the fp64 instance and agrees with it to
    fp32 rounding on every output and gradient."""
    inp = workloads.make("tiny")
    d = inp["dims"]
    names = ("x", "w_r", "w_gate", "w_up", "w_down", "dy")
    runs = {}
    for dt in (np.float64, np.float32):
        w = {n: O.widen_bf16(inp[n], dt) for n in names}
        assert all(v.dtype == dt for v in w.values())
        f = O.moe_forward(w["x"], w["w_r"], w["w_gate"], w["w_up"], w["w_down"], d["k"])
        b = O.moe_backward(w["x"], w["w_r"], w["w_gate"], w["w_up"], w["w_down"], f, w["dy"])
        for n in ("Y", "G", "O"):
            assert f[n].dtype == dt, n
        for n in ("dx", "dw_r", "dw_gate", "dw_down"):
            assert b[n].dtype == dt, n
        runs[dt] = (f, b)
    (f64, b64), (f32, b32) = runs[np.float64], runs[np.float32]
    st, ot = O.near_ties(f64["z"], d["k"])
    clean = ~(st | ot)
    assert np.array_equal(f32["idx"][clean], f64["idx"][clean])
    # a set tie may route differently in fp32: such a token, and the experts it
    # reaches either way, are left out of the comparison
    flipped = np.array([set(a) != set(b) for a, b in zip(f32["idx"].tolist(), f64["idx"].tolist())])
    assert not (flipped & ~st).any()
    keep = ~flipped
    cols = ~touched_experts(flipped, f32["idx"], f64["idx"], d["E"])
    assert keep.sum() >= d["T"] - 2 and cols.sum() >= d["E"] - 4
    assert np.abs(f32["Y"] - f64["Y"])[keep].max() <= 1e-5 * np.abs(f64["Y"]).max()
    assert np.abs(b32["dx"] - b64["dx"])[keep].max() <= 1e-4 * np.abs(b64["dx"]).max()
    for n in ("dw_gate", "dw_up", "dw_down"):
        assert np.abs(b32[n] - b64[n])[cols].max() <= 1e-4 * np.abs(b64[n]).max(), n
    assert np.abs(b32["dw_r"] - b64["dw_r"])[:, cols].max() <= 1e-4 * np.abs(b64["dw_r"]).max()
