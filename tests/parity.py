"""Shared helpers of the GPU parity tests: device transfer of the seeded
inputs, the tolerance measures, and routing checks that allow for near ties.

The expected values always come from the fp64 oracle run on the seeded
inputs; nothing computed by the GPU is ever fed to the oracle."""
from __future__ import annotations

import numpy as np

from oracle import moe_oracle as O

# Spec tolerance for outputs and gradients: bf16 storage, fp32
# accumulation, measured per tensor as max|gpu - ref| / max|ref|.
TOL = 2e-2
# Router logits are fp32 sums of exact bf16 products.
LOGIT_TOL = 1e-5
GATE_TOL = 1e-5
TIE_GAP = 1e-4


def dev_bf16(bits, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device).view(torch.bfloat16)


def host(t):
    """GPU tensor -> float64 / int64 numpy."""
    import torch
    if t.dtype in (torch.bfloat16, torch.float16, torch.float32):
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy().astype(np.int64)


def max_rel_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    scale = np.abs(ref).max()
    if scale == 0:
        return float(np.abs(got).max())
    return float(np.abs(got - ref).max() / scale)


def frac_outside(got, ref, rel=TOL, floor=1e-3):
    """Fraction of elements with |got - ref| > rel |ref| + floor max|ref|."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    lim = rel * np.abs(ref) + floor * np.abs(ref).max()
    return float(np.mean(np.abs(got - ref) > lim))


def assert_close(name, got, ref, tol=TOL):
    e = max_rel_err(got, ref)
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    assert e <= tol, f"{name}: max rel err {e:.3e} > {tol:.1e} (outside-frac {frac_outside(got, ref):.2e})"
    return e


def router_grad_bound(f, dY, x):
    """Elementwise bound on the error of dW_r that a relative error TOL on every
    element of O (the expert outputs) produces through dg -> dz -> dW_r.

    dg_j = <dY_t, O_j> then carries at most TOL a_j with a_j = sum_h |dY_th O_jh|,
    and dz_j = g_j (dg_j - sum_j' g_j' dg_j') at most TOL c_j with
    c_j = g_j (a_j + sum_j' g_j' a_j'); dW_r = x^T dz sums |x_th| TOL c_t(e).
    A single token's dz is a difference of such dot products, so its relative
    error is unbounded when they nearly cancel; this bound is what a 2e-2 budget
    on O allows there."""
    T, k = f["idx"].shape
    E = f["z"].shape[1]
    C = np.zeros((T, E))
    g = f["gates"]
    a = np.zeros((T, k))
    for j in range(k):
        valid = f["row_of"][:, j] >= 0
        a[valid, j] = np.sum(np.abs(dY[valid]) * np.abs(f["O"][f["row_of"][valid, j]]), axis=1)
    c = g * (a + np.sum(g * a, axis=1, keepdims=True))
    for j in range(k):
        valid = f["idx"][:, j] >= 0
        C[np.nonzero(valid)[0], f["idx"][valid, j]] = c[valid, j]
    return TOL * (np.abs(x).T @ C)


def assert_router_grad(got, ref, bound):
    """dW_r within TOL (max-relative) or, where cancellation makes that measure
    ill-conditioned, within the propagated bound of router_grad_bound."""
    if max_rel_err(got, ref) <= TOL:
        return
    excess = np.abs(got - ref) - bound
    assert np.all(excess <= 1e-12), f"dw_r: {np.sum(excess > 0)} elements beyond the propagated bound"


def check_routing(z_ref, idx_ref, gates_ref, gpu_logits, gpu_idx, gpu_gates, k, mask=None):
    """Compare the GPU's routing with the oracle's.

    Tokens whose fp32 logits hold a near tie (oracle logits, gap < 1e-4) may
    legitimately differ: their selection is checked for validity instead.
    Returns (n_set_ties, n_order_ties, flipped) where `flipped` marks tokens
    whose selected expert *set* differs from the oracle's."""
    T = z_ref.shape[0]
    valid = np.ones(T, dtype=bool) if mask is None else mask.astype(bool)
    assert max_rel_err(gpu_logits[valid], z_ref[valid]) <= LOGIT_TOL
    set_tie, order_tie = O.near_ties(z_ref, k, gap=TIE_GAP, mask=valid)
    clean = valid & ~set_tie & ~order_tie
    assert np.array_equal(gpu_idx[clean], idx_ref[clean]), "expert indices differ away from near ties"
    assert np.all(gpu_idx[~valid] == -1) and np.all(gpu_gates[~valid] == 0)
    np.testing.assert_allclose(gpu_gates[clean], gates_ref[clean], rtol=0, atol=GATE_TOL)
    # near ties: the GPU's choice must be a valid top-k under a TIE_GAP slack
    key = z_ref.astype(np.float32).astype(np.float64)
    flipped = np.zeros(T, dtype=bool)
    for t in np.nonzero(valid & (set_tie | order_tie))[0]:
        sel = gpu_idx[t]
        assert len(set(sel.tolist())) == k and sel.min() >= 0
        kth = np.sort(key[t])[::-1][k - 1]
        assert np.all(key[t, sel] >= kth - TIE_GAP), f"token {t}: invalid selection"
        assert np.all(np.diff(key[t, sel]) <= TIE_GAP), f"token {t}: slots out of order"
        assert abs(gpu_gates[t].sum() - 1) < 1e-5
        flipped[t] = set(sel.tolist()) != set(idx_ref[t].tolist())
    return int(set_tie.sum()), int(order_tie.sum()), flipped


def check_permutation_valid(idx, counts, offsets, row_token, row_of, E):
    """The GPU permutation is the unique stable expert-major permutation of
    its own selection (validity of integer outputs)."""
    T, k = idx.shape
    hist = np.bincount(idx[idx >= 0].ravel(), minlength=E)
    assert np.array_equal(counts, hist)
    assert offsets[0] == 0 and np.array_equal(np.diff(offsets), counts)
    R = offsets[E]
    assert np.all(row_token[R:] == -1)
    tok = np.repeat(np.arange(T), k).reshape(T, k)
    val = idx >= 0
    assert np.all(row_of[~val] == -1)
    rows = row_of[val]
    assert np.array_equal(np.sort(rows), np.arange(R)), "rows are not a bijection onto [0, R)"
    assert np.array_equal(row_token[rows], tok[val])
    # row r of expert e lies in [offsets[e], offsets[e+1]) and tokens ascend within an expert
    exp_of_row = np.empty(R, dtype=np.int64)
    exp_of_row[rows] = idx[val]
    for e in range(E):
        seg = slice(offsets[e], offsets[e + 1])
        assert np.all(exp_of_row[seg] == e)
        assert np.all(np.diff(row_token[seg]) > 0)
