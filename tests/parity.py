"""Shared helpers of the GPU parity tests: device transfer of the seeded
inputs, the tolerance measure, routing checks that allow for near ties, and a
record of every measured error.

The expected values always come from the fp64 oracle run on the seeded
inputs; nothing computed by the GPU is ever fed to the oracle."""
from __future__ import annotations

import json
import os

import numpy as np

from oracle import moe_oracle as O

# Tolerance for outputs and gradients: bf16 storage, fp32 accumulation,
# measured per tensor as max|gpu - ref| / max|ref|.
TOL = 2e-2
# Router logits are fp32 sums of exact bf16 products.
LOGIT_TOL = 1e-5
GATE_TOL = 1e-5
TIE_GAP = 1e-4

# case -> {quantity: value}: every error and near-tie count the GPU tests
# measured in this process (written out by conftest at the end of the session).
RECORD: dict = {}


def record(case, **vals):
    RECORD.setdefault(case, {}).update(vals)


def write_record(path):
    if not RECORD:
        return
    os.makedirs(os.path.dirname(os.path.abspath(path)), exist_ok=True)
    old = {}
    if os.path.exists(path):
        try:
            old = json.load(open(path))
        except ValueError:
            old = {}
    old.update(RECORD)
    json.dump(old, open(path, "w"), indent=1, sort_keys=True)


GUARD_BYTES = 4096  # sentinel bytes before and after every guarded caller buffer
SENTINEL = 0xA5


class Guards:
    """Caller-owned buffers inside larger allocations whose extra bytes on
    both sides hold a sentinel: a write outside a buffer's own extent changes
    a sentinel and `check` fails."""

    def __init__(self):
        self.raws = []

    def like(self, t):
        import torch
        n = t.numel() * t.element_size()
        raw = torch.full((n + 2 * GUARD_BYTES,), SENTINEL, dtype=torch.uint8, device=t.device)
        self.raws.append((raw, n))
        return raw[GUARD_BYTES:GUARD_BYTES + n].view(t.dtype).view(t.shape)

    def check(self):
        for raw, n in self.raws:
            head = raw[:GUARD_BYTES].cpu().numpy()
            tail = raw[GUARD_BYTES + n:].cpu().numpy()
            assert np.all(head == SENTINEL) and np.all(tail == SENTINEL), \
                f"a write landed outside a {n}-byte caller buffer"


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
    if got.size == 0:
        return 0.0
    scale = np.abs(ref).max()
    if scale == 0:
        return float(np.abs(got).max())
    return float(np.abs(got - ref).max() / scale)


def frac_outside(got, ref, rel=TOL, floor=1e-3):
    """Fraction of elements with |got - ref| > rel |ref| + floor max|ref|."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if got.size == 0:
        return 0.0
    lim = rel * np.abs(ref) + floor * np.abs(ref).max()
    return float(np.mean(np.abs(got - ref) > lim))


def assert_close(name, got, ref, tol=TOL, case=None):
    """Per-tensor max-relative error within `tol`; the error is recorded
    under `case` when one is given."""
    e = max_rel_err(got, ref)
    if case is not None:
        rec = RECORD.setdefault(case, {})
        rec[name] = max(e, rec.get(name, 0.0))
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    assert e <= tol, f"{name}: max rel err {e:.3e} > {tol:.1e} (outside-frac {frac_outside(got, ref):.2e})"
    return e


def check_routing(z_ref, idx_ref, gates_ref, gpu_logits, gpu_idx, gpu_gates, k, mask=None, case=None):
    """Compare the GPU's routing with the oracle's.

    Tokens whose fp32 logits hold a near tie (oracle logits, gap < 1e-4) may
    legitimately differ: their selection is checked for validity instead.
    Returns (n_set_ties, n_order_ties, flipped) where `flipped` marks tokens
    whose selected expert *set* differs from the oracle's.  A flip is only
    possible on a set tie: every other token's experts are compared exactly."""
    T = z_ref.shape[0]
    valid = np.ones(T, dtype=bool) if mask is None else mask.astype(bool)
    le = max_rel_err(gpu_logits[valid], z_ref[valid])
    assert le <= LOGIT_TOL, f"logits: max rel err {le:.3e}"
    set_tie, order_tie = O.near_ties(z_ref, k, gap=TIE_GAP, mask=valid)
    clean = valid & ~set_tie & ~order_tie
    assert np.array_equal(gpu_idx[clean], idx_ref[clean]), "expert indices differ away from near ties"
    assert np.all(gpu_idx[~valid] == -1) and np.all(gpu_gates[~valid] == 0)
    ge = float(np.abs(gpu_gates[clean] - gates_ref[clean]).max()) if clean.any() else 0.0
    assert ge <= GATE_TOL, f"gates: max abs err {ge:.3e}"
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
    assert not (flipped & ~set_tie).any(), "an expert set differs on a token without a set tie"
    if case is not None:
        record(case, logits=le, gates_abs=ge, near_ties_set=int(set_tie.sum()),
               near_ties_order=int(order_tie.sum()), flipped=int(flipped.sum()), tokens=int(valid.sum()))
    return int(set_tie.sum()), int(order_tie.sum()), flipped


def touched_experts(flipped, gpu_idx, ref_idx, E):
    """Experts that a flipped token reaches under either routing: their rows,
    and so their weight gradients and dW_r columns, differ between the two
    runs legitimately; every other expert sees the same tokens in both."""
    touched = np.zeros(E, dtype=bool)
    for t in np.nonzero(flipped)[0]:
        for e in np.concatenate([gpu_idx[t], ref_idx[t]]):
            if e >= 0:
                touched[e] = True
    return touched


def row_pairs(gpu_idx, gpu_row_of, ref_idx, ref_row_of, tokens):
    """For each routed (token, expert) pair of the given tokens, the GPU's row
    and the oracle's row holding it (slot order may differ on order ties)."""
    g_rows, r_rows = [], []
    for t in tokens:
        ref_slot = {int(e): j for j, e in enumerate(ref_idx[t]) if e >= 0}
        for j, e in enumerate(gpu_idx[t]):
            if e < 0:
                continue
            g_rows.append(gpu_row_of[t, j])
            r_rows.append(ref_row_of[t, ref_slot[int(e)]])
    return np.asarray(g_rows, dtype=np.int64), np.asarray(r_rows, dtype=np.int64)


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
