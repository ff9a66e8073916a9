"""Plain fp64 CPU oracle of the mixture-of-experts FFN block, forward and backward.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the bench's
CPU-baseline leg may import this module.  The GPU path shares no code with it.

What is computed.  The paper (§3, Expert-Parallel MoE Training) trains a
Qwen3-30B-A3B reranker whose MoE layers hold 128 experts and send each token to
its top-8 experts; expert parallelism dispatches routed tokens to the ranks
holding their experts (§3, "Expert parallelism and topology").  The paper does
not print the block's equations, so this oracle writes out the standard
dropless top-k MoE with SwiGLU experts, under these readings:

* router logits z = x W_r in full precision; the selection is made on the fp32
  rounding of z (the precision the GPU path decides in); ties go to the lower
  expert index; slots are ordered by descending logit;
* gates are the softmax over the k selected logits (equal to the full softmax
  renormalised over the selection);
* no capacity limit, no dropped tokens, no shared expert, no router bias;
  by default no auxiliary loss; optionally (the paper is silent on it; see
  router_aux_loss) a load-balancing loss and a z-loss on the router logits;
* masked (padding) tokens are not routed: they get no rows, Y = 0, dX = 0;
* rows are permuted expert-major and, within an expert, by ascending token;
* gates multiply the expert outputs at combine time;
* the router gradient flows through the gates only (the selection is
  piecewise constant).

Precision: every float array is computed in the dtype the inputs are widened
to (widen_bf16's `dtype`): float64 by default, the reference the GPU tests
compare against; float32 gives the single-precision instance of the same
code, which the CPU baseline times.  bf16 inputs arrive as uint16 bit patterns
and are widened exactly.  Each function is a direct transcription of one step; there is
no blocking, fusion or reordering beyond what the definition states.
"""
from __future__ import annotations

import numpy as np


# ---------------------------------------------------------------- inputs
def widen_bf16(bits, dtype=np.float64) -> np.ndarray:
    """bf16 bit pattern (uint16) -> `dtype` (float64 or float32), exactly."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(dtype)


def silu(v):
    return v / (1.0 + np.exp(-v))


def sigmoid(v):
    return 1.0 / (1.0 + np.exp(-v))


# ---------------------------------------------------------------- forward
def router_logits(x, w_r):
    """z[t,e] = sum_h x[t,h] W_r[h,e]  (router GEMM)."""
    return x @ w_r


def select_topk(z, k, mask=None):
    """Top-k expert selection per valid token.

    Selection key: the fp32 rounding of z.  k rounds of argmax over the experts
    not yet taken; np.argmax returns the first maximum, so equal keys go to the
    lower expert index.  Slot j holds the j-th largest key.  Masked tokens get
    idx = -1."""
    T, E = z.shape
    key = z.astype(np.float32).astype(np.float64)
    idx = np.full((T, k), -1, dtype=np.int64)
    taken = np.zeros((T, E), dtype=bool)
    rows = np.arange(T)
    for j in range(k):
        cand = np.where(taken, -np.inf, key)
        e = np.argmax(cand, axis=1)
        idx[:, j] = e
        taken[rows, e] = True
    if mask is not None:
        idx[~mask] = -1
    return idx


def topk_gates(z, idx):
    """g[t,j] = exp(z[t,idx_j] - m) / sum_j' exp(z[t,idx_j'] - m), m the largest
    selected logit.  Masked tokens (idx = -1) get g = 0."""
    T, k = idx.shape
    valid = idx[:, 0] >= 0
    zs = np.take_along_axis(z, np.where(idx < 0, 0, idx), axis=1)
    m = zs.max(axis=1, keepdims=True)
    w = np.exp(zs - m)
    g = w / w.sum(axis=1, keepdims=True)
    g[~valid] = 0.0
    return g


def permutation(idx, E):
    """Counting sort of the routed (token, slot) pairs by expert.

    counts[e]   number of valid (t, j) with idx[t,j] = e
    offsets     exclusive prefix sum of counts, length E+1; R = offsets[E]
    row_token   row_token[r] = t for r < R, -1 beyond (length T*k)
    row_of      row_of[t,j] = r, -1 for masked tokens
    Rows are expert-major; within one expert the tokens ascend."""
    T, k = idx.shape
    counts = np.zeros(E, dtype=np.int64)
    for e in range(E):
        counts[e] = np.count_nonzero(idx == e)
    offsets = np.zeros(E + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    row_token = np.full(T * k, -1, dtype=np.int64)
    row_of = np.full((T, k), -1, dtype=np.int64)
    for e in range(E):
        r = offsets[e]
        toks, slots = np.nonzero(idx == e)  # row-major scan: tokens ascend
        for t, j in zip(toks, slots):
            row_token[r] = t
            row_of[t, j] = r
            r += 1
        assert r == offsets[e + 1]
    return counts, offsets, row_token, row_of


def gather_rows(x, row_token, R):
    """Xp[r] = x[row_token[r]] for r < R."""
    return x[row_token[:R]]


def experts_forward(xp, offsets, w_gate, w_up, w_down):
    """Per expert e on its rows [offsets[e], offsets[e+1]):
    G = Xp_e W_gate[e], U = Xp_e W_up[e], A = silu(G) * U, O = A W_down[e]."""
    R = xp.shape[0]
    F = w_gate.shape[2]
    H = w_down.shape[2]
    G = np.zeros((R, F), dtype=xp.dtype)
    U = np.zeros((R, F), dtype=xp.dtype)
    A = np.zeros((R, F), dtype=xp.dtype)
    O = np.zeros((R, H), dtype=xp.dtype)
    for e in range(w_gate.shape[0]):
        lo, hi = offsets[e], offsets[e + 1]
        if hi == lo:
            continue
        G[lo:hi] = xp[lo:hi] @ w_gate[e]
        U[lo:hi] = xp[lo:hi] @ w_up[e]
        A[lo:hi] = silu(G[lo:hi]) * U[lo:hi]
        O[lo:hi] = A[lo:hi] @ w_down[e]
    return G, U, A, O


def combine(O, gates, row_of):
    """Y[t] = sum over slots j (in order) of g[t,j] * O[row_of[t,j]]; Y = 0 for
    masked tokens."""
    T, k = row_of.shape
    Y = np.zeros((T, O.shape[1]), dtype=O.dtype)
    for j in range(k):
        valid = row_of[:, j] >= 0
        Y[valid] += gates[valid, j:j + 1] * O[row_of[valid, j]]
    return Y


def moe_forward(x, w_r, w_gate, w_up, w_down, k, mask=None):
    """Whole block forward.  Float arguments all float64 (or all float32);
    mask bool[T] or None."""
    E = w_r.shape[1]
    z = router_logits(x, w_r)
    idx = select_topk(z, k, mask)
    g = topk_gates(z, idx)
    counts, offsets, row_token, row_of = permutation(idx, E)
    R = int(offsets[E])
    xp = gather_rows(x, row_token, R)
    G, U, A, O = experts_forward(xp, offsets, w_gate, w_up, w_down)
    Y = combine(O, g, row_of)
    return dict(z=z, idx=idx, gates=g, counts=counts, offsets=offsets,
                row_token=row_token, row_of=row_of, R=R, xp=xp, G=G, U=U, A=A,
                O=O, Y=Y)


# ---------------------------------------------------------------- backward
def combine_backward(dY, O, gates, row_of):
    """dO[row_of[t,j]] = g[t,j] dY[t];  dg[t,j] = <dY[t], O[row_of[t,j]]>."""
    T, k = row_of.shape
    dO = np.zeros_like(O)
    dg = np.zeros((T, k), dtype=O.dtype)
    for j in range(k):
        valid = row_of[:, j] >= 0
        r = row_of[valid, j]
        dO[r] = gates[valid, j:j + 1] * dY[valid]
        dg[valid, j] = np.sum(dY[valid] * O[r], axis=1)
    return dO, dg


def experts_backward(xp, offsets, w_gate, w_up, w_down, G, U, A, dO):
    """Per expert: dA = dO W_down^T; dW_down = A^T dO;
    SwiGLU backward with s = sigmoid(G): dG = dA U s (1 + G (1 - s)),
    dU = dA silu(G); dXp = dG W_gate^T + dU W_up^T; dW_gate = Xp^T dG,
    dW_up = Xp^T dU.  Experts with no rows get zero weight gradients."""
    E = w_gate.shape[0]
    dxp = np.zeros_like(xp)
    dw_gate = np.zeros_like(w_gate)
    dw_up = np.zeros_like(w_up)
    dw_down = np.zeros_like(w_down)
    dG = np.zeros_like(G)
    dU = np.zeros_like(U)
    for e in range(E):
        lo, hi = offsets[e], offsets[e + 1]
        if hi == lo:
            continue
        dA = dO[lo:hi] @ w_down[e].T
        dw_down[e] = A[lo:hi].T @ dO[lo:hi]
        s = sigmoid(G[lo:hi])
        dG[lo:hi] = dA * U[lo:hi] * s * (1.0 + G[lo:hi] * (1.0 - s))
        dU[lo:hi] = dA * silu(G[lo:hi])
        dxp[lo:hi] = dG[lo:hi] @ w_gate[e].T + dU[lo:hi] @ w_up[e].T
        dw_gate[e] = xp[lo:hi].T @ dG[lo:hi]
        dw_up[e] = xp[lo:hi].T @ dU[lo:hi]
    return dict(dxp=dxp, dw_gate=dw_gate, dw_up=dw_up, dw_down=dw_down,
                dG=dG, dU=dU)


def router_backward(gates, dg, idx, E):
    """Softmax-over-selection backward: with dg_j = dL/dg_j,
    dz[t, idx_j] = g_j (dg_j - sum_j' g_j' dg_j'), zero on unselected experts
    and on masked tokens."""
    T, k = idx.shape
    dz = np.zeros((T, E), dtype=dg.dtype)
    inner = np.sum(gates * dg, axis=1, keepdims=True)
    dzs = gates * (dg - inner)
    for j in range(k):
        valid = idx[:, j] >= 0
        dz[np.nonzero(valid)[0], idx[valid, j]] = dzs[valid, j]
    return dz


def unpermute_sum(dxp, row_of, T):
    """sum over slots j of dXp[row_of[t,j]] (zero for masked tokens)."""
    k = row_of.shape[1]
    out = np.zeros((T, dxp.shape[1]), dtype=dxp.dtype)
    for j in range(k):
        valid = row_of[:, j] >= 0
        out[valid] += dxp[row_of[valid, j]]
    return out


# ---------------------------------------------------------------- router losses
def router_probs(z, mask=None):
    """Full softmax over the experts of each token, and its log-normaliser
    lse_t = log sum_e exp z[t,e].  Masked tokens: p = 0, lse = 0."""
    m = np.max(z, axis=1, keepdims=True)
    ez = np.exp(z - m)
    s = np.sum(ez, axis=1, keepdims=True)
    p = ez / s
    lse = (m + np.log(s))[:, 0]
    if mask is not None:
        p = np.where(mask[:, None], p, 0.0)
        lse = np.where(mask, lse, 0.0)
    return p, lse


def router_aux_loss(z, idx, aux_coef, z_coef, mask=None):
    """Auxiliary router losses over the T_v valid tokens (the paper is silent
    on them; these are the load-balancing loss of Switch/GShard-style MoE
    training and the router z-loss):
        L_aux = aux_coef * E * sum_e f_e P_e,
            f_e = (routed slots of expert e) / (T_v k),  P_e = mean_t p[t,e];
        L_z   = z_coef * mean_t lse_t^2.
    Returns (L_aux, L_z)."""
    T, E = z.shape
    k = idx.shape[1]
    valid = np.ones(T, dtype=bool) if mask is None else mask
    Tv = int(valid.sum())
    if Tv == 0:
        return 0.0, 0.0
    p, lse = router_probs(z, valid)
    f = np.zeros(E)
    for e in range(E):
        f[e] = np.count_nonzero(idx[valid] == e) / (Tv * k)
    P = p[valid].sum(axis=0) / Tv
    l_aux = aux_coef * E * float(np.dot(f, P))
    l_z = z_coef * float(np.sum(lse[valid] ** 2)) / Tv
    return l_aux, l_z


def router_aux_dz(z, idx, aux_coef, z_coef, mask=None):
    """d(L_aux + L_z)/dz with the routing fractions f held constant (they
    are piecewise constant in z):
        dL_aux/dz[t,i] = aux_coef E / T_v * p[t,i] (f_i - sum_e f_e p[t,e]),
        dL_z/dz[t,i]   = z_coef 2 / T_v * lse_t p[t,i];
    zero on masked tokens."""
    T, E = z.shape
    k = idx.shape[1]
    valid = np.ones(T, dtype=bool) if mask is None else mask
    Tv = int(valid.sum())
    dz = np.zeros((T, E))
    if Tv == 0:
        return dz
    p, lse = router_probs(z, valid)
    f = np.array([np.count_nonzero(idx[valid] == e) for e in range(E)]) / (Tv * k)
    fp = p @ f
    dz += aux_coef * E / Tv * p * (f[None, :] - fp[:, None])
    dz += z_coef * 2.0 / Tv * lse[:, None] * p
    dz[~valid] = 0.0
    return dz


def moe_backward(x, w_r, w_gate, w_up, w_down, fwd, dY, aux=None, mask=None):
    """Whole block backward: dX, dW_r, dW_gate, dW_up, dW_down.  With
    aux = (aux_coef, z_coef) the router losses' gradient joins dz (the
    losses enter the objective with weight 1)."""
    E = w_r.shape[1]
    T = x.shape[0]
    dO, dg = combine_backward(dY, fwd["O"], fwd["gates"], fwd["row_of"])
    eb = experts_backward(fwd["xp"], fwd["offsets"], w_gate, w_up, w_down,
                          fwd["G"], fwd["U"], fwd["A"], dO)
    dz = router_backward(fwd["gates"], dg, fwd["idx"], E)
    if aux is not None:
        dz = dz + router_aux_dz(fwd["z"], fwd["idx"], aux[0], aux[1], mask)
    dw_r = x.T @ dz
    dx = unpermute_sum(eb["dxp"], fwd["row_of"], T) + dz @ w_r.T
    return dict(dx=dx, dw_r=dw_r, dw_gate=eb["dw_gate"], dw_up=eb["dw_up"],
                dw_down=eb["dw_down"], dO=dO, dg=dg, dz=dz, dxp=eb["dxp"],
                dG=eb["dG"], dU=eb["dU"])


# ---------------------------------------------------------------- expert LoRA
def lora_forward(x, w_r, w_gate, w_up, w_down, lora, k, mask=None):
    """Block forward with rank-r adapters on every expert's gate/up (the fused
    first projection) and down projections, base weights and router frozen
    (§3, "LoRA target groups for MoE": adapters on the experts, router left
    frozen).  lora = dict(scale, a1 [E,H,r], b1_gate [E,r,F], b1_up [E,r,F],
    a2 [E,F,r], b2 [E,r,H]); per expert e the effective weights are
        W_gate + scale a1 b1_gate,  W_up + scale a1 b1_up,  W_down + scale a2 b2,
    computed through the rank-r intermediates P1 = scale Xp a1 and
    P2 = scale A a2:
        G = Xp W_gate + P1 b1_gate,  U = Xp W_up + P1 b1_up,  A = silu(G) U,
        O = A W_down + P2 b2."""
    E = w_r.shape[1]
    s = lora["scale"]
    z = router_logits(x, w_r)
    idx = select_topk(z, k, mask)
    g = topk_gates(z, idx)
    counts, offsets, row_token, row_of = permutation(idx, E)
    R = int(offsets[E])
    xp = gather_rows(x, row_token, R)
    F = w_gate.shape[2]
    r = lora["a1"].shape[2]
    G = np.zeros((R, F), dtype=xp.dtype)
    U = np.zeros((R, F), dtype=xp.dtype)
    A = np.zeros((R, F), dtype=xp.dtype)
    O = np.zeros((R, w_down.shape[2]), dtype=xp.dtype)
    P1 = np.zeros((R, r), dtype=xp.dtype)
    P2 = np.zeros((R, r), dtype=xp.dtype)
    for e in range(E):
        lo, hi = offsets[e], offsets[e + 1]
        if hi == lo:
            continue
        P1[lo:hi] = s * (xp[lo:hi] @ lora["a1"][e])
        G[lo:hi] = xp[lo:hi] @ w_gate[e] + P1[lo:hi] @ lora["b1_gate"][e]
        U[lo:hi] = xp[lo:hi] @ w_up[e] + P1[lo:hi] @ lora["b1_up"][e]
        A[lo:hi] = silu(G[lo:hi]) * U[lo:hi]
        P2[lo:hi] = s * (A[lo:hi] @ lora["a2"][e])
        O[lo:hi] = A[lo:hi] @ w_down[e] + P2[lo:hi] @ lora["b2"][e]
    Y = combine(O, g, row_of)
    return dict(z=z, idx=idx, gates=g, counts=counts, offsets=offsets,
                row_token=row_token, row_of=row_of, R=R, xp=xp, G=G, U=U, A=A,
                O=O, Y=Y, P1=P1, P2=P2)


def lora_backward(x, w_r, w_gate, w_up, w_down, lora, fwd, dY):
    """Backward of lora_forward with the base weights and the router frozen:
    dX and the adapter gradients.  Per expert, with Q2 = scale dO b2^T and
    Q1 = scale (dG b1_gate^T + dU b1_up^T):
        dA = dO W_down^T + Q2 a2^T,   d a2 = A^T Q2,   d b2 = P2^T dO,
        dG, dU from dA (SwiGLU backward),
        dXp = dG W_gate^T + dU W_up^T + Q1 a1^T,
        d a1 = Xp^T Q1,  d b1_gate = P1^T dG,  d b1_up = P1^T dU;
    dX = unpermute-sum of dXp + dz W_r^T (the router's input gradient; no
    dW_r).  Experts with no rows get zero adapter gradients."""
    E = w_r.shape[1]
    T = x.shape[0]
    s = lora["scale"]
    dO, dg = combine_backward(dY, fwd["O"], fwd["gates"], fwd["row_of"])
    R = fwd["R"]
    xp, G, U, A = fwd["xp"], fwd["G"], fwd["U"], fwd["A"]
    offsets = fwd["offsets"]
    dxp = np.zeros_like(xp)
    grads = {n: np.zeros_like(lora[n]) for n in ("a1", "b1_gate", "b1_up", "a2", "b2")}
    r = lora["a1"].shape[2]
    Q1 = np.zeros((R, r), dtype=xp.dtype)
    Q2 = np.zeros((R, r), dtype=xp.dtype)
    dG = np.zeros_like(G)
    dU = np.zeros_like(U)
    for e in range(E):
        lo, hi = offsets[e], offsets[e + 1]
        if hi == lo:
            continue
        Q2[lo:hi] = s * (dO[lo:hi] @ lora["b2"][e].T)
        dA = dO[lo:hi] @ w_down[e].T + Q2[lo:hi] @ lora["a2"][e].T
        grads["a2"][e] = A[lo:hi].T @ Q2[lo:hi]
        grads["b2"][e] = fwd["P2"][lo:hi].T @ dO[lo:hi]
        sg = sigmoid(G[lo:hi])
        dG[lo:hi] = dA * U[lo:hi] * sg * (1.0 + G[lo:hi] * (1.0 - sg))
        dU[lo:hi] = dA * silu(G[lo:hi])
        Q1[lo:hi] = s * (dG[lo:hi] @ lora["b1_gate"][e].T + dU[lo:hi] @ lora["b1_up"][e].T)
        dxp[lo:hi] = (dG[lo:hi] @ w_gate[e].T + dU[lo:hi] @ w_up[e].T
                      + Q1[lo:hi] @ lora["a1"][e].T)
        grads["a1"][e] = xp[lo:hi].T @ Q1[lo:hi]
        grads["b1_gate"][e] = fwd["P1"][lo:hi].T @ dG[lo:hi]
        grads["b1_up"][e] = fwd["P1"][lo:hi].T @ dU[lo:hi]
    dz = router_backward(fwd["gates"], dg, fwd["idx"], E)
    dx = unpermute_sum(dxp, fwd["row_of"], T) + dz @ w_r.T
    out = dict(dx=dx, dO=dO, dG=dG, dU=dU, dxp=dxp, Q1=Q1, Q2=Q2, dz=dz)
    out.update({"d" + n: v for n, v in grads.items()})
    return out


# ---------------------------------------------------------------- one EP rank
def offsets_of(counts):
    offsets = np.zeros(len(counts) + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    return offsets


def experts_share_forward(xp, counts, w_gate, w_up, w_down):
    """One expert-parallel rank's local experts (§3): rows already grouped
    expert-major, counts[e] rows for local expert e."""
    offsets = offsets_of(counts)
    G, U, A, O = experts_forward(xp, offsets, w_gate, w_up, w_down)
    return dict(offsets=offsets, G=G, U=U, A=A, O=O)


def experts_share_backward(xp, counts, w_gate, w_up, w_down, fwd, d_o):
    offsets = offsets_of(counts)
    return experts_backward(xp, offsets, w_gate, w_up, w_down,
                            fwd["G"], fwd["U"], fwd["A"], d_o)


# ---------------------------------------------------------------- sampled checks
def token_forward(x_t, w_r, w_gate, w_up, w_down, k):
    """Forward of the block for single tokens (rows of x_t), independent of the
    rest of the batch: used to check full-size outputs on sampled tokens."""
    z = router_logits(x_t, w_r)
    idx = select_topk(z, k)
    g = topk_gates(z, idx)
    Y = np.zeros((x_t.shape[0], w_down.shape[2]))
    O = np.zeros((x_t.shape[0], k, w_down.shape[2]))
    for i in range(x_t.shape[0]):
        for j in range(k):
            e = idx[i, j]
            a = silu(x_t[i] @ w_gate[e]) * (x_t[i] @ w_up[e])
            O[i, j] = a @ w_down[e]
            Y[i] += g[i, j] * O[i, j]
    return dict(z=z, idx=idx, gates=g, O=O, Y=Y)


def near_ties(z, k, gap=1e-4, mask=None):
    """Tokens whose selection may legitimately differ between two correct
    implementations whose fp32 logits differ by rounding.

    set_tie[t]    the k-th and (k+1)-th largest keys differ by less than `gap`
                  (the selected set itself is uncertain);
    order_tie[t]  two adjacent keys among the k largest differ by less than
                  `gap` (the set is certain, the slot order is not)."""
    key = np.sort(z.astype(np.float32).astype(np.float64), axis=1)[:, ::-1]
    T, E = z.shape
    set_tie = np.zeros(T, dtype=bool)
    if k < E:
        set_tie = (key[:, k - 1] - key[:, k]) < gap
    order_tie = np.zeros(T, dtype=bool)
    if k > 1:
        order_tie = np.any((key[:, :k - 1] - key[:, 1:k]) < gap, axis=1)
    if mask is not None:
        set_tie &= mask
        order_tie &= mask
    return set_tie, order_tie
