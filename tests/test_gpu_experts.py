"""GPU parity of the expert-parallel share (moe_experts_fwd / moe_experts_bwd)
against the oracle at small sizes: ragged and empty experts, rows left over
past the counts, and counts that overflow the row capacity (rows past the
capacity are dropped: never read, computed or written)."""
import numpy as np
import pytest

import workloads
from oracle import moe_oracle as O
from tests.parity import assert_close, dev_bf16, host

pytestmark = pytest.mark.gpu


def run(rows, H, E, F, counts, seed, dw_fp32=False):
    import torch
    import paper_2608_00916_amd as moe
    s = np.random.SeedSequence(seed).spawn(5)
    xp = workloads.normal_bf16(s[0], (rows, H), 1.0)
    wg = workloads.normal_bf16(s[1], (E, H, F), 0.02)
    wu = workloads.normal_bf16(s[2], (E, H, F), 0.02)
    wd = workloads.normal_bf16(s[3], (E, F, H), 0.02)
    d_o = workloads.normal_bf16(s[4], (rows, H), 1.0)
    counts = np.asarray(counts, dtype=np.int32)
    print(f"GPU experts rows={rows} H={H} E={E} F={F} counts={counts.tolist()}", flush=True)
    ex = moe.MoEExperts(rows, H, E, F, dw_fp32=dw_fp32)
    # sentinel in the output rows that must stay untouched
    ex.o.fill_(7.0)
    ex.dxp.fill_(7.0)
    t = {n: dev_bf16(a) for n, a in (("xp", xp), ("wg", wg), ("wu", wu), ("wd", wd), ("d_o", d_o))}
    ex.forward(t["xp"], torch.from_numpy(counts).cuda(), t["wg"], t["wu"], t["wd"])
    ex.backward(t["xp"], t["wg"], t["wu"], t["wd"], t["d_o"])
    torch.cuda.synchronize()
    # rows beyond the capacity are dropped: the definition restricted to the first `rows` rows
    used = np.minimum(np.cumsum(counts), rows)
    eff = np.diff(np.concatenate([[0], used]))
    R = int(used[-1])
    w = {n: O.widen_bf16(a) for n, a in (("xp", xp), ("wg", wg), ("wu", wu), ("wd", wd), ("d_o", d_o))}
    f = O.experts_share_forward(w["xp"][:R], eff, w["wg"], w["wu"], w["wd"])
    b = O.experts_share_backward(w["xp"][:R], eff, w["wg"], w["wu"], w["wd"], f, w["d_o"][:R])
    o = host(ex.o)
    dxp = host(ex.dxp)
    assert np.array_equal(host(ex.views["offsets"]), f["offsets"])
    if R:
        assert_close("o", o[:R], f["O"])
        assert_close("dxp", dxp[:R], b["dxp"])
    assert np.all(o[R:] == 7.0) and np.all(dxp[R:] == 7.0), "rows past the counts were written"
    tol = 5e-3 if dw_fp32 else 2e-2
    for n, got in (("dw_gate", ex.dw_gate), ("dw_up", ex.dw_up), ("dw_down", ex.dw_down)):
        got = host(got)
        for e in range(E):
            if eff[e] == 0:
                assert np.all(got[e] == 0), f"{n}[{e}] of an empty expert"
            else:
                assert_close(f"{n}[{e}]", got[e], b[n][e], tol)


def test_ragged_and_empty_experts():
    run(700, 256, 6, 128, [130, 0, 257, 1, 0, 300], seed=1)


def test_rows_left_over():
    run(600, 128, 4, 256, [100, 0, 200, 50], seed=2)


def test_counts_overflow_capacity():
    run(300, 128, 4, 128, [200, 150, 100, 0], seed=3)


def test_fp32_weight_grads():
    run(512, 256, 3, 128, [200, 150, 162], seed=4, dw_fp32=True)


def test_recompute_is_bit_identical():
    """The experts path with MOE_F_RECOMPUTE matches the run that kept G and U
    bit for bit."""
    import torch
    import paper_2608_00916_amd as moe
    rows, H, E, F = 700, 256, 6, 256
    counts = np.array([130, 0, 257, 1, 0, 300], dtype=np.int32)
    s = np.random.SeedSequence(5).spawn(5)
    t = {n: dev_bf16(workloads.normal_bf16(q, shape, std)) for n, q, shape, std in (
        ("xp", s[0], (rows, H), 1.0), ("wg", s[1], (E, H, F), 0.02), ("wu", s[2], (E, H, F), 0.02),
        ("wd", s[3], (E, F, H), 0.02), ("d_o", s[4], (rows, H), 1.0))}
    print(f"GPU experts recompute rows={rows} H={H} E={E} F={F}", flush=True)
    c = torch.from_numpy(counts).cuda()
    outs = []
    for recompute in (False, True):
        ex = moe.MoEExperts(rows, H, E, F, recompute=recompute)
        ex.o.zero_()
        ex.dxp.zero_()
        ex.forward(t["xp"], c, t["wg"], t["wu"], t["wd"])
        ex.backward(t["xp"], t["wg"], t["wu"], t["wd"], t["d_o"])
        torch.cuda.synchronize()
        outs.append({n: host(getattr(ex, n)) for n in ("o", "dxp", "dw_gate", "dw_up", "dw_down")})
        outs[-1]["a"] = host(ex.views["a"][:int(counts.sum())])  # rows past the counts are undefined
        if recompute:
            assert ex.views["g"] is None and ex.views["u"] is None
    for n in outs[0]:
        assert np.array_equal(outs[0][n], outs[1][n]), n
