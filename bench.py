#!/usr/bin/env python3
"""Throughput of the MoE block, forward + backward, on one MI355X.

One step = moe_fwd + moe_bwd over one batch of the workload (router, top-k,
permutation, SwiGLU expert products, combine, and the whole backward), inputs
resident in HBM before the timed region.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload qwen3_30b_a3b]

The workload defaults to the Qwen3-30B-A3B-shaped layer on one GPU (T=8192
tokens, H=2048, E=128 experts, top-8, F=768, bf16).  The dominant kernel's
roofline comes from HIP events recorded around every library kernel launch
over a second pass of the timed steps.  The Zipf-routed (T=32768) and the
masked long-passage (T=65536) workloads are timed after it as extra lines.
The CPU baseline is the oracle's fp32 instance on a bounded sample of the main
workload, timed on this host's cores; the same sample through the fp64
oracle gives the parity block (near ties, flips, per-tensor errors).
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

import workloads

METRIC = "MoE block fwd+bwd tokens/sec and TFLOP/s (% bf16 MFMA peak), 1 MI355X"
ROOT = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(ROOT, "paper_2608_00916_amd", "csrc")
TRAFFIC = os.path.join(ROOT, "profiles", "hbm_traffic_{}.json")
COPY_TAG = "copy calibration"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def kernel_work(name, T, Tv, H, E, F, k, R):
    """Algorithmic work of one launch of each kernel: (kind, amount).
    FLOP for matrix products, bytes for data-movement kernels."""
    b = 2  # bf16
    return {
        "router_logits": ("flop", 2.0 * T * H * E),
        "gateup_fwd": ("flop", 4.0 * H * F * R),
        "down_fwd": ("flop", 2.0 * H * F * R),
        "down_dgrad_swiglu": ("flop", 2.0 * H * F * R),
        "down_wgrad": ("flop", 2.0 * H * F * R),
        "gateup_dgrad": ("flop", 4.0 * H * F * R),
        "gateup_wgrad": ("flop", 4.0 * H * F * R),
        "dwr_partial": ("flop", 2.0 * Tv * H * E),
        "permute_rows": ("byte", float(Tv * H * b + R * H * b)),
        "combine": ("byte", float(R * H * b + Tv * H * b)),
        "combine_bwd": ("byte", float(Tv * H * b + R * H * b)),
        "router_dx": ("byte", float(R * H * b + Tv * H * b)),
    }.get(name, ("none", 0.0))


def kernel_source_hash():
    """sha256 over the kernel sources: stored counter readings apply only to
    the kernels they were taken from."""
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(CSRC, "*"))):
        h.update(os.path.basename(f).encode())
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def short_kernel_name(name):
    """rocprofv3 kernel name -> the library's trace name."""
    m = re.search(r"k_stream<[^>]*?::(\w+)Jobs", name)
    if m:
        base = {"DownWgrad": "down_wgrad", "GateUpWgrad": "gateup_wgrad", "GateUpFwd": "gateup_fwd",
                "DownFwd": "down_fwd", "DownDgrad": "down_dgrad_swiglu", "GateUpDgrad": "gateup_dgrad",
                "LoraWgrad": "lora_wgrad"}.get(m.group(1), m.group(1))
        # the adapter (rank-r) variants of the row-grouped products
        lora = re.search(r"(?:Fwd|Dgrad)Jobs<(?:[^<>]*<[^<>]*>, )?true>", name) is not None
        return base + ("_lora" if lora else "")
    m = re.search(r"k_(\w+?)(?:<|\(|$)", name)
    if m:
        return m.group(1)
    return name[:40]


def pmc_summary(fetch_dir, write_dir, workload, copy_mib):
    """Turn two rocprofv3 --pmc runs of `bench.py --copy-calibration N` (one
    with FETCH_SIZE, one with WRITE_SIZE, KiB per dispatch) into HBM bytes per
    launch for each library kernel.  Each counter is scaled by the ratio of
    the known bytes of the torch copy kernel (N MiB read, N MiB written) to
    what the counter read for it."""
    def read(d, counter):
        rows = list(csv.DictReader(open(os.path.join(d, "run_counter_collection.csv"))))
        per = {}
        for r in rows:
            if r["Counter_Name"] != counter:
                continue
            per.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return per
    f = read(fetch_dir, "FETCH_SIZE")
    w = read(write_dir, "WRITE_SIZE")
    copy_bytes = copy_mib * 2 ** 20
    # the calibration copy is the dispatch reading about copy_mib MiB outside the library
    cands = [(n, max(v)) for n, v in f.items() if "moe::" not in n]
    cname, cfetch = min(cands, key=lambda x: abs(x[1] * 1024 - copy_bytes))
    cwrite = max(w[cname])
    ff = copy_bytes / (cfetch * 1024)
    wf = copy_bytes / (cwrite * 1024)
    kernels = {}
    for n, v in f.items():
        if "moe::" not in n:
            continue
        kn = short_kernel_name(n)
        fb = sum(v) / len(v) * 1024 * ff
        wb = sum(w.get(n, [0.0])) / max(1, len(w.get(n, []))) * 1024 * wf
        kernels[kn] = {"fetch_bytes": round(fb), "write_bytes": round(wb), "hbm_bytes": round(fb + wb)}
    out = {"workload": workload, "source_hash": kernel_source_hash(), "copy_kernel": cname[:80],
           "copy_bytes": copy_bytes, "fetch_factor": ff, "write_factor": wf, "kernels": kernels}
    path = TRAFFIC.format(workload)
    json.dump(out, open(path, "w"), indent=1)
    print(f"wrote {path}: fetch x{ff:.3f}, write x{wf:.3f}")


def stored_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the stored counter summary, or
    None if there is none or the kernels changed since it was taken."""
    try:
        d = json.load(open(TRAFFIC.format(workload)))
    except (OSError, ValueError):
        return None
    if d.get("source_hash") != kernel_source_hash():
        return None
    k = d.get("kernels", {}).get(kernel)
    return None if k is None else k["hbm_bytes"]


def host_cores():
    """Cores this process may run on (its affinity mask), the host's share."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def cpu_baseline(inp, k, tokens, gpu=None):
    """The CPU baseline leg: the oracle, as it stands, on the first `tokens`
    tokens of the workload.

    Timed: the oracle's fp32 instance (inputs widened to float32), one
    fwd+bwd.  Then, with `gpu` (host copies of the GPU's routing, Y, dX and
    gradients of the timed step), the same sample through the fp64 instance is
    the reference of a parity block: near ties (set / order), tokens whose
    expert set flipped, whether the routing tables are bit-exact, and the
    per-tensor max-relative errors of Y and dX on the sample (forward and dX
    are separable over tokens) and, when the sample is the whole batch, of
    dW_r and every expert's weight gradients."""
    from threadpoolctl import threadpool_info

    from oracle import moe_oracle as O
    names = ("w_r", "w_gate", "w_up", "w_down")
    mask = None if inp["mask"] is None else inp["mask"][:tokens].astype(bool)
    w32 = {n: O.widen_bf16(inp[n], np.float32) for n in names}
    x32 = O.widen_bf16(inp["x"][:tokens], np.float32)
    dy32 = O.widen_bf16(inp["dy"][:tokens], np.float32)
    t0 = time.perf_counter()
    f = O.moe_forward(x32, w32["w_r"], w32["w_gate"], w32["w_up"], w32["w_down"], k, mask)
    O.moe_backward(x32, w32["w_r"], w32["w_gate"], w32["w_up"], w32["w_down"], f, dy32)
    dt = time.perf_counter() - t0
    del w32, x32, dy32, f
    blas = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    T = inp["dims"]["T"]
    out = {"value": tokens / dt, "unit": "tokens/s", "cores": host_cores(), "blas_threads": int(blas),
           "kind": "oracle",
           "sample": f"first {tokens} of {T} tokens of the same workload (all {inp['dims']['E']} experts' "
                     f"weights), one fwd+bwd, the oracle's fp32 instance, {dt:.1f} s"}
    if gpu is None:
        return out, None
    w = {n: O.widen_bf16(inp[n]) for n in names}
    x = O.widen_bf16(inp["x"][:tokens])
    dy = O.widen_bf16(inp["dy"][:tokens])
    f = O.moe_forward(x, w["w_r"], w["w_gate"], w["w_up"], w["w_down"], k, mask)
    b = O.moe_backward(x, w["w_r"], w["w_gate"], w["w_up"], w["w_down"], f, dy)
    return out, parity_block(O, f, b, gpu, k, tokens, T, mask)


def max_rel(got, ref):
    scale = float(np.abs(ref).max())
    d = float(np.abs(np.asarray(got, dtype=np.float64) - ref).max()) if ref.size else 0.0
    return d / scale if scale > 0 else d


def parity_block(O, f, b, gpu, k, tokens, T, mask):
    """Agreement of the timed step's GPU outputs with the fp64 oracle on the
    CPU-baseline sample (the first `tokens` tokens)."""
    E = f["z"].shape[1]
    st, ot = O.near_ties(f["z"], k, gap=1e-4, mask=mask)
    gidx = gpu["topk_idx"][:tokens]
    valid = np.ones(tokens, dtype=bool) if mask is None else mask
    flipped = np.array([set(a) != set(c) for a, c in zip(gidx.tolist(), f["idx"].tolist())]) & valid
    clean = valid & ~st & ~ot
    res = {"reference": "oracle fp64", "tokens": tokens, "tie_gap": 1e-4,
           "near_ties_set": int(st.sum()), "near_ties_order": int(ot.sum()), "flipped": int(flipped.sum()),
           "experts_bit_exact_off_ties": bool(np.array_equal(gidx[clean], f["idx"][clean]))}
    keep = ~flipped
    res["y_max_rel"] = max_rel(gpu["y"][:tokens][keep], f["Y"][keep])
    res["dx_max_rel"] = max_rel(gpu["dx"][:tokens][keep], b["dx"][keep])
    if tokens == T:  # the whole batch: routing tables and weight gradients too
        same = not flipped.any()
        res["counts_offsets_bit_exact"] = bool(same and np.array_equal(gpu["counts"], f["counts"])
                                               and np.array_equal(gpu["offsets"], f["offsets"]))
        res["row_token_bit_exact"] = bool(same and np.array_equal(gpu["row_token"], f["row_token"]))
        touched = np.zeros(E, dtype=bool)
        for t in np.nonzero(flipped)[0]:
            touched[[e for e in list(gidx[t]) + list(f["idx"][t]) if e >= 0]] = True
        cols = ~touched
        res["dw_r_max_rel"] = max_rel(gpu["dw_r"][:, cols], b["dw_r"][:, cols])
        for n in ("dw_gate", "dw_up", "dw_down"):
            res[n + "_max_rel"] = max(max_rel(gpu[n](e), b[n][e]) for e in np.nonzero(cols)[0])
        res["experts_compared"] = int(cols.sum())
    res["within_2e-2"] = all(v <= 2e-2 for n, v in res.items() if n.endswith("_max_rel"))
    return res


def serving_forward(moe, t, tm, T, H, E, F, k, Tv, steps, warmup):
    """The forward-only entry point (moe_infer) on the same batch, timed after
    the fwd+bwd region: tokens/s of the serving pass."""
    import torch
    inf = moe.MoEInfer(T, H, E, F, k, mask=tm is not None)

    def run():
        inf.forward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], tm)

    for _ in range(warmup):
        run()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    print(f"[bench] forward only (moe_infer): {ms:.3f} ms/step", file=sys.stderr, flush=True)
    return {"entry": "moe_infer", "tokens_per_s": Tv / (ms * 1e-3), "ms_per_step": ms, "steps": steps,
            "tflops": 6.0 * H * F * Tv * k / (ms * 1e-3) / 1e12}


def lora_step(moe, t, tm, T, H, E, F, k, Tv, rank, steps, warmup):
    """Forward + backward with rank-r expert adapters (base weights and router
    frozen) on the same batch, timed after the other regions."""
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(7)

    def w(*shape):
        return (0.02 * torch.randn(shape, generator=g, device="cuda")).to(torch.bfloat16)
    ad = dict(a1=w(E, H, rank), b1_gate=w(E, rank, F), b1_up=w(E, rank, F), a2=w(E, F, rank), b2=w(E, rank, H))
    lora = moe.lora_args(rank, 2.0, ad["a1"], ad["b1_gate"], ad["b1_up"], ad["a2"], ad["b2"])
    blk = moe.MoELoRA(T, H, E, F, k, rank, mask=tm is not None)

    def run():
        blk.forward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], lora, tm)
        blk.backward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], lora, t["dy"])

    for _ in range(warmup):
        run()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    print(f"[bench] expert LoRA (rank {rank}) fwd+bwd: {ms:.3f} ms/step", file=sys.stderr, flush=True)
    return {"entry": "moe_lora_fwd + moe_lora_bwd", "rank": rank, "tokens_per_s": Tv / (ms * 1e-3),
            "ms_per_step": ms, "steps": steps}


def ep_share_step(moe, steps, warmup):
    """One expert-parallel rank's share on its own (the ep_share workload: 16
    local experts, the 8359 rows a top-8 router sends them from a T=8192
    batch, already grouped by expert): moe_experts_fwd +
    moe_experts_bwd, timed after the other regions."""
    import torch
    import workloads
    inp = workloads.make("ep_share")
    d = inp["dims"]
    R, H, E, F = d["R"], d["H"], d["E"], d["F"]

    def dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)
    t = {n: dev(inp[n]) for n in ("xp", "w_gate", "w_up", "w_down", "d_o")}
    counts = torch.from_numpy(inp["counts"]).cuda()
    ex = moe.MoEExperts(R, H, E, F)

    def run():
        ex.forward(t["xp"], counts, t["w_gate"], t["w_up"], t["w_down"])
        ex.backward(t["xp"], t["w_gate"], t["w_up"], t["w_down"], t["d_o"])

    for _ in range(warmup):
        run()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    print(f"[bench] EP share (16 local experts, {R} rows) fwd+bwd: {ms:.3f} ms/step", file=sys.stderr, flush=True)
    return {"entry": "moe_experts_fwd + moe_experts_bwd", "workload": "ep_share", "rows": R, "local_experts": E,
            "rows_per_s": R / (ms * 1e-3), "ms_per_step": ms, "steps": steps,
            "tflops": 18.0 * H * F * R / (ms * 1e-3) / 1e12}


GEMM_NAMES = ("gateup_fwd", "down_fwd", "down_dgrad_swiglu", "down_wgrad", "gateup_dgrad", "gateup_wgrad")


def kernel_table(kern, workload, T, Tv, H, E, F, k, R):
    """Per-kernel average launch time and achieved rate, the grouped products'
    fraction of the bf16 peak, and the dominant kernel's roofline."""
    per = {}
    for name, (tot, n) in kern.items():
        avg_ms = tot / n
        kind, amt = kernel_work(name, T, Tv, H, E, F, k, R)
        row = {"avg_us": round(avg_ms * 1e3, 2), "launches": n}
        if kind == "flop":
            row["tflops"] = round(amt / (avg_ms * 1e-3) / 1e12, 1)
        elif kind == "byte":
            row["gbs"] = round(amt / (avg_ms * 1e-3) / 1e9, 1)
        per[name] = row
    out = {"kernels": per}
    gemm_ms = sum(kern[n][0] / kern[n][1] for n in GEMM_NAMES if n in kern)
    out["grouped_gemm_frac_bf16_peak"] = 18.0 * H * F * R / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS
    dom = max(kern, key=lambda n: kern[n][0])
    tot, n = kern[dom]
    avg_s = tot / n * 1e-3
    kind, amt = kernel_work(dom, T, Tv, H, E, F, k, R)
    traffic = stored_traffic(workload, dom)
    if kind == "flop":
        ach = amt / avg_s / 1e12
        out["roofline"] = {"kernel": dom, "bound": "mfma", "achieved": ach, "peak": PEAK_BF16_TFLOPS,
                           "unit": "TFLOP/s", "frac": ach / PEAK_BF16_TFLOPS, "traffic": traffic}
    else:
        ach = amt / avg_s / 1e9
        out["roofline"] = {"kernel": dom, "bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS,
                           "unit": "GB/s", "frac": ach / PEAK_HBM_GBS, "traffic": traffic}
    return out


def time_block(moe, name, steps, warmup, trace, copy_mib=0, keep=False):
    """Times `steps` fwd+bwd steps of block workload `name` after `warmup`
    untimed ones (inputs resident in HBM), then, with `trace`, the same steps
    again with per-launch HIP events.  Returns (result dict, state), state
    holding the inputs and the block when `keep`."""
    import torch
    cfg = workloads.CONFIGS[name]
    inp = workloads.make(name)
    d = inp["dims"]
    T, H, E, F, k = d["T"], d["H"], d["E"], d["F"], d["k"]
    mask_np = inp["mask"]
    Tv = T if mask_np is None else int(mask_np.sum())
    R = Tv * k

    def dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)

    t = {n: dev(inp[n]) for n in ("x", "w_r", "w_gate", "w_up", "w_down", "dy")}
    tm = None if mask_np is None else torch.from_numpy(mask_np.astype(np.uint8)).cuda()
    blk = moe.MoEBlock(T, H, E, F, k, mask=tm is not None)

    if copy_mib:
        n = copy_mib * 2 ** 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    def step(marks=None):
        if marks:
            marks[0].record()
        blk.forward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], tm)
        if marks:
            marks[1].record()
        blk.backward(t["x"], t["w_r"], t["w_gate"], t["w_up"], t["w_down"], t["dy"])
        if marks:
            marks[2].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] {name}: warmup {warmup} done", file=sys.stderr, flush=True)

    # Timed region: exactly `steps` steps, bracketed by synchronisations, with
    # no event inside it (a timing event recorded between launches leaves the
    # GPU idle for ~5 us while the stream processes it).
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record()
    for i in range(steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = ev0.elapsed_time(ev1) / steps
    print(f"[bench] {name}: timed {steps} steps: {ms:.3f} ms/step (wall {1e3 * wall / steps:.3f})",
          file=sys.stderr, flush=True)

    # Split region: the same steps again with three events per step, for the
    # forward / backward split and the per-step spread.
    marks = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    for i in range(steps):
        step(marks[i])
    torch.cuda.synchronize()

    def pct(v):
        q = np.percentile(np.asarray(v), [10, 50, 90])
        return {"p10": round(float(q[0]), 4), "p50": round(float(q[1]), 4), "p90": round(float(q[2]), 4)}
    res = {"ms_per_step": ms, "tokens_per_s": Tv / (ms * 1e-3),
           "config": {"workload": f"{name} MoE block fwd+bwd", "T": T, "T_valid": Tv, "H": H, "E": E,
                      "top_k": k, "F": F, "routed_rows": R, "seed": cfg["seed"]},
           "block_tflops": (18.0 * H * F * R + 6.0 * H * E * Tv) / (ms * 1e-3) / 1e12,
           "timing": {"fwd_ms": pct([m[0].elapsed_time(m[1]) for m in marks]),
                      "bwd_ms": pct([m[1].elapsed_time(m[2]) for m in marks]),
                      "step_ms": pct([m[0].elapsed_time(m[2]) for m in marks])}}
    res["block_frac_bf16_peak"] = res["block_tflops"] / PEAK_BF16_TFLOPS
    if mask_np is not None:
        res["valid_fraction"] = Tv / T

    # Kernel region: the same steps again with the library's per-launch HIP
    # events (recorded on the launch stream around every kernel), for the
    # per-kernel table and the roofline.  The events themselves lengthen a
    # step by a few percent, which is why they stay out of the timed region.
    if trace:
        moe.moe_trace_read()  # drop anything recorded before
        moe.moe_trace_enable(True)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            step()
        e1.record()
        torch.cuda.synchronize()
        moe.moe_trace_enable(False)
        kern = moe.moe_trace_read()
        res["kernel_region_ms_per_step"] = e0.elapsed_time(e1) / steps
        print(f"[bench] {name}: kernel region {res['kernel_region_ms_per_step']:.3f} ms/step with per-kernel "
              f"events", file=sys.stderr, flush=True)
        if kern:
            res.update(kernel_table(kern, name, T, Tv, H, E, F, k, R))
    state = dict(inp=inp, t=t, tm=tm, blk=blk, dims=(T, H, E, F, k, Tv)) if keep else None
    if not keep:
        del t, tm, blk
        torch.cuda.empty_cache()
    return res, state


def gpu_outputs(blk):
    """Host copies of the last step's routing, Y, dX and dW_r; the expert
    weight gradients are copied one expert at a time on demand."""
    def h(t):
        if t.dtype in (__import__("torch").bfloat16, __import__("torch").float32):
            return t.float().cpu().numpy().astype(np.float64)
        return t.cpu().numpy().astype(np.int64)
    v = blk.views
    out = {n: h(v[n]) for n in ("topk_idx", "counts", "offsets", "row_token")}
    out.update(y=h(blk.y), dx=h(blk.dx), dw_r=h(blk.dw_r))
    for n in ("dw_gate", "dw_up", "dw_down"):
        out[n] = (lambda g: (lambda e: h(g[e])))(getattr(blk, n))
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="qwen3_30b_a3b",
                    choices=[n for n, c in workloads.CONFIGS.items() if c["kind"] == "block"])
    ap.add_argument("--cpu-tokens", type=int, default=8192,
                    help="tokens of the oracle's CPU-baseline sample (0 = skip)")
    ap.add_argument("--no-trace", action="store_true",
                    help="skip the kernel region (per-kernel events, roofline)")
    ap.add_argument("--no-forward-only", action="store_true",
                    help="skip the forward-only (moe_infer), expert-LoRA and EP-share timings")
    ap.add_argument("--lora-rank", type=int, default=16, help="rank of the expert-LoRA timing")
    ap.add_argument("--no-ep-share", action="store_true",
                    help="skip the EP-share timing (its expert products have another shape, so a kernel "
                         "trace of the block leaves it out)")
    ap.add_argument("--extra-workloads", default="zipf,long_passage",
                    help="comma-separated block workloads timed after the main one ('' = none)")
    ap.add_argument("--extra-steps", type=int, default=20, help="timed steps of each extra workload")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="run one torch copy of MIB MiB before the steps (counter calibration)")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 --pmc runs into profiles/ and exit")
    args = ap.parse_args()
    if args.pmc_summary:
        pmc_summary(args.pmc_summary[0], args.pmc_summary[1], args.workload, args.copy_calibration)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the block runs on a single MI355X and this build has "
              f"no multi-GPU path (--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2608_00916_amd as moe

    res, st = time_block(moe, args.workload, args.steps, args.warmup, not args.no_trace,
                         copy_mib=args.copy_calibration, keep=True)
    T, H, E, F, k, Tv = st["dims"]
    t, tm = st["t"], st["tm"]
    forward_only = None if args.no_forward_only else serving_forward(moe, t, tm, T, H, E, F, k, Tv, args.steps,
                                                                     args.warmup)
    lora = None if args.no_forward_only else lora_step(moe, t, tm, T, H, E, F, k, Tv, args.lora_rank,
                                                       args.steps, args.warmup)
    out = {
        "metric": METRIC,
        "value": res["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": res["config"],
    }
    for n in ("block_tflops", "block_frac_bf16_peak", "valid_fraction", "timing", "kernel_region_ms_per_step",
              "kernels", "grouped_gemm_frac_bf16_peak", "roofline"):
        if n in res:
            out[n] = res[n]
    out["forward_only"] = forward_only
    out["expert_lora"] = lora
    gpu = gpu_outputs(st["blk"]) if args.cpu_tokens > 0 else None
    inp = st["inp"]
    del st, t, tm
    torch.cuda.empty_cache()
    out["ep_share"] = None if (args.no_forward_only or args.no_ep_share) else ep_share_step(moe, args.steps,
                                                                                             args.warmup)
    extra = {}
    for name in [n for n in args.extra_workloads.split(",") if n and n != args.workload]:
        r, _ = time_block(moe, name, args.extra_steps, min(args.warmup, 5), not args.no_trace)
        extra[name] = {n: r[n] for n in ("ms_per_step", "tokens_per_s", "config", "block_tflops",
                                         "block_frac_bf16_peak", "valid_fraction", "grouped_gemm_frac_bf16_peak",
                                         "roofline", "kernels") if n in r}
        extra[name]["steps"] = args.extra_steps
    if extra:
        out["extra_workloads"] = extra
    if args.cpu_tokens > 0:
        print(f"[bench] CPU baseline: oracle on {args.cpu_tokens} tokens", file=sys.stderr, flush=True)
        out["cpu_baseline"], out["parity"] = cpu_baseline(inp, k, min(args.cpu_tokens, T), gpu)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
