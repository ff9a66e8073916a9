#!/usr/bin/env python3
"""Throughput of the MoE block, forward + backward, on one MI355X.

One step = moe_fwd + moe_bwd over one batch of the workload (router, top-k,
permutation, SwiGLU expert products, combine, and the whole backward), inputs
resident in HBM before the timed region.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload qwen3_30b_a3b]

The workload defaults to the Qwen3-30B-A3B-shaped layer on one GPU (T=8192
tokens, H=2048, E=128 experts, top-8, F=768, bf16).  The dominant kernel's
roofline comes from HIP events recorded around every library kernel launch
over the timed region; the CPU baseline is the fp64 oracle on a bounded
sample of the same workload, timed on this host's cores.
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


def cpu_baseline(inp, k, tokens):
    """The fp64 oracle, as it stands, on the first `tokens` tokens."""
    from threadpoolctl import threadpool_info

    from oracle import moe_oracle as O
    w = {n: O.widen_bf16(inp[n]) for n in ("w_r", "w_gate", "w_up", "w_down")}
    x = O.widen_bf16(inp["x"][:tokens])
    dy = O.widen_bf16(inp["dy"][:tokens])
    mask = None if inp["mask"] is None else inp["mask"][:tokens].astype(bool)
    t0 = time.perf_counter()
    f = O.moe_forward(x, w["w_r"], w["w_gate"], w["w_up"], w["w_down"], k, mask)
    O.moe_backward(x, w["w_r"], w["w_gate"], w["w_up"], w["w_down"], f, dy)
    dt = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {"value": tokens / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"first {tokens} of {inp['dims']['T']} tokens of the same workload "
                      f"(all {inp['dims']['E']} experts' weights), one fwd+bwd, fp64, "
                      f"{dt:.1f} s"}


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
    local experts, 8192 rows already grouped by expert): moe_experts_fwd +
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

    cfg = workloads.CONFIGS[args.workload]
    inp = workloads.make(args.workload)
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

    if args.copy_calibration:
        n = args.copy_calibration * 2 ** 20
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

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] {args.workload}: warmup {args.warmup} done", file=sys.stderr, flush=True)

    # Timed region: exactly K steps, bracketed by synchronisations, without
    # per-kernel events (three events per step give the fwd/bwd split).
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    marks = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record()
    for i in range(args.steps):
        step(marks[i])
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = ev0.elapsed_time(ev1) / args.steps
    print(f"[bench] timed {args.steps} steps: {ms:.3f} ms/step (wall {1e3 * wall / args.steps:.3f})",
          file=sys.stderr, flush=True)

    # Kernel region: the same K steps again with the library's per-launch HIP
    # events (recorded on the launch stream around every kernel), for the
    # per-kernel table and the roofline.  The events themselves lengthen a
    # step by a few percent, which is why they stay out of the timed region.
    kern = {}
    traced_ms = None
    if not args.no_trace:
        moe.moe_trace_read()  # drop anything recorded before
        moe.moe_trace_enable(True)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(args.steps):
            step()
        e1.record()
        torch.cuda.synchronize()
        moe.moe_trace_enable(False)
        kern = moe.moe_trace_read()
        traced_ms = e0.elapsed_time(e1) / args.steps
        print(f"[bench] kernel region: {traced_ms:.3f} ms/step with per-kernel events", file=sys.stderr,
              flush=True)

    def pct(v):
        q = np.percentile(np.asarray(v), [10, 50, 90])
        return {"p10": round(float(q[0]), 4), "p50": round(float(q[1]), 4), "p90": round(float(q[2]), 4)}
    timing = {"fwd_ms": pct([m[0].elapsed_time(m[1]) for m in marks]),
              "bwd_ms": pct([m[1].elapsed_time(m[2]) for m in marks]),
              "step_ms": pct([m[0].elapsed_time(m[2]) for m in marks])}
    forward_only = None if args.no_forward_only else serving_forward(moe, t, tm, T, H, E, F, k, Tv, args.steps,
                                                                     args.warmup)
    lora = None if args.no_forward_only else lora_step(moe, t, tm, T, H, E, F, k, Tv, args.lora_rank,
                                                       args.steps, args.warmup)
    ep = None if (args.no_forward_only or args.no_ep_share) else ep_share_step(moe, args.steps, args.warmup)

    gemm_flop = 18.0 * H * F * R
    router_flop = 6.0 * H * E * Tv
    tflops = (gemm_flop + router_flop) / (ms * 1e-3) / 1e12
    out = {
        "metric": METRIC,
        "value": Tv / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.workload} MoE block fwd+bwd", "T": T, "T_valid": Tv, "H": H,
                   "E": E, "top_k": k, "F": F, "routed_rows": R, "seed": cfg["seed"]},
        "block_tflops": tflops,
        "block_frac_bf16_peak": tflops / PEAK_BF16_TFLOPS,
        "timing": timing,
        "forward_only": forward_only,
        "expert_lora": lora,
        "ep_share": ep,
    }
    if traced_ms is not None:
        out["kernel_region_ms_per_step"] = traced_ms
    if kern:
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
        out["kernels"] = per
        gemm_names = ("gateup_fwd", "down_fwd", "down_dgrad_swiglu", "down_wgrad", "gateup_dgrad",
                      "gateup_wgrad")
        gemm_ms = sum(kern[n][0] / kern[n][1] for n in gemm_names if n in kern)
        out["grouped_gemm_frac_bf16_peak"] = gemm_flop / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS
        dom = max(kern, key=lambda n: kern[n][0])
        tot, n = kern[dom]
        avg_s = tot / n * 1e-3
        kind, amt = kernel_work(dom, T, Tv, H, E, F, k, R)
        traffic = stored_traffic(args.workload, dom)
        if kind == "flop":
            ach = amt / avg_s / 1e12
            out["roofline"] = {"kernel": dom, "bound": "mfma", "achieved": ach, "peak": PEAK_BF16_TFLOPS,
                               "unit": "TFLOP/s", "frac": ach / PEAK_BF16_TFLOPS, "traffic": traffic}
        else:
            ach = amt / avg_s / 1e9
            out["roofline"] = {"kernel": dom, "bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS,
                               "unit": "GB/s", "frac": ach / PEAK_HBM_GBS, "traffic": traffic}
    if args.cpu_tokens > 0:
        print(f"[bench] CPU baseline: oracle on {args.cpu_tokens} tokens", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(inp, k, min(args.cpu_tokens, T))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
