"""Host logic of bench.py (no GPU): kernel-name mapping of the rocprofv3
summaries, the copy-kernel calibration of the HBM counters, and the
source-hash guard on stored traffic."""
import csv
import json
import os

import pytest

import bench

NS = "moe::(anonymous namespace)::"


@pytest.mark.parametrize("name,short", [
    (f"void {NS}k_stream<{NS}GateUpFwdJobs<false>, true, false>({NS}GateUpFwdJobs<false>)", "gateup_fwd"),
    (f"void {NS}k_stream<{NS}GateUpFwdJobs<true>, true, false>(x)", "gateup_fwd_lora"),
    (f"void {NS}k_stream<{NS}DownFwdJobs<moe::Tile<128, 256, 1, 2, 4>, false>, true, false>(x)", "down_fwd"),
    (f"void {NS}k_stream<{NS}DownDgradJobs<moe::Tile<128, 256, 1, 2, 4>, true>, true, true>(x)",
     "down_dgrad_swiglu_lora"),
    (f"void {NS}k_stream<{NS}GateUpDgradJobs<moe::Tile<128, 256, 1, 2, 4>, false>, true, true>(x)", "gateup_dgrad"),
    (f"void {NS}k_stream<{NS}GateUpWgradJobs<moe::Tile<128, 256, 2, 2, 4>, false>, false, false>(x)",
     "gateup_wgrad"),
    (f"void {NS}k_stream<{NS}DownWgradJobs<moe::Tile<128, 256, 1, 2, 4>, true>, false, false>(x)", "down_wgrad"),
    (f"void {NS}k_stream<{NS}LoraWgradJobs<false>, false, false>(x)", "lora_wgrad"),
    (f"void {NS}k_gateup_fwd_rows(unsigned short const*)", "gateup_fwd_rows"),
    (f"void {NS}k_topk<2, false>(float const*)", "topk"),
    (f"void {NS}k_permute_rows<8>(unsigned short const*)", "permute_rows"),
])
def test_short_kernel_name(name, short):
    assert bench.short_kernel_name(name) == short


def _write_counters(path, counter, rows):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, value in rows:
            w.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": value})


def test_pmc_summary_scales_by_the_copy_calibration(tmp_path, monkeypatch):
    """A 1 MiB copy read as 512 KiB by FETCH_SIZE and 1024 KiB by WRITE_SIZE
    gives scales 2 and 1; a library kernel's readings (two dispatches) are
    averaged and scaled by them."""
    copy = "__amd_rocclr_copyBuffer"
    k = f"void {NS}k_combine<8>(unsigned short const*)"
    _write_counters(tmp_path / "fetch", "FETCH_SIZE", [(copy, 512.0), (k, 100.0), (k, 300.0)])
    _write_counters(tmp_path / "write", "WRITE_SIZE", [(copy, 1024.0), (k, 50.0), (k, 50.0)])
    out = tmp_path / "traffic_{}.json"
    monkeypatch.setattr(bench, "TRAFFIC", str(out))
    bench.pmc_summary(str(tmp_path / "fetch"), str(tmp_path / "write"), "w", 1)
    d = json.load(open(str(out).format("w")))
    assert d["fetch_factor"] == pytest.approx(2.0)
    assert d["write_factor"] == pytest.approx(1.0)
    c = d["kernels"]["combine"]
    assert c["fetch_bytes"] == 200 * 1024 * 2
    assert c["write_bytes"] == 50 * 1024
    assert c["hbm_bytes"] == c["fetch_bytes"] + c["write_bytes"]
    # the stored summary applies only to the kernel sources it was taken from
    assert bench.stored_traffic("w", "combine") == c["hbm_bytes"]
    d["source_hash"] = "0" * 16
    json.dump(d, open(str(out).format("w"), "w"))
    assert bench.stored_traffic("w", "combine") is None


def test_kernel_work_units():
    """Matrix products count flops (2 per multiply-add), data movement bytes."""
    T, Tv, H, E, F, k = 8192, 8192, 2048, 128, 768, 8
    R = Tv * k
    assert bench.kernel_work("gateup_fwd", T, Tv, H, E, F, k, R) == ("flop", 4.0 * H * F * R)
    assert bench.kernel_work("down_wgrad", T, Tv, H, E, F, k, R) == ("flop", 2.0 * H * F * R)
    assert bench.kernel_work("combine", T, Tv, H, E, F, k, R) == ("byte", float(R * H * 2 + Tv * H * 2))
    assert bench.kernel_work("topk", T, Tv, H, E, F, k, R)[0] == "none"


def test_cpu_baseline_leg_and_parity_block():
    """The CPU-baseline leg times the oracle's fp32 instance and reports the
    affinity cores; its parity block compares GPU-shaped outputs with the fp64
    oracle (here outputs built from the oracle itself, so every error is 0
    except for bf16 rounding, and a flipped token is detected and left out)."""
    import numpy as np

    import bench
    import workloads
    from oracle import moe_oracle as O
    inp = workloads.make("tiny")
    d = inp["dims"]
    w = {n: O.widen_bf16(inp[n]) for n in ("x", "w_r", "w_gate", "w_up", "w_down", "dy")}
    f = O.moe_forward(w["x"], w["w_r"], w["w_gate"], w["w_up"], w["w_down"], d["k"])
    b = O.moe_backward(w["x"], w["w_r"], w["w_gate"], w["w_up"], w["w_down"], f, w["dy"])
    idx = f["idx"].copy()
    t_flip = 5
    idx[t_flip] = [e for e in range(d["E"]) if e not in idx[t_flip]][:d["k"]]
    gpu = dict(topk_idx=idx, counts=f["counts"], offsets=f["offsets"], row_token=f["row_token"],
               y=f["Y"], dx=b["dx"], dw_r=b["dw_r"])
    for n in ("dw_gate", "dw_up", "dw_down"):
        gpu[n] = (lambda a: (lambda e: a[e]))(b[n])
    base, par = bench.cpu_baseline(inp, d["k"], d["T"], gpu)
    assert base["kind"] == "oracle" and base["cores"] >= 1 and base["value"] > 0
    assert "fp32" in base["sample"]
    assert par["flipped"] == 1 and not par["counts_offsets_bit_exact"]
    assert par["experts_compared"] == d["E"] - len(set(idx[t_flip]) | set(f["idx"][t_flip]))
    assert par["y_max_rel"] == 0 and par["dx_max_rel"] == 0 and par["dw_r_max_rel"] == 0
    assert par["within_2e-2"]
