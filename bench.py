#!/usr/bin/env python3
"""Throughput of the AFNO spectral filter on one MI355X, as one JSON line.

A step is one full filter call (operand preparation, W-axis forward transform, column
kernel with the H transforms and the block MLP, W-axis inverse transform + residual) on the
90 x 180 x 768 bf16 workload with B = 4 (8 blocks of 96; synthetic N(0,1) fields
scaled per channel by U(0.5, 2), complex weights N(0, 0.02^2), lambda 0.01, keep 1),
with inputs resident in HBM.  value = samples per second = B / (time per step), measured
after the GPU's clocks have settled (an untimed 0.3 s run of the filter before the W
counted warm-up steps).

Alongside: the median, p10 and p90 of single calls (a second run of the same steps with
one event between calls), per-kernel HIP-event times on the launch stream over a third run
(the headline timing records no events between its steps),
the roofline of the dominant kernel (algorithmic bytes or FLOPs per launch divided by
its mean launch time), measured HBM traffic from stored rocprofv3 counters when they
belong to the current kernel sources, the backward pass on the same workload (dx and the
parameter gradients for an upstream gradient), one AFNO block on the same workload (LayerNorm,
filter, LayerNorm, channel MLP C -> 4C -> C), the 100-member ensemble workload, the other
workloads' throughput, and the float64 CPU oracle timed on a bounded sample on the host
cores.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-backward] [--no-block]
                    [--no-ensemble] [--no-cpu-baseline] [--no-others]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0      # dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3       # fp32 matrix
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_afno90x180_c768_nb8_bf16_b4.json")
PREWARM_S = 0.3                # untimed sustained run before the counted warm-up (clock ramp)
# timed after the headline for context: fp32 at the headline grid, the 180 x 360 grid with 8
# blocks of 128, the paper's own 180 x 360 filter with 32 blocks of 32, and the headline grid
# with 192 hidden units per block of 96 (hidden-size factor 2)
OTHER_WORKLOADS = ("afno90x180_c768_nb8_fp32", "afno180x360_c1024_nb8_bf16",
                   "afno180x360_c1024_nb32_bf16", "afno90x180_c768_nb8_hs192_bf16_b4")
# the five workloads whose oracle time per sample the CPU baseline reports
CPU_CONFIGS = ("afno16x32_c64_nb4_fp32", "afno90x180_c768_nb8_fp32", "afno90x180_c768_nb8_bf16_b4",
               "afno180x360_c1024_nb8_bf16", "afno90x180_c768_nb8_bf16_ens100_keep0.5")
# how the column kernel evaluates the H-axis DFTs of the headline workload: matrix-core
# products (bf16 operands, fp32 accumulation) against a DFT table whose entries are rounded to
# bf16 with the rounding error carried down each column
H_TRANSFORM = "matrix-core DFT, bf16 table with error-carrying rounding, fp32 accumulation"
H_TRANSFORM_VALU = "vector-ALU FFT, fp32 arithmetic (bf16 storage between passes)"
# HBM traffic measured with rocprofv3 FETCH_SIZE / WRITE_SIZE, per launch, keyed by the
# sha256 of the kernel sources it was measured on (null once the kernels change)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2208_05419_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def algorithmic_work(wl, es: int):
    """Per-launch algorithmic bytes and FLOPs of each kernel (minimum traffic of each
    standalone pass: read its input once, write its output once)."""
    B, H, W, C, bs, hs = wl.B, wl.H, wl.W, wl.C, wl.bs, wl.hs
    kept_h = int((H // 2 + 1) * wl.keep)
    kw = int((W // 2 + 1) * wl.keep)
    rows_kept = sum(1 for r in range(H) if abs(r if r <= H // 2 else r - H) < kept_h)
    x_bytes = B * H * W * C * es
    s_bytes = B * H * kw * C * 2 * es           # spectrum workspace, complex in dtype
    flops = 16 * C * hs * B * rows_kept * kw     # two complex GEMMs, 8 real FLOP per complex MAC
    nb = wl.num_blocks
    w_bytes = 2 * nb * bs * hs * 2 * es          # w1, w2 read
    frag_bytes = nb * 2 * (2 * bs) ** 2 * es     # both layers real-ified, fragment order
    hp = 32 if H <= 32 else (64 if H <= 64 else 96)
    tab_bytes = 2 * hp * hp * 2 if es == 2 and H <= 96 else 0  # bf16 DFT table
    return {
        "prep": {"bytes": w_bytes + frag_bytes + tab_bytes, "flops": 0},
        "row_r2c": {"bytes": x_bytes + s_bytes, "flops": 0},
        "column": {"bytes": 2 * s_bytes, "flops": flops},
        "row_c2r": {"bytes": s_bytes + 2 * x_bytes, "flops": 0},
    }


def time_workload(wl, steps: int, warmup: int, seed: int = 0):
    import numpy as np
    import torch

    import paper_2208_05419_amd as afno
    from paper_2208_05419_amd import synth

    def dev(a):
        if wl.dtype == "fp32":
            return torch.from_numpy(np.ascontiguousarray(a)).cuda()
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    x = dev(synth.make_x(wl, seed=seed))
    w = {k: dev(v) for k, v in synth.make_weights(wl, seed=seed).items()}
    out = torch.empty_like(x)
    stream = torch.cuda.current_stream()

    def step():
        afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam, wl.keep,
                            out=out, stream=stream)

    # the GPU's clocks ramp up over tens of milliseconds of sustained work: run the filter for
    # at least PREWARM_S seconds (untimed) before the counted warm-up steps
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < PREWARM_S:
        for _ in range(10):
            step()
        torch.cuda.synchronize()
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    # the timed steps: one event pair around all of them, nothing recorded in between
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record(stream)
    for _ in range(steps):
        step()
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    # per-call distribution: the same steps again, one event between consecutive calls
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    evs[0].record(stream)
    for i in range(steps):
        step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    per_call = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(steps))
    pick = lambda q: per_call[min(steps - 1, int(q * steps))]  # noqa: E731
    dist = {"median": round(pick(0.5), 5), "p10": round(pick(0.1), 5), "p90": round(pick(0.9), 5)}
    # the per-kernel breakdown: the same steps again with the library's per-phase events
    afno.profile_begin(steps)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    kernel_ms, calls = afno.profile_end()
    del x, w, out
    torch.cuda.empty_cache()
    return total_ms / steps, {k: v / max(calls, 1) for k, v in kernel_ms.items()}, calls, dist


def time_backward(wl, steps: int, warmup: int, seed: int = 0):
    """Mean time of one backward call (dx and the four parameter gradients for an upstream
    gradient g) with inputs resident in HBM; one event pair around all timed calls."""
    import numpy as np
    import torch

    import paper_2208_05419_amd as afno
    from paper_2208_05419_amd import synth

    def dev(a):
        if wl.dtype == "fp32":
            return torch.from_numpy(np.ascontiguousarray(a)).cuda()
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    x = dev(synth.make_x(wl, seed=seed))
    w = {k: dev(v) for k, v in synth.make_weights(wl, seed=seed).items()}
    g = dev(synth.quantize(np.random.default_rng(1000 + seed).standard_normal(x.shape), wl.dtype))
    stream = torch.cuda.current_stream()

    def step():
        afno.filter_backward(x, w["w1"], w["b1"], w["w2"], w["b2"], g, wl.num_blocks, wl.lam,
                             wl.keep, stream=stream)

    t0 = time.perf_counter()
    while time.perf_counter() - t0 < PREWARM_S:
        for _ in range(5):
            step()
        torch.cuda.synchronize()
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record(stream)
    for _ in range(steps):
        step()
    t_end.record(stream)
    torch.cuda.synchronize()
    ms = t_start.elapsed_time(t_end) / steps
    es = 2 if wl.dtype == "bf16" else 4
    io_bytes = 3 * wl.B * wl.H * wl.W * wl.C * es   # read x and g, write dx: any backward's floor
    del x, w, g
    torch.cuda.empty_cache()
    return {"workload": wl.name, "samples_per_s": round(wl.B / (ms * 1e-3), 2),
            "ms_per_step": round(ms, 5), "io_bytes": io_bytes,
            "io_GB_s": round(io_bytes / (ms * 1e-3) / 1e9, 1)}


def time_block(wl, steps: int, warmup: int, seed: int = 0):
    """Mean time of one AFNO block (LayerNorm, filter, LayerNorm, channel MLP C -> 4C -> C,
    residuals) with inputs resident in HBM; one event pair around all timed calls."""
    import numpy as np
    import torch

    import paper_2208_05419_amd as afno
    from paper_2208_05419_amd import synth

    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    x = dev(synth.make_x(wl, seed=seed))
    p = {k: dev(v) for k, v in synth.make_block_params(wl, seed=seed).items()}
    out = torch.empty_like(x)
    stream = torch.cuda.current_stream()

    def step():
        afno.block_forward(x, p, wl.num_blocks, wl.lam, wl.keep, out=out, stream=stream)

    t0 = time.perf_counter()
    while time.perf_counter() - t0 < PREWARM_S:
        for _ in range(5):
            step()
        torch.cuda.synchronize()
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record(stream)
    for _ in range(steps):
        step()
    t_end.record(stream)
    torch.cuda.synchronize()
    ms = t_start.elapsed_time(t_end) / steps
    M = wl.B * wl.H * wl.W
    mlp_flops = 16 * M * wl.C * wl.C   # two GEMMs M x C x 4C, 2 FLOP per MAC
    del x, p, out
    torch.cuda.empty_cache()
    return {"workload": wl.name, "samples_per_s": round(wl.B / (ms * 1e-3), 2),
            "ms_per_step": round(ms, 5), "mlp_flops": mlp_flops}


def roofline(wl, kern_ms: dict, es: int):
    work = algorithmic_work(wl, es)
    if kern_ms.get("prep", 0.0) < 5e-4:
        # the preparation ran inside the W-axis forward launch: its bytes belong to that phase
        work["row_r2c"]["bytes"] += work["prep"]["bytes"]
        work["prep"]["bytes"] = 0
    per = {}
    for k, ms in kern_ms.items():
        s = ms * 1e-3
        if k == "prep" and not work[k]["bytes"]:
            per[k] = {"ms": round(ms, 5), "folded_into": "row_r2c"}
            continue
        gbs = work[k]["bytes"] / s / 1e9 if s > 0 else 0.0
        tfl = work[k]["flops"] / s / 1e12 if s > 0 else 0.0
        per[k] = {"ms": round(ms, 5), "bytes": work[k]["bytes"], "flops": work[k]["flops"],
                  "GB_s": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}
        if work[k]["flops"]:
            peak = BF16_PEAK_TFLOPS if es == 2 else FP32_PEAK_TFLOPS
            per[k]["TFLOP_s"] = round(tfl, 2)
            per[k]["mfma_frac"] = round(tfl / peak, 4)
    dom = max((k for k in kern_ms if k != "prep"), key=lambda k: kern_ms[k])
    d = per[dom]
    peak_tf = BF16_PEAK_TFLOPS if es == 2 else FP32_PEAK_TFLOPS
    # roofline bound of the dominant kernel: the larger of its two lower-bound times
    t_hbm = work[dom]["bytes"] / (HBM_PEAK_GBS * 1e9)
    t_mma = work[dom]["flops"] / (peak_tf * 1e12)
    if t_mma > t_hbm:
        roof = {"bound": "mfma", "achieved": d["TFLOP_s"], "peak": peak_tf, "unit": "TFLOP/s",
                "frac": d["mfma_frac"]}
    else:
        roof = {"bound": "hbm", "achieved": d["GB_s"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": d["hbm_frac"]}
    roof["kernel"] = dom
    roof["traffic"] = None
    try:
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        if tr.get("source_sha256") == kernel_source_hash() and dom in tr.get("kernels", {}):
            roof["traffic"] = tr["kernels"][dom]["hbm_bytes_per_launch"]
    except (OSError, ValueError, KeyError):
        pass
    return roof, per


def cpu_baseline(wl, min_seconds: float):
    """The float64 oracle on the workload's samples, one sample per call, repeated until
    at least min_seconds of wall time have passed; then one sample of each of the other four
    workloads alone (per_config: wall seconds per sample and samples/s)."""
    import oracle
    from paper_2208_05419_amd import synth

    def one(w_, x_, b):
        oracle.filter_forward(x_[b:b + 1], w_["w1"], w_["b1"], w_["w2"], w_["b2"],
                              w_["nb"], w_["lam"], w_["keep"])

    def inputs(wl_, members=None):
        x_ = synth.widen(synth.make_x(wl_, members=members), wl_.dtype)
        w_ = {k: synth.widen(v, wl_.dtype) for k, v in synth.make_weights(wl_).items()}
        w_.update(nb=wl_.num_blocks, lam=wl_.lam, keep=wl_.keep)
        return x_, w_

    x, w = inputs(wl)
    done = 0
    t0 = time.perf_counter()
    while True:
        one(w, x, done % wl.B)
        done += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    per_config = {wl.name: {"sample_s": round(dt / done, 4), "samples_per_s": round(done / dt, 4),
                            "timed": f"{done} samples"}}
    for name in CPU_CONFIGS:
        if name == wl.name:
            continue
        c = synth.WORKLOADS[name]
        xc, wc = inputs(c, members=[0] if c.x_kind == "ensemble" else None)
        note = "sample 0" if c.x_kind != "ensemble" else "member 0"
        t1 = time.perf_counter()
        one(wc, xc, 0)
        s = time.perf_counter() - t1
        per_config[name] = {"sample_s": round(s, 4), "samples_per_s": round(1.0 / s, 4),
                            "timed": note}
    return {"value": round(done / dt, 4), "unit": "samples/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{done} single-sample calls cycling over the {wl.B} samples of {wl.name} "
                      f"(float64 direct DFT, {dt:.1f} s wall); per_config: the oracle's time per sample "
                      f"of each of the five workloads",
            "per_config": per_config}


def calibration_copy(mib: int):
    """One device-to-device copy of exactly mib MiB (a plain copy kernel of known size that
    hardware-counter runs use to scale FETCH_SIZE and WRITE_SIZE)."""
    import torch

    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-ensemble", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-others", action="store_true", help="skip the other workloads' timings")
    ap.add_argument("--no-backward", action="store_true", help="skip the backward-pass timing")
    ap.add_argument("--no-block", action="store_true", help="skip the AFNO-block timing")
    ap.add_argument("--block-only", action="store_true",
                    help="time only the AFNO block (one JSON object; for kernel traces)")
    ap.add_argument("--backward-only", action="store_true",
                    help="time only the backward pass (one JSON object; for kernel traces)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MiB",
                    help="run one plain copy of this many MiB first (for counter scaling)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this filter runs on one GPU; --gpus must be 1 (no multi-GPU path)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2208_05419_amd as afno
    from paper_2208_05419_amd import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    afno.load_library()
    if args.calibrate_copy:
        calibration_copy(args.calibrate_copy)
    wl = synth.WORKLOADS[synth.HEADLINE]
    es = 2 if wl.dtype == "bf16" else 4
    if args.backward_only:
        print(json.dumps({"backward": time_backward(wl, args.steps, args.warmup)}), flush=True)
        return
    if args.block_only:
        print(json.dumps({"block": time_block(wl, args.steps, args.warmup)}), flush=True)
        return
    ms, kern_ms, calls, dist = time_workload(wl, args.steps, args.warmup)
    roof, per_kernel = roofline(wl, kern_ms, es)
    value = wl.B / (ms * 1e-3)
    line = {
        "metric": "AFNO-filter samples/s @90x180x768 bf16",
        "value": round(value, 2),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "B": wl.B, "H": wl.H, "W": wl.W, "C": wl.C,
                   "num_blocks": wl.num_blocks, "lambda": wl.lam, "keep_fraction": wl.keep,
                   "h_transform": H_TRANSFORM},
        "roofline": roof,
        "kernels": per_kernel,
        "timed_calls": calls,
        "call_ms": dist,
    }
    if not args.no_others:
        # the same workload with the H transforms as vector-ALU FFTs in fp32 arithmetic (the
        # precision of the paper's own FFTs), for comparison with the matrix-core table
        afno.set_kernel_path(afno.AFNO_PATH_VALU_DFT)
        try:
            v_ms, v_kern, _, _ = time_workload(wl, args.steps, max(args.warmup // 2, 3))
        finally:
            afno.set_kernel_path(afno.AFNO_PATH_AUTO)
        _, v_per = roofline(wl, v_kern, es)
        line["h_transform_valu_fft"] = {
            "h_transform": H_TRANSFORM_VALU, "samples_per_s": round(wl.B / (v_ms * 1e-3), 2),
            "ms_per_step": round(v_ms, 5), "kernel_ms": {k: v["ms"] for k, v in v_per.items()}}
    if not args.no_backward:
        line["backward"] = time_backward(wl, max(args.steps // 2, 10), max(args.warmup // 2, 3))
    if not args.no_block:
        line["block"] = time_block(wl, max(args.steps // 2, 10), max(args.warmup // 2, 3))
    if not args.no_ensemble:
        ens = synth.WORKLOADS["afno90x180_c768_nb8_bf16_ens100_keep0.5"]
        e_ms, e_kern, _, e_dist = time_workload(ens, max(args.steps // 5, 5), max(args.warmup // 5, 3))
        e_roof, e_per = roofline(ens, e_kern, 2)
        e_roof["traffic"] = None
        line["ensemble"] = {"workload": ens.name, "samples_per_s": round(ens.B / (e_ms * 1e-3), 2),
                            "ms_per_step": round(e_ms, 4), "call_ms": e_dist, "kernels": e_per,
                            "roofline": e_roof}
    if not args.no_others:
        # the remaining workloads: samples/s and per-kernel times (context; not the headline)
        others = {}
        for name in OTHER_WORKLOADS:
            o = synth.WORKLOADS[name]
            o_es = 2 if o.dtype == "bf16" else 4
            o_ms, o_kern, _, _ = time_workload(o, max(args.steps, 100), max(args.warmup // 5, 3))
            _, o_per = roofline(o, o_kern, o_es)
            others[name] = {"samples_per_s": round(o.B / (o_ms * 1e-3), 2), "ms_per_step": round(o_ms, 4),
                            "kernel_ms": {k: v["ms"] for k, v in o_per.items()}}
        line["other_workloads"] = others
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
