#!/usr/bin/env python3
"""Benchmark: one decode token's GEMV sweep of Llama-2 110M on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
every weight matrix of a Llama-2 110M decode step (12 layers x wq, wk, wv, wo
[768x768], w1, w3 [2048x768], w2 [768x2048], plus the 32000x768 classifier;
85 fp32 GEMVs, 438,874,112 algorithmic bytes) computed by ONE launch of the
grouped sweep kernel (a plan run).  The weights, the 85 x vectors and the 85
y buffers are resident in HBM before timing starts.

Two copies of the weights (877 MB together) are alternated step by step, so
the 256 MB last-level cache cannot hand one sweep's weights to the next: the
figure is HBM streaming.  ``--warm`` times a single copy instead (reported as
context only).

Prints ONE JSON line (rank 0) with the metric, a roofline object for the
sweep kernel and the CPU oracle's throughput on the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_GBS = 8000.0  # MI355X HBM3E, decimal GB/s
METRIC = "achieved HBM GB/s (% of peak) + µs per full-model GEMV sweep (tok/s equiv)"
WORKLOAD = "sweep110m"
TRAFFIC_JSON = os.path.join(ROOT, "profiles", "sweep110m_fp32_traffic.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2601_03324_amd", "csrc", "tvl_kernels.hip")


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def kernel_hash() -> str:
    return hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()[:16]


def measured_traffic(algo_bytes: int):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when there is none or the kernel source changed since it was taken."""
    try:
        t = json.load(open(TRAFFIC_JSON))
    except (OSError, ValueError):
        return None
    if t.get("kernel_src_sha256_16") != kernel_hash():
        return None
    return t.get("bytes_per_launch")


def cpu_baseline(wl, hosts, seconds: float) -> dict:
    """The oracle as it stands (single-threaded naive double GEMV) over whole
    110M sweeps on this host, for about ``seconds`` of CPU time."""
    import oracle
    xs = [m.x() for m in wl.mats]
    t0 = time.perf_counter()
    reps = 0
    while True:
        for m, W, x in zip(wl.mats, hosts, xs):
            oracle.gemv_f32(W, x)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    gbs = wl.algo_bytes() * reps / el / 1e9
    return {"value": round(gbs, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{reps} full 110M sweeps (85 fp32 GEMVs, double accumulation) in "
                      f"{el:.1f} s on one host thread ({platform.processor() or platform.machine()}"
                      f"); {el / reps * 1e6:.0f} us per sweep"}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--warm", action="store_true", help="time one weight copy (cache-warm)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--rows-per-wave", type=int, default=0)
    ap.add_argument("--waves-per-block", type=int, default=0)
    ap.add_argument("--unroll", type=int, default=0)
    ap.add_argument("--grid", type=int, default=0)
    ap.add_argument("--x-mode", choices=("auto", "lds", "direct"), default="auto",
                    help="how wavefronts get x (default: the library's choice)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="run one plain copy of this many MiB before timing (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the GEMV sweep runs on a single MI355X; "
              "--gpus N > 1 is not supported", file=sys.stderr)
        return 2

    import numpy as np
    import torch
    import synth
    import synth.device as sdev
    from paper_2601_03324_amd import tvl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    torch.cuda.set_device(0)
    wl = synth.WORKLOADS[WORKLOAD]
    algo = wl.algo_bytes()

    log(f"generating {wl.name}: {len(wl.mats)} GEMVs, {wl.weight_bytes() / 1e6:.1f} MB of weights")
    hosts = [m.weights() for m in wl.mats]
    gemvs_a = []
    for m, W in zip(wl.mats, hosts):
        Wd = tvl.upload_matrix(W, 0, "cuda")
        x = torch.from_numpy(m.x()).cuda()
        y = torch.empty(m.M, dtype=torch.float32, device="cuda")
        gemvs_a.append(sdev.DevGemv(m, Wd, x, y))
    copies = [gemvs_a] if args.warm else [gemvs_a, sdev.clone_weights(gemvs_a)]
    tuning = dict(rows_per_wave=args.rows_per_wave, waves_per_block=args.waves_per_block,
                  unroll=args.unroll, grid=args.grid,
                  flags={"auto": 0, "lds": 1, "direct": 2}[args.x_mode])
    plans = [tvl.tvl_sweep_plan_create([g.item() for g in c], tuning) for c in copies]
    info = plans[0].info()
    torch.cuda.synchronize()

    if args.calib_copy_mib:
        nb = args.calib_copy_mib << 20
        a = torch.empty(nb // 4, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        tvl.tvl_util_copy(b, a, nb)
        torch.cuda.synchronize()
        del a, b

    # read-only streaming ceiling with the same load kind (context)
    ceil_gbs = None
    try:
        nb = 2 << 30
        src = torch.ones(nb // 4, dtype=torch.float32, device="cuda")
        sink = torch.empty(4096, dtype=torch.float32, device="cuda")
        for _ in range(3):
            tvl.tvl_util_read_stream(src, nb, sink, 4096)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(10):
            tvl.tvl_util_read_stream(src, nb, sink, 4096)
        e1.record()
        torch.cuda.synchronize()
        ceil_gbs = nb * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e9
        del src, sink
    except Exception as exc:  # context only; never fatal
        log(f"read ceiling skipped: {exc}")

    for i in range(args.warmup):
        plans[i % len(plans)].run()
    torch.cuda.synchronize()

    # timed region: K back-to-back sweeps on torch's current stream, the
    # stream every launch goes to; events bracket the whole region
    stream = torch.cuda.current_stream()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(args.steps):
        plans[i % len(plans)].run()
    end.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps

    # per-sweep latency distribution (separate pass, not the headline)
    n_lat = min(args.steps, 200)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n_lat + 1)]
    evs[0].record(stream)
    for i in range(n_lat):
        plans[i % len(plans)].run()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    lat = np.array([evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(n_lat)])

    # spot parity of the last sweep of copy 0 against the oracle (5 matrices)
    import oracle
    plans[0].run()
    torch.cuda.synchronize()
    worst = 0.0
    for j in (0, 4, 6, 83, 84):
        g = copies[0][j]
        yref, S = oracle.gemv_f32(hosts[j], g.x.cpu().numpy())
        r = oracle.check(g.y.cpu().numpy(), yref, S, 1e-5)
        worst = max(worst, r["max_err"])
        if r["bad"]:
            log(f"PARITY FAILURE in {g.spec.name}: {r}")
            return 1

    us = ms * 1e3
    gbs = algo / (ms * 1e-3) / 1e9
    traffic = measured_traffic(algo)
    out = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded SplitMix64; W ~ N(0, 0.02^2), x ~ N(0, 1) per matrix)",
        "config": {
            "workload": "sweep110m: one decode token of Llama-2 110M, 85 fp32 GEMVs "
                        "(12 x {768x768 x4, 2048x768 x2, 768x2048} + 32000x768), one launch",
            "algorithmic_bytes": algo,
            "weight_copies_alternated": len(copies),
            "tiles": info["ntiles"],
            "rows_per_tile": info["rows_per_tile"],
            "grid": info["grid"],
        },
        "pct_of_peak": round(100.0 * gbs / PEAK_GBS, 2),
        "us_per_sweep": round(us, 3),
        "tok_s_equiv": round(1e6 / us, 1),
        "latency_us": {"p5": round(float(np.percentile(lat, 5)), 3),
                       "p50": round(float(np.percentile(lat, 50)), 3),
                       "p95": round(float(np.percentile(lat, 95)), 3),
                       "p99": round(float(np.percentile(lat, 99)), 3)},
        "read_ceiling_GBs": None if ceil_gbs is None else round(ceil_gbs, 1),
        "parity_spot_max_err": worst,
        "roofline": {
            "bound": "hbm",
            "achieved": round(gbs, 2),
            "peak": PEAK_GBS,
            "unit": "GB/s",
            "frac": round(gbs / PEAK_GBS, 4),
            "traffic": traffic,
        },
        "paper_context": "paper: >60 tok/s for the 110M model, one thread on Apple M2 Pro "
                         "(whole decode step, not this GEMV sweep alone)",
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle baseline")
        out["cpu_baseline"] = cpu_baseline(wl, hosts, args.cpu_seconds)
    for p in plans:
        p.destroy()
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
