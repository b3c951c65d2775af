#!/usr/bin/env python3
"""Benchmark: one decode token's GEMV sweep of Llama-2 110M on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
every weight matrix of a Llama-2 110M decode step (12 layers x wq, wk, wv, wo
[768x768], w1, w3 [2048x768], w2 [768x2048], plus the 32000x768 classifier;
85 fp32 GEMVs, 438,874,112 algorithmic bytes) computed by ONE launch of the
grouped sweep kernel (a plan run).  The weights, the 85 x vectors and the 85
y buffers are resident in HBM before timing starts.

Copies of the weights are rotated step by step (three for this workload,
1.3 GB together; as many as it takes to span 1 GB for smaller weight sets),
so the 256 MB last-level cache cannot hand one sweep's weights to the next:
the figure is HBM streaming.  ``--warm`` times a single copy instead.

``--workload`` measures the other workloads the same way (not the headline):
sweep7b (Llama-2 7B token, fp32), stack70b8 (8 layers of a 70B-shaped stack,
fp16 weights), cls32000 (the 110M classifier alone, 100 fresh x, 6 weight
copies rotated), gemv768 (one 768x768 fp32 GEMV, cache-resident), and the
decode tokens with RMSNorm and SwiGLU fused into the GEMVs: fused110m (fp32,
2 weight copies alternated) and fused70b8 (fp16 weights); the 110M and 7B
tokens with block-quantised 8-bit / 4-bit weights (sweep110m_q8, sweep110m_q4,
sweep7b_q8, sweep7b_q4; small weight sets are rotated over enough copies to
span 1 GB); beam4_110m / beam8_110m / beam16_110m (several x vectors per
weight read) and beam8_70b / beam16_70b (the same over one 70B-shaped fp16
layer).

Prints ONE JSON line with the metric, a roofline object for the dominant
kernel and the CPU oracle's throughput on a bounded sample of the workload.
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
CSRC = os.path.join(ROOT, "paper_2601_03324_amd", "csrc")
# The sources each workload's dominant kernel is compiled from: the shared
# declarations and device code, plus its family's translation unit.
KERNEL_COMMON = ("tvl_internal.h", "tvl_device.h")
KERNEL_FAMILY = {"fused110m": "tvl_fused.hip", "fused70b8": "tvl_fused.hip",
                 "beam4_110m": "tvl_multi.hip", "beam8_110m": "tvl_multi.hip",
                 "beam16_110m": "tvl_multi.hip", "beam8_70b": "tvl_multi.hip",
                 "beam16_70b": "tvl_multi.hip"}

DESCRIBE = {
    "sweep110m": "sweep110m: one decode token of Llama-2 110M, 85 fp32 GEMVs "
                 "(12 x {768x768 x4, 2048x768 x2, 768x2048} + 32000x768), one launch",
    "sweep7b": "sweep7b: one decode token of Llama-2 7B, 225 fp32 GEMVs "
               "(32 x {4096x4096 x4, 11008x4096 x2, 4096x11008} + 32000x4096), one launch",
    "stack70b8": "stack70b8: 8 layers of a Llama-2 70B-shaped stack, 56 GEMVs, fp16 weights "
                 "(8 x {8192x8192 x2, 1024x8192 x2, 28672x8192 x2, 8192x28672}), one launch",
    "cls32000": "cls32000: the 110M classifier 32000x768 fp32, one GEMV per step, "
                "100 seeded x and 6 weight copies rotated",
    "gemv768": "gemv768: one 768x768 fp32 GEMV per step (cache-resident, launch-bound)",
    "fused110m": "fused110m: one decode token of Llama-2 110M as 73 fused items (RMSNorm -> "
                 "wq/wk/wv, wo, RMSNorm -> SwiGLU(w1, w3), w2, RMSNorm -> classifier), fp32, "
                 "one launch",
    "fused70b8": "fused70b8: 8 layers of the 70B-shaped stack as 48 fused items (RMSNorm -> "
                 "wq/wk/wv, wo, RMSNorm -> SwiGLU(w1, w3), w2), fp16 weights, one launch",
    "beam4_110m": "beam4_110m: one decode token of Llama-2 110M for 4 beam hypotheses: 85 fp32 "
                  "GEMVs x 4 x vectors, weights read once, one launch",
    "beam8_110m": "beam8_110m: one decode token of Llama-2 110M for 8 beam hypotheses: 85 fp32 "
                  "GEMVs x 8 x vectors, weights read once, one launch",
    "beam16_110m": "beam16_110m: one decode token of Llama-2 110M for 16 beam hypotheses: 85 "
                   "fp32 GEMVs x 16 x vectors, weights read once, one launch",
    "beam8_70b": "beam8_70b: one Llama-2 70B-shaped decoder layer for 8 beam hypotheses: 7 "
                 "GEMVs (wq, wk, wv, wo, w1, w3, w2; 1.71 GB of fp16 weights) x 8 x vectors, "
                 "weights read once, one launch",
    "beam16_70b": "beam16_70b: one Llama-2 70B-shaped decoder layer for 16 beam hypotheses: 7 "
                  "GEMVs (1.71 GB of fp16 weights) x 16 x vectors, weights read once, one launch",
}
for _nm, _tok, _n in (("110m", "Llama-2 110M", 85), ("7b", "Llama-2 7B", 225)):
    for _b in (8, 4):
        DESCRIBE[f"sweep{_nm}_q{_b}"] = (
            f"sweep{_nm}_q{_b}: one decode token of {_tok}, {_n} GEMVs with {_b}-bit "
            f"block-quantised weights (one fp32 scale per 64 columns), one launch")
# beam workloads: (source workload, x vectors, leading matrices used or None)
BEAMS = {"beam4_110m": ("sweep110m", 4, None), "beam8_110m": ("sweep110m", 8, None),
         "beam16_110m": ("sweep110m", 16, None), "beam8_70b": ("stack70b8", 8, 7),
         "beam16_70b": ("stack70b8", 16, 7)}


def oracle_rows(oracle, synth, m, rows, x):
    """Oracle (y, S) of the sampled rows of matrix ``m``, each row regenerated
    on its own from the counter-based generator."""
    import numpy as np
    if m.quantised:
        ys, Ss = [], []
        for r in rows:
            y, S = oracle.gemv_q(m.weights(int(r), 1), m.bits, synth.q_row_bytes(m.K, m.bits),
                                 1, m.K, x)
            ys.append(y[0])
            Ss.append(S[0])
        return np.array(ys), np.array(Ss)
    Wr = np.stack([m.weights(int(r), 1)[0] for r in rows])
    return (oracle.gemv_f32 if m.dtype == "f32" else oracle.gemv_f16)(Wr, x)


def oracle_gemv(oracle, synth, m, W, x):
    if m.quantised:
        return oracle.gemv_q(W, m.bits, synth.q_row_bytes(m.K, m.bits), m.M, m.K, x)
    return (oracle.gemv_f32 if m.dtype == "f32" else oracle.gemv_f16)(W, x)


def dtype_label(m) -> str:
    if m.quantised:
        return f"{m.dtype} weights (fp32 scale per 64 columns), f32 x/accumulation"
    return "f16 weights, f32 x/accumulation" if m.dtype == "f16" else "f32"


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def kernel_sources(workload: str) -> list:
    if workload in KERNEL_FAMILY:
        fam = KERNEL_FAMILY[workload]
    elif workload.endswith(("_q8", "_q4")):
        fam = "tvl_quant.hip"
    else:
        fam = "tvl_gemv.hip"
    return [*KERNEL_COMMON, fam]


def kernel_hash(workload: str) -> str:
    """sha256[:16] over the sources of the workload's kernel family, in order."""
    h = hashlib.sha256()
    for f in kernel_sources(workload):
        h.update(open(os.path.join(CSRC, f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when there is none or the kernel source changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"{workload}_traffic.json")
    try:
        t = json.load(open(path))
    except (OSError, ValueError):
        return None
    if t.get("kernel_src_sha256_16") != kernel_hash(workload):
        return None
    return t.get("bytes_per_launch")


def cpu_baseline(samples, seconds: float, what: str, threads: int = 1) -> dict:
    """The oracle as it stands (single-threaded naive double GEMV), cycling over
    (spec, W, x) samples of the workload for about ``seconds`` of CPU time; with
    ``threads`` > 1 also the same calls on that many host threads at once."""
    import oracle
    import synth
    t0 = time.perf_counter()
    nbytes, ngemv = 0, 0
    while True:
        for m, W, x in samples:
            oracle_gemv(oracle, synth, m, W, x)
            nbytes += m.algo_bytes()
            ngemv += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    gbs = nbytes / el / 1e9
    out = {"value": round(gbs, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
           "sample": f"{ngemv} GEMVs of {what} ({nbytes / 1e9:.2f} GB algorithmic) in "
                     f"{el:.1f} s on one host thread",
           "cpu": cpu_model()}
    if threads > 1:
        out["all_cores"] = cpu_baseline_threads(samples, seconds / 2, what, threads)
    return out


def cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo), else the platform's."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def host_threads() -> int:
    """Host threads for the all-cores leg: the CPUs this process may run on,
    capped by OMP_NUM_THREADS when set (a container's share of its host)."""
    n = len(os.sched_getaffinity(0))
    omp = os.environ.get("OMP_NUM_THREADS", "")
    return min(n, int(omp)) if omp.isdigit() and int(omp) > 0 else n


def cpu_baseline_threads(samples, seconds: float, what: str, threads: int) -> dict:
    """The same oracle calls on `threads` host threads at once, each taking
    whole GEMVs of the sample in turn (ctypes releases the GIL during a call,
    so the GEMVs run in parallel; the per-row arithmetic is unchanged)."""
    import itertools
    import threading
    import oracle
    import synth
    nxt = itertools.count()
    done = [0] * threads
    t0 = time.perf_counter()

    def worker(t):
        while time.perf_counter() - t0 < seconds:
            m, W, x = samples[next(nxt) % len(samples)]
            oracle_gemv(oracle, synth, m, W, x)
            done[t] += m.algo_bytes()

    ts = [threading.Thread(target=worker, args=(t,)) for t in range(threads)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    el = time.perf_counter() - t0
    return {"value": round(sum(done) / el / 1e9, 4), "unit": "GB/s", "cores": threads,
            "sample": f"GEMVs of {what} on {threads} host threads, whole GEMVs per thread, "
                      f"{sum(done) / 1e9:.2f} GB algorithmic in {el:.1f} s"}


def emit(out: dict) -> None:
    """Print the JSON line, with the device it was measured on."""
    import torch
    p = torch.cuda.get_device_properties(0)
    out["device"] = {"name": p.name, "arch": getattr(p, "gcnArchName", ""),
                     "compute_units": p.multi_processor_count,
                     "hbm_GiB": round(p.total_memory / 2**30, 1),
                     "hip_runtime": torch.version.hip}
    print(json.dumps(out), flush=True)


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", choices=sorted(DESCRIBE), default="sweep110m")
    ap.add_argument("--warm", action="store_true", help="one weight copy (cache-warm)")
    ap.add_argument("--graph", choices=("auto", "on", "off"), default="auto",
                    help="single-GEMV workloads: time the K steps as one captured HIP graph "
                         "(auto: on for gemv768, whose launches are host-bound)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--rows-per-wave", type=int, default=0)
    ap.add_argument("--waves-per-block", type=int, default=0)
    ap.add_argument("--unroll", type=int, default=0)
    ap.add_argument("--grid", type=int, default=0)
    ap.add_argument("--ksplit", type=int, default=0, help="single-GEMV workloads only")
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
    import oracle
    import synth
    import synth.device as sdev
    from paper_2601_03324_amd import tvl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    torch.cuda.set_device(0)
    if args.calib_copy_mib:
        # one plain copy of known size: its FETCH_SIZE / WRITE_SIZE counters
        # calibrate what those counters read for the kernels of this run
        nb = args.calib_copy_mib << 20
        a = torch.empty(nb // 4, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        tvl.tvl_util_copy(b, a, nb)
        torch.cuda.synchronize()
        del a, b
    if args.workload in synth.FUSED_WORKLOADS:
        return run_fused(args, tvl, torch, np, oracle, synth, sdev)
    if args.workload in BEAMS:
        return run_beam(args, tvl, torch, np, oracle, synth, sdev)
    wl = synth.WORKLOADS[args.workload]
    single = args.workload in ("cls32000", "gemv768")
    algo = wl.mats[0].algo_bytes() if single else wl.algo_bytes()
    tuning = dict(rows_per_wave=args.rows_per_wave, waves_per_block=args.waves_per_block,
                  unroll=args.unroll, grid=args.grid, ksplit=args.ksplit,
                  flags={"auto": 0, "lds": 1, "direct": 2}[args.x_mode])
    if not single and args.ksplit:
        print("--ksplit applies to single-GEMV workloads", file=sys.stderr)
        return 2
    use_tuning = any(tuning.values())

    log(f"generating {wl.name}: {len(wl.mats)} GEMVs, {wl.weight_bytes() / 1e6:.1f} MB of weights")
    big = wl.weight_bytes() > 4e9
    cpu_samples = []  # (spec, host W, x) for the CPU baseline and the spot check
    gemvs = []
    for i, m in enumerate(wl.mats):
        W = m.weights()
        Wd = sdev.upload(m, W, "cuda")
        x = m.x()
        gemvs.append(sdev.DevGemv(m, Wd, torch.from_numpy(x).cuda(),
                                  torch.empty(m.M, dtype=torch.float32, device="cuda")))
        if not big or i < 7:
            cpu_samples.append((m, W, x))
        if big and i % 16 == 0:
            log(f"  uploaded {i + 1}/{len(wl.mats)}")
    stream = torch.cuda.current_stream()

    if single:
        m, g = wl.mats[0], gemvs[0]
        ncopy = 1 if (args.warm or args.workload == "gemv768") else 6
        Ws = [g.W] + [tvl.TvlMatrix(g.W.buf.clone(), m.M, m.K, g.W.ldw, g.W.dtype)
                      for _ in range(ncopy - 1)]
        xs = [torch.from_numpy(m.x(r)).cuda() for r in range(wl.reps)]
        y = torch.empty(m.M, dtype=torch.float32, device="cuda")
        # arguments marshalled once: plain ints for every pointer and the
        # stream handle, so a step costs the C call and its launch, not the
        # tensor and current-stream lookups of the Python layer
        sid = int(torch.cuda.current_stream().cuda_stream)
        wp = [(int(Wc.ptr), Wc.ldw, Wc.dtype) for Wc in Ws]
        xp = [int(xc.data_ptr()) for xc in xs]
        yp = int(y.data_ptr())
        tun = tvl._tuning(tuning) if use_tuning else None

        def step(i):
            w, ldw, dt = wp[i % ncopy]
            if use_tuning:
                tvl.tvl_gemv_ex(w, ldw, dt, xp[i % len(xp)], yp, m.M, m.K, tun, sid)
            else:
                tvl.tvl_gemv(w, ldw, dt, xp[i % len(xp)], yp, m.M, m.K, sid)

        copies_used = ncopy
        plan_info = {}
    else:
        # enough copies that the rotation spans >= 1 GB (4x the last-level cache)
        ncopy = 1 if (args.warm or big) else max(2, -(-1_000_000_000 // wl.weight_bytes()))
        copies = [gemvs] + [sdev.clone_weights(gemvs) for _ in range(ncopy - 1)]
        plans = [tvl.tvl_sweep_plan_create([g.item() for g in c], tuning if use_tuning else None)
                 for c in copies]
        plan_info = plans[0].info()

        sid = int(torch.cuda.current_stream().cuda_stream)

        def step(i):
            plans[i % ncopy].run(sid)

        copies_used = ncopy
    torch.cuda.synchronize()

    # read-only streaming ceiling with the same load kind (context)
    ceil_gbs = None
    try:
        nb = 2 << 30
        src = torch.ones(nb // 4, dtype=torch.float32, device="cuda")
        sink = torch.empty(1 << 16, dtype=torch.float32, device="cuda")
        grid = 8192  # 256 KB per workgroup: the fastest plain read measured on MI355X
        for _ in range(3):
            tvl.tvl_util_read_stream(src, nb, sink, grid)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(10):
            tvl.tvl_util_read_stream(src, nb, sink, grid)
        e1.record(stream)
        torch.cuda.synchronize()
        ceil_gbs = nb * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e9
        del src, sink
    except Exception as exc:  # context only; never fatal
        log(f"read ceiling skipped: {exc}")
    same = read_ceiling_same_bytes(algo, tvl, torch, stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # timed region: K back-to-back steps on torch's current stream, the
    # stream every launch goes to; events bracket the whole region
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(args.steps):
        step(i)
    end.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps
    ms_eager = ms

    # launch-bound single GEMV: the same K steps captured once as a HIP graph
    # (no allocation, memset or host sync inside a step), replayed in the
    # timed region; the replayed output is checked bitwise against eager
    use_graph = single and (args.graph == "on" or (args.graph == "auto"
                                                   and args.workload == "gemv768"))
    if use_graph:
        gs = torch.cuda.Stream()
        gs.wait_stream(stream)
        with torch.cuda.stream(gs):
            sid_eager, sid = sid, int(gs.cuda_stream)
            step(args.steps - 1)  # the steps' launch path, once on the capture stream
            gs.synchronize()
            y_eager = y.clone()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=gs):
                for i in range(args.steps):
                    step(i)
            sid = sid_eager
        torch.cuda.synchronize()
        for rep in range(3):  # replays, eager work and syncs in between (bitwise)
            y.fill_(float("nan"))
            graph.replay()
            torch.cuda.synchronize()
            if not torch.equal(y, y_eager):
                log("graph replay differs from the eager result")
                return 1
            step(0)
            torch.cuda.synchronize()
        start.record(stream)
        graph.replay()
        end.record(stream)
        torch.cuda.synchronize()
        ms = start.elapsed_time(end) / args.steps

    # per-step latency distribution (separate pass, not the headline)
    n_lat = min(args.steps, 200)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n_lat + 1)]
    evs[0].record(stream)
    for i in range(n_lat):
        step(i)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    lat = np.array([evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(n_lat)])

    # spot parity against the oracle: sampled outputs of the first copy
    worst = 0.0
    step(0)  # copy 0 (and x rep 0 for single GEMVs)
    torch.cuda.synchronize()
    checks = cpu_samples[:3] + ([] if single else [(gemvs[-1].spec, None, None)])
    for m, W, x in checks:
        g = next(gg for gg in gemvs if gg.spec is m)
        ydev = (y if single else g.y).cpu().numpy()
        rows = sdev.sample_rows(m.M, 64, 7)
        yref, S = oracle_rows(oracle, synth, m, rows, m.x(0))
        r = oracle.check(ydev[rows], yref, S, 2e-3 if m.dtype == "f16" else 1e-5)
        worst = max(worst, r["max_err"])
        if r["bad"]:
            log(f"PARITY FAILURE in {m.name}: {r}")
            return 1

    us = ms * 1e3
    gbs = algo / (ms * 1e-3) / 1e9
    dtype = dtype_label(wl.mats[0])
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
        "dtype": dtype,
        "data": "synthetic (seeded SplitMix64; W ~ N(0, 0.02^2), x ~ N(0, 1) per matrix)",
        "config": {
            "workload": DESCRIBE[args.workload],
            "algorithmic_bytes_per_step": algo,
            "weight_copies_rotated": copies_used,
            **({"tiles": plan_info["ntiles"], "rows_per_tile": plan_info["rows_per_tile"],
                "grid": plan_info["grid"]} if plan_info else {}),
            **({"launch": f"{args.steps} steps captured as one HIP graph, replayed once; "
                          f"eager launches: {ms_eager * 1e3:.2f} us per step"}
               if use_graph else {}),
        },
        "pct_of_peak": round(100.0 * gbs / PEAK_GBS, 2),
        ("us_per_gemv" if single else "us_per_sweep"): round(us, 3),
        "latency_us": {"p5": round(float(np.percentile(lat, 5)), 3),
                       "p50": round(float(np.percentile(lat, 50)), 3),
                       "p95": round(float(np.percentile(lat, 95)), 3),
                       "p99": round(float(np.percentile(lat, 99)), 3)},
        "read_ceiling_GBs": None if ceil_gbs is None else round(ceil_gbs, 1),
        "read_ceiling_same_bytes": same,
        "parity_spot_max_err": worst,
        "roofline": {
            "bound": "hbm",
            "achieved": round(gbs, 2),
            "peak": PEAK_GBS,
            "unit": "GB/s",
            "frac": round(gbs / PEAK_GBS, 4),
            "traffic": measured_traffic(args.workload),
        },
    }
    if not single:
        out["tok_s_equiv"] = round(1e6 / us, 1)
    if args.workload == "sweep110m":
        out["paper_context"] = ("paper: >60 tok/s for the 110M model, one thread on Apple M2 Pro "
                                "(whole decode step, not this GEMV sweep alone)")
    if not args.no_cpu_baseline:
        log("timing the CPU oracle baseline")
        out["cpu_baseline"] = cpu_baseline(cpu_samples, args.cpu_seconds, wl.name,
                                           host_threads())
    if not single:
        for p in plans:
            p.destroy()
    emit(out)
    return 0


def read_ceiling_same_bytes(nbytes: int, tvl, torch, stream) -> dict:
    """The plain streaming read (the GEMV's load kind, no arithmetic) over the
    same number of bytes as one launch of the workload: what this GPU reads
    in a launch of that size, ramp-up and drain included.  Copies are rotated
    over >= 1 GB (4x the last-level cache), so every launch reads from HBM;
    the best of several grids is reported (context for the roofline
    fraction, not a target).  The reads of each grid are captured once as a
    HIP graph and replayed, so host launch overhead cannot starve the GPU
    between launches of a few microseconds (the first replay's sink is
    checked bitwise against the eager launches' first)."""
    nb = min(int(nbytes) // 256 * 256, 2 << 30)
    ncopy = max(2, -(-1_000_000_000 // nb)) if nb < (1 << 30) else 1
    src = torch.ones(nb * ncopy // 4, dtype=torch.float32, device="cuda")
    base = int(src.data_ptr())
    sink = torch.zeros(1 << 16, dtype=torch.float32, device="cuda")
    best = (0.0, 0)
    for grid in (512, 1024, 2048, 4096, 8192, 16384, 32768):
        reps = max(20, 2 * ncopy)
        gs = torch.cuda.Stream()
        gs.wait_stream(stream)
        sid = int(gs.cuda_stream)
        with torch.cuda.stream(gs):
            for i in range(reps):  # eager first: warms up and gives the reference sink
                tvl.tvl_util_read_stream(base + (i % ncopy) * nb, nb, sink, grid, sid)
            gs.synchronize()
            ref = sink[:grid].clone()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=gs):
                for i in range(reps):
                    tvl.tvl_util_read_stream(base + (i % ncopy) * nb, nb, sink, grid, sid)
        sink.zero_()
        graph.replay()
        torch.cuda.synchronize()
        if not torch.equal(sink[:grid], ref):
            raise RuntimeError("read-ceiling graph replay differs from the eager launches")
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        gbs = nb * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
        best = max(best, (gbs, grid))
        del graph
    del src, sink
    return {"GBs": round(best[0], 1), "bytes": nb, "grid": best[1], "copies_rotated": ncopy,
            "frac_of_peak": round(best[0] / PEAK_GBS, 4),
            "timing": "one HIP graph of back-to-back launches per grid, best of 7 grids"}


def time_steps(step, steps, warmup, torch, np, stream):
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for i in range(steps):
        step(i)
    end.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / steps
    n_lat = min(steps, 200)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n_lat + 1)]
    evs[0].record(stream)
    for i in range(n_lat):
        step(i)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    lat = np.array([evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(n_lat)])
    return ms, lat


def run_beam(args, tvl, torch, np, oracle, synth, sdev) -> int:
    """A decode token (or one layer) for B beam hypotheses (several x vectors
    per GEMV)."""
    src, B, nmats = BEAMS[args.workload]
    wl = synth.WORKLOADS[src]
    if nmats:
        wl = synth.Workload(f"{src}[:{nmats}]", wl.cfg, tuple(wl.mats[:nmats]))
    big = wl.weight_bytes() > 1e9  # far beyond the caches: one copy is cold
    algo = sum(m.wbytes + B * (4 * m.K + 4 * m.M) for m in wl.mats)
    log(f"generating {args.workload}: {len(wl.mats)} GEMVs x {B} vectors")
    a = sdev.load_multi(wl, B, "cuda")
    copies = [a]
    if not (args.warm or big):
        copies.append(sdev.load_multi(wl, B, "cuda", share_from=[
            sdev.DevGemv(d.spec, tvl.TvlMatrix(d.W.buf.clone(), d.W.M, d.W.K, d.W.ldw, d.W.dtype),
                         None, None) for d in a]))
    tuning = dict(rows_per_wave=args.rows_per_wave, waves_per_block=args.waves_per_block,
                  unroll=args.unroll, grid=args.grid,
                  flags={"auto": 0, "lds": 1, "direct": 2}[args.x_mode])
    use_tuning = any(tuning.values())
    plans = [tvl.tvl_sweep_plan_create([d.item() for d in c], tuning if use_tuning else None)
             for c in copies]
    info = plans[0].info()
    stream = torch.cuda.current_stream()
    sid = int(stream.cuda_stream)

    def step(i):
        plans[i % len(plans)].run(sid)

    ms, lat = time_steps(step, args.steps, args.warmup, torch, np, stream)
    same = read_ceiling_same_bytes(algo, tvl, torch, stream)
    plans[0].run()
    torch.cuda.synchronize()
    worst = 0.0
    for j in sorted({0, min(6, len(a) - 1), len(a) - 1}):
        d = a[j]
        m = d.spec
        rows = sdev.sample_rows(m.M, 64, 13)
        Y = d.Y.cpu().numpy()
        for b in range(B):
            ref, S = oracle_rows(oracle, synth, m, rows, m.x(b))
            r = oracle.check(Y[b][rows], ref, S, 2e-3 if m.dtype == "f16" else 1e-5)
            worst = max(worst, r["max_err"])
            if r["bad"]:
                log(f"PARITY FAILURE in {m.name} vector {b}: {r}")
                return 1
    us = ms * 1e3
    gbs = algo / (ms * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": round(gbs, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": dtype_label(wl.mats[0]),
        "data": "synthetic (seeded SplitMix64; W ~ N(0, 0.02^2), x ~ N(0, 1) per vector)",
        "config": {"workload": DESCRIBE[args.workload], "algorithmic_bytes_per_step": algo,
                   "vectors": B, "weight_copies_rotated": len(copies), "tiles": info["ntiles"],
                   "rows_per_tile": info["rows_per_tile"], "grid": info["grid"]},
        "pct_of_peak": round(100.0 * gbs / PEAK_GBS, 2),
        "us_per_sweep": round(us, 3),
        "tok_s_equiv": round(B * 1e6 / us, 1),
        "latency_us": {"p5": round(float(np.percentile(lat, 5)), 3),
                       "p50": round(float(np.percentile(lat, 50)), 3),
                       "p95": round(float(np.percentile(lat, 95)), 3),
                       "p99": round(float(np.percentile(lat, 99)), 3)},
        "read_ceiling_same_bytes": same,
        "parity_spot_max_err": worst,
        "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / PEAK_GBS, 4),
                     "traffic": measured_traffic(args.workload)},
    }
    if not args.no_cpu_baseline:
        samples = [(m, m.weights(), m.x(0)) for m in wl.mats[:7]]
        out["cpu_baseline"] = cpu_baseline(samples, args.cpu_seconds, f"{wl.name} (per vector)")
    for p in plans:
        p.destroy()
    emit(out)
    return 0


def run_fused(args, tvl, torch, np, oracle, synth, sdev) -> int:
    """A decode token as fused items (RMSNorm / SwiGLU folded into the GEMVs)."""
    wl = synth.FUSED_WORKLOADS[args.workload]
    algo = wl.algo_bytes()
    big = wl.weight_bytes() > 4e9
    log(f"generating {wl.name}: {len(wl.items)} items, {wl.weight_bytes() / 1e6:.1f} MB of weights")
    items_a = sdev.load_fused(wl, "cuda", progress=big)
    copies = [items_a]
    if not (args.warm or big):
        clone = []
        for d in items_a:
            W = tvl.TvlMatrix(d.W.buf.clone(), d.W.M, d.W.K, d.W.ldw, d.W.dtype)
            W3 = (tvl.TvlMatrix(d.W3.buf.clone(), d.W3.M, d.W3.K, d.W3.ldw, d.W3.dtype)
                  if d.W3 is not None else None)
            clone.append(sdev.DevFused(d.spec, W, W3, d.x, d.g, torch.empty_like(d.y)))
        copies.append(clone)
    tuning = dict(rows_per_wave=args.rows_per_wave, waves_per_block=args.waves_per_block,
                  unroll=args.unroll, grid=args.grid,
                  flags={"auto": 0, "lds": 1, "direct": 2}[args.x_mode])
    use_tuning = any(tuning.values())
    plans = [tvl.tvl_sweep_plan_create([d.item() for d in c], tuning if use_tuning else None)
             for c in copies]
    info = plans[0].info()
    stream = torch.cuda.current_stream()
    sid = int(stream.cuda_stream)

    def step(i):
        plans[i % len(plans)].run(sid)

    ms, lat = time_steps(step, args.steps, args.warmup, torch, np, stream)
    same = read_ceiling_same_bytes(algo, tvl, torch, stream)
    # spot parity: three items of copy 0 (a normalised GEMV, a SwiGLU pair, a plain GEMV)
    plans[0].run()
    torch.cuda.synchronize()
    worst = 0.0
    picks = [d for d in items_a if d.W3 is None and d.g is not None][:1] + \
            [d for d in items_a if d.W3 is not None][:1] + \
            [d for d in items_a if d.W3 is None and d.g is None][:1]
    samples = []
    for d in picks:
        it = d.spec
        rows = sdev.sample_rows(it.M, 64, 11)
        W = np.stack([it.W.weights(int(r), 1)[0] for r in rows])
        x = it.x.values()
        g = it.g.values() if it.g is not None else None
        y = d.y.cpu().numpy()[rows]
        tol = 1e-5 if it.W.dtype == "f32" else 2e-3
        if it.W3 is None:
            xd = oracle.rmsnorm(x, g, it.eps) if g is not None else x.astype(np.float64)
            yref, S = oracle.gemv_dx(W, xd)
            r = oracle.check(y, yref, S, tol)
        else:
            W3 = np.stack([it.W3.weights(int(rr), 1)[0] for rr in rows])
            href, a, b, Sa, Sb = oracle.swiglu_ffn_in(W, W3, x, g, it.eps)
            r = oracle.check(y, href, oracle.swiglu_bound(a, b, Sa, Sb), tol)
        worst = max(worst, r["max_err"])
        if r["bad"]:
            log(f"PARITY FAILURE in {it.name}: {r}")
            return 1
        samples.append((it, W, x, g))
    us = ms * 1e3
    gbs = algo / (ms * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": round(gbs, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f16 weights, f32 x/accumulation" if wl.items[0].W.dtype == "f16" else "f32",
        "data": "synthetic (seeded SplitMix64; W ~ N(0, 0.02^2), x ~ N(0, 1), g ~ U(0.5, 1.5))",
        "config": {"workload": DESCRIBE[args.workload], "algorithmic_bytes_per_step": algo,
                   "weight_copies_rotated": len(copies), "tiles": info["ntiles"],
                   "rows_per_tile": info["rows_per_tile"], "grid": info["grid"]},
        "pct_of_peak": round(100.0 * gbs / PEAK_GBS, 2),
        "us_per_sweep": round(us, 3),
        "tok_s_equiv": round(1e6 / us, 1),
        "latency_us": {"p5": round(float(np.percentile(lat, 5)), 3),
                       "p50": round(float(np.percentile(lat, 50)), 3),
                       "p95": round(float(np.percentile(lat, 95)), 3),
                       "p99": round(float(np.percentile(lat, 99)), 3)},
        "read_ceiling_same_bytes": same,
        "parity_spot_max_err": worst,
        "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / PEAK_GBS, 4),
                     "traffic": measured_traffic(args.workload)},
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle baseline")
        full = [(it, it.W.weights(), it.W3.weights() if it.W3 is not None else None, x, g)
                for it, _, x, g in samples]
        t0 = time.perf_counter()
        nbytes, n = 0, 0
        while time.perf_counter() - t0 < args.cpu_seconds:
            for it, W, W3, x, g in full:
                if W3 is None:
                    xd = oracle.rmsnorm(x, g, it.eps) if g is not None else x.astype(np.float64)
                    oracle.gemv_dx(W, xd)
                else:
                    oracle.swiglu_ffn_in(W, W3, x, g, it.eps)
                nbytes += it.algo_bytes()
                n += 1
        el = time.perf_counter() - t0
        out["cpu_baseline"] = {
            "value": round(nbytes / el / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{n} fused items of {wl.name} (a normalised GEMV, a SwiGLU pair, a plain "
                      f"GEMV in turn; {nbytes / 1e9:.2f} GB algorithmic) in {el:.1f} s on one "
                      f"host thread", "cpu": cpu_model()}
    for p in plans:
        p.destroy()
    emit(out)
    return 0


if __name__ == "__main__":
    sys.exit(main())
