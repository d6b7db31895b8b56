#!/usr/bin/env python3
"""Benchmark of the fused fp16 GEMM + bias + ReLU on one MI355X.

Default workload: M = N = K = 4096, A row-major, B column-major, fp16
uniform[-1,1] inputs, fp32 accumulation, bias + ReLU epilogue.  A step is one
call of the fused kernel; the metric is 2MNK / time in TFLOP/s.

Prints ONE JSON line (see the keys below).  Besides the headline it reports
the unfused three-launch chain (GEMM, bias add, ReLU) and the plain GEMM on
the same inputs, the roofline position of the fused kernel, and the CPU
oracle timed on a bounded sample of the same problem.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--tile ID]
                    [--report PATH] [--no-cpu]
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_F16_TFLOPS = 2500.0      # MI355X dense fp16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
METRIC = "fused GEMM+bias+ReLU TFLOP/s (2MNK/t) fp16 on 1 MI355X; % of MFMA peak"
HEADLINE = "cube4096_RC"
PROFILES = os.path.join(ROOT, "profiles")


def kernel_source_digest():
    """sha256 over the HIP sources, to tell whether stored counters are stale."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2006_12645_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".hpp")):
            h.update(name.encode())
            h.update(open(os.path.join(csrc, name), "rb").read())
    return h.hexdigest()


def stored_traffic(workload):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary, or
    None when absent or taken on different kernel sources."""
    path = os.path.join(PROFILES, f"gemm_bias_act_{workload}_pmc.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_sha = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text)
    m_b = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_sha or not m_b or m_sha.group(1) != kernel_source_digest():
        return None
    return float(m_b.group(1))


def time_launches(fn, steps, warmup, torch):
    """Average ms per call of fn over `steps` calls (after `warmup`), timed
    with events on the current stream, which is where the library launches."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        fn()
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) / steps


def cpu_baseline(w, A, B, bias, target_s=12.0):
    """The oracle on a bounded sample of output rows of the same problem."""
    import numpy as np
    from oracle import oracle as O
    from paper_2006_12645_amd import datagen as D
    a_st, b_st = D.store(A, D.ROW), D.store(B, D.COL)
    threads = O.default_threads()
    rows = list(range(min(w.M, 4 * threads)))
    t0 = time.perf_counter()
    O.gemm_bias_act(a_st, D.ROW, b_st, D.COL, w.M, w.N, w.K, bias=bias, rows=rows, nthreads=threads)
    dt = time.perf_counter() - t0
    # grow the sample to about target_s of work
    nrows = int(min(w.M, max(len(rows), len(rows) * target_s / max(dt, 1e-3))))
    rows = list(range(nrows))
    t0 = time.perf_counter()
    O.gemm_bias_act(a_st, D.ROW, b_st, D.COL, w.M, w.N, w.K, bias=bias, rows=rows, nthreads=threads)
    dt = time.perf_counter() - t0
    flops = 2.0 * nrows * w.N * w.K
    del np
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{nrows} of {w.M} output rows (all {w.N} columns, full K={w.K}) of the "
                      f"same {w.name} problem, fp64, {dt:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--tile", type=int, default=None)
    ap.add_argument("--report", default=None, help="also write per-variant numbers here (JSON)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--fused-only", action="store_true",
                    help="time only the fused kernel (for profiler runs); implies --no-cpu")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run 5 plain device-to-device copies of MIB MiB (the reference "
                         "kernel for scaling rocprofv3 FETCH_SIZE/WRITE_SIZE) and exit")
    args = ap.parse_args()

    if args.calibrate_copy:
        import torch
        n = args.calibrate_copy * (1 << 20)
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_per_launch": n, "launches": 5}), flush=True)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the fused kernel has no multi-GPU path; "
              "run with --gpus 1", file=sys.stderr, flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2006_12645_amd import datagen as D
    from paper_2006_12645_amd import gba

    gba.lib()  # raises if the HIP library is not built
    w = D.WORKLOADS[args.workload]
    A, B, bias = D.logical_inputs(w)
    dA = torch.from_numpy(A).cuda()                                    # row-major
    dB = torch.from_numpy(np.ascontiguousarray(B.T)).cuda().t()        # column-major
    dbias = torch.from_numpy(bias).cuda()
    out = torch.empty((w.M, w.N), dtype=torch.float16, device="cuda")
    tile = args.tile if args.tile is not None else gba.select_tile(w.M, w.N, w.K)

    fused = lambda: gba.gemm_bias_act(dA, dB, dbias, act="relu", out=out, tile=tile)
    plain = lambda: gba.gemm_bias_act(dA, dB, None, act="none", out=out, tile=tile)
    unfused = lambda: gba.unfused_gemm_bias_relu(dA, dB, dbias, out=out, tile=tile)

    torch.cuda.synchronize()
    ms = time_launches(fused, args.steps, args.warmup, torch)
    torch.cuda.synchronize()
    if args.fused_only:
        args.no_cpu = True
        ms_plain = ms_unfused = ms_fused2 = float("nan")
    else:
        # the comparison legs get the same warmup, then the fused kernel is
        # timed once more right after the unfused chain
        ms_plain = time_launches(plain, args.steps, args.warmup, torch)
        ms_unfused = time_launches(unfused, args.steps, args.warmup, torch)
        ms_fused2 = time_launches(fused, args.steps, 0, torch)

    flops = 2.0 * w.M * w.N * w.K
    tflops = flops / (ms * 1e-3) / 1e12
    algo_bytes = 2.0 * (w.M * w.K + w.K * w.N + w.M * w.N + w.N)
    info = gba.tile_info(tile)

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(w, A, B, bias)

    traffic = stored_traffic(w.name)
    line = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: fused fp16 GEMM+bias+ReLU M={w.M} N={w.N} K={w.K}, "
                               f"A row-major, B column-major, fp32 accumulation",
                   "M": w.M, "N": w.N, "K": w.K, "layout": "RC", "accum": "f32",
                   "tile": dict(id=tile, **info), "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "mfma", "achieved": round(tflops, 2), "peak": PEAK_F16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(tflops / PEAK_F16_TFLOPS, 4),
                     "traffic": traffic},
        "cpu_baseline": cpu,
        "extra": None if args.fused_only else {
            "frac_of_fp16_peak": round(tflops / PEAK_F16_TFLOPS, 4),
            "fused_ms_second_pass": round(ms_fused2, 5),
            "plain_gemm_ms": round(ms_plain, 5),
            "plain_gemm_tflops": round(flops / (ms_plain * 1e-3) / 1e12, 2),
            "unfused_3launch_ms": round(ms_unfused, 5),
            "fused_vs_unfused_speedup": round(ms_unfused / ms, 3),
            "fused_algorithmic_GBps": round(algo_bytes / (ms * 1e-3) / 1e9, 1),
        },
    }
    if args.report:
        with open(args.report, "w") as f:
            json.dump(line, f, indent=1)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
