#!/usr/bin/env python3
"""Benchmark of the fused fp16 GEMM + bias + ReLU on one MI355X.

Default workload: M = N = K = 4096, A row-major, B column-major, fp16
uniform[-1,1] inputs, fp32 accumulation, bias + ReLU epilogue.  A step is one
call of the fused kernel; the metric is 2MNK / time in TFLOP/s.

Prints ONE JSON line (see the keys below).  Besides the headline it reports
the unfused three-launch chain (GEMM, bias add, ReLU) and the plain GEMM on
the same inputs, the roofline position of the fused kernel, and the CPU
oracle timed on a bounded sample of the same problem.

--workload prologue4096_RC times relu(A).B + bias -> ReLU (against a ReLU
pass over A followed by the fused GEMM), --workload sum4096_RC times
A.B + P.Q + bias -> ReLU with K2 = K (against two GEMMs, an add, a bias add
and a ReLU); their metric counts 2MN(K + K2) flops.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--tile ID]
                    [--report PATH] [--no-cpu]
    python bench.py --configs      # every workload configuration, one line each
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


def cpu_baseline(w, A, B, bias, P=None, Q=None, target_s=12.0):
    """The oracle on a bounded sample of output rows of the same problem."""
    from oracle import oracle as O
    from paper_2006_12645_amd import datagen as D
    a_st, b_st = D.store(A, D.ROW), D.store(B, D.COL)
    K2 = w.extra.get("K2", 0) if P is not None else 0
    kw = dict(prologue_relu=w.extra.get("prologue") == "relu", bias=bias, act=O.ACT_RELU)
    if P is not None:
        kw.update(second=1, p_store=D.store(P, D.ROW), q_store=D.store(Q, D.COL), K2=K2)
    threads = O.default_threads()

    def run(rows):
        t0 = time.perf_counter()
        O.fused(a_st, D.ROW, b_st, D.COL, w.M, w.N, w.K, rows=rows, nthreads=threads, **kw)
        return time.perf_counter() - t0

    rows = list(range(min(w.M, 4 * threads)))
    dt = run(rows)
    # grow the sample to about target_s of work
    nrows = int(min(w.M, max(len(rows), len(rows) * target_s / max(dt, 1e-3))))
    dt = run(list(range(nrows)))
    flops = 2.0 * nrows * w.N * (w.K + K2)
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{nrows} of {w.M} output rows (all {w.N} columns, full reduction "
                      f"K={w.K}{f' + K2={K2}' if K2 else ''}) of the same {w.name} problem, "
                      f"fp64, {dt:.1f} s"}


def time_graph(fns, launches, replays, torch):
    """Average ms per launch of `launches` calls (cycling through fns)
    captured in one HIP graph and replayed: device time without the host's
    per-call launch cost."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for f in fns[:3]:
            f()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(launches):
            fns[i % len(fns)]()
    g.replay()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(replays):
        g.replay()
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) / (replays * launches)


COLD_POOL_BYTES = 1 << 30


def cold_operands(torch, dA, dB, M, N, nsets):
    """nsets copies of (A, B, C) in distinct memory, same layouts and values,
    so that rotating through them misses the caches (L2 and the 256 MB
    last-level cache) on every launch."""
    def pool(t):
        if t.stride(-1) == 1:
            p = torch.empty((nsets,) + tuple(t.shape), dtype=t.dtype, device=t.device)
            p.copy_(t.unsqueeze(0).expand_as(p))
            return [p[i] for i in range(nsets)]
        tt = t.t()
        p = torch.empty((nsets,) + tuple(tt.shape), dtype=t.dtype, device=t.device)
        p.copy_(tt.unsqueeze(0).expand_as(p))
        return [p[i].t() for i in range(nsets)]
    outs = torch.empty((nsets, M, N), dtype=torch.float16, device=dA.device)
    return list(zip(pool(dA), pool(dB), [outs[i] for i in range(nsets)]))


def configs(args, np, torch, D, gba):
    """Every single-product workload configuration: layouts x accumulations,
    the library's tile choice.  `us` is device time per launch from a
    captured graph of back-to-back launches on the same (cache-resident)
    operands; `us_eager` the same launches issued one by one from Python.
    The roofline bound is HBM below the ridge point (peak flops / peak
    bytes) and MFMA above it; HBM-bound rows also give a cold-cache figure
    (`cold`), rotating through at least 1 GiB of operand copies."""
    ridge = PEAK_F16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    for w in D.WORKLOADS.values():
        if w.extra:
            continue
        A, B, bias = D.logical_inputs(w)
        dbias = torch.from_numpy(bias).cuda()
        out = torch.empty((w.M, w.N), dtype=torch.float16, device="cuda")
        flops = 2.0 * w.M * w.N * w.K
        nbytes = 2.0 * (w.M * w.K + w.K * w.N + w.M * w.N + w.N)
        hbm = flops / nbytes < ridge
        for layout in w.layouts:
            la, lb = D.LAYOUT_NAMES[layout]
            dA = (torch.from_numpy(A).cuda() if la == D.ROW
                  else torch.from_numpy(np.ascontiguousarray(A.T)).cuda().t())
            dB = (torch.from_numpy(B).cuda() if lb == D.ROW
                  else torch.from_numpy(np.ascontiguousarray(B.T)).cuda().t())
            for acc in w.accum:
                call = lambda a, b, c: (lambda: gba.gemm_bias_act(a, b, dbias, act="relu", accum=acc, out=c))
                ms_eager = time_launches(call(dA, dB, out), args.steps, args.warmup, torch)
                ms = time_graph([call(dA, dB, out)], args.steps, 10, torch)
                tf = flops / (ms * 1e-3) / 1e12
                gbs = nbytes / (ms * 1e-3) / 1e9
                line = {
                    "workload": w.name, "M": w.M, "N": w.N, "K": w.K, "layout": layout, "accum": acc,
                    "tile": gba.select_tile(w.M, w.N, w.K, la, lb, acc), "us": round(ms * 1e3, 2),
                    "us_eager": round(ms_eager * 1e3, 2), "TFLOP/s": round(tf, 1), "GB/s": round(gbs, 1),
                    "roofline": {"bound": "hbm" if hbm else "mfma",
                                 "frac": round(gbs / PEAK_HBM_GBS if hbm else tf / PEAK_F16_TFLOPS, 4)},
                }
                if hbm:
                    nsets = -(-COLD_POOL_BYTES // int(nbytes))
                    sets = cold_operands(torch, dA, dB, w.M, w.N, nsets)
                    ms_cold = time_graph([call(*s) for s in sets], nsets, 3, torch)
                    del sets
                    gbs_cold = nbytes / (ms_cold * 1e-3) / 1e9
                    line["cold"] = {"us": round(ms_cold * 1e3, 2), "GB/s": round(gbs_cold, 1),
                                    "frac": round(gbs_cold / PEAK_HBM_GBS, 4), "sets": nsets}
                print(json.dumps(line), flush=True)


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
    ap.add_argument("--configs", action="store_true",
                    help="instead of the headline line: one JSON line per workload "
                         "configuration (every layout and accumulation it lists) with its "
                         "roofline position")
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
    if args.configs:
        configs(args, np, torch, D, gba)
        return
    w = D.WORKLOADS[args.workload]
    A, B, bias = D.logical_inputs(w)
    dA = torch.from_numpy(A).cuda()                                    # row-major
    dB = torch.from_numpy(np.ascontiguousarray(B.T)).cuda().t()        # column-major
    dbias = torch.from_numpy(bias).cuda()
    out = torch.empty((w.M, w.N), dtype=torch.float16, device="cuda")
    prologue = w.extra.get("prologue")
    P = Q = None
    K2 = 0
    if "second" in w.extra:
        P, Q = D.second_inputs(w)
        K2 = w.extra["K2"]
        dP = torch.from_numpy(P).cuda()
        dQ = torch.from_numpy(np.ascontiguousarray(Q.T)).cuda().t()
    tile = args.tile if args.tile is not None else gba.select_tile(w.M, w.N, w.K + K2)

    if prologue is None and P is None:
        # the headline: gemm_bias_act, and the paper's unfused three-launch chain
        fused = lambda: gba.gemm_bias_act(dA, dB, dbias, act="relu", out=out, tile=tile)
        plain = lambda: gba.gemm_bias_act(dA, dB, None, act="none", out=out, tile=tile)
        unfused = lambda: gba.unfused_gemm_bias_relu(dA, dB, dbias, out=out, tile=tile)
        idiom = "GEMM+bias+ReLU"
        chain = "GEMM, bias add, ReLU"
        plain_leg = "GEMM only (no bias, no activation)"

        # context: the same problem through torch's library path (hipBLASLt
        # GEMM, torch's elementwise kernels), the counterpart of the paper's
        # library baseline
        def lib_chain():
            torch.matmul(dA, dB, out=out)
            out.add_(dbias)
            out.relu_()

        def lib_addmm_relu():
            torch.addmm(dbias, dA, dB, out=out)
            out.relu_()
        library = {"library_gemm": lambda: torch.matmul(dA, dB, out=out),
                   "library_chain": lib_chain, "library_addmm_relu": lib_addmm_relu}
    elif P is None:
        # relu(A).B + bias -> ReLU; unfused: ReLU pass over A, then the fused GEMM
        a_relu = dA.clone()
        fused = lambda: gba.fused_gemm(dA, dB, prologue="relu", bias=dbias, act="relu", out=out,
                                       tile=tile)
        plain = lambda: gba.gemm_bias_act(dA, dB, dbias, act="relu", out=out, tile=tile)

        def unfused():
            gba.relu_(a_relu)
            gba.gemm_bias_act(a_relu, dB, dbias, act="relu", out=out, tile=tile)
        idiom = "ReLU-prologue GEMM+bias+ReLU"
        library = {}
        chain = "ReLU over A, GEMM+bias+ReLU"
        plain_leg = "GEMM+bias+ReLU without the prologue"
    else:
        # A.B + P.Q + bias -> ReLU; unfused: two GEMMs, add, bias add, ReLU
        tmp = torch.empty_like(out)
        fused = lambda: gba.fused_gemm(dA, dB, P=dP, Q=dQ, bias=dbias, act="relu", out=out,
                                       tile=tile)
        plain = lambda: gba.gemm_bias_act(dA, dB, dbias, act="relu", out=out, tile=tile)

        def unfused():
            gba.gemm_bias_act(dA, dB, None, act="none", out=out, tile=tile)
            gba.gemm_bias_act(dP, dQ, None, act="none", out=tmp, tile=tile)
            gba.add_(out, tmp)
            gba.bias_add_(out, dbias)
            gba.relu_(out)
        idiom = "Add(GEMM,GEMM)+bias+ReLU"
        library = {}
        chain = "GEMM, GEMM, add, bias add, ReLU"
        plain_leg = "GEMM+bias+ReLU of A.B alone"

    torch.cuda.synchronize()
    ms = time_launches(fused, args.steps, args.warmup, torch)
    torch.cuda.synchronize()
    if args.fused_only:
        args.no_cpu = True
        ms_plain = ms_unfused = ms_fused2 = float("nan")
        ms_library = {}
    else:
        # the comparison legs get the same warmup, then the fused kernel is
        # timed once more right after the unfused chain
        ms_plain = time_launches(plain, args.steps, args.warmup, torch)
        ms_unfused = time_launches(unfused, args.steps, args.warmup, torch)
        ms_fused2 = time_launches(fused, args.steps, 0, torch)
        ms_library = {k: time_launches(f, args.steps, args.warmup, torch) for k, f in library.items()}

    flops = 2.0 * w.M * w.N * (w.K + K2)
    tflops = flops / (ms * 1e-3) / 1e12
    algo_bytes = 2.0 * (w.M * w.K + w.K * w.N + w.M * K2 + K2 * w.N + w.M * w.N + w.N)
    info = gba.tile_info(tile)

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(w, A, B, bias, P, Q)

    traffic = stored_traffic(w.name)
    metric = METRIC if w.name == HEADLINE else (
        f"fused {idiom} TFLOP/s (2MN(K+K2)/t) fp16 on 1 MI355X; % of MFMA peak")
    line = {
        "metric": metric,
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
        "config": {"workload": f"{w.name}: fused fp16 {idiom} M={w.M} N={w.N} K={w.K}"
                               f"{f' K2={K2}' if K2 else ''}, A row-major, B column-major, "
                               f"fp32 accumulation",
                   "M": w.M, "N": w.N, "K": w.K, **({"K2": K2} if K2 else {}),
                   "layout": "RC", "accum": "f32",
                   "tile": dict(id=tile, **info), "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "mfma", "achieved": round(tflops, 2), "peak": PEAK_F16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(tflops / PEAK_F16_TFLOPS, 4),
                     "traffic": traffic},
        "cpu_baseline": cpu,
        "extra": None if args.fused_only else {
            "frac_of_fp16_peak": round(tflops / PEAK_F16_TFLOPS, 4),
            "fused_ms_second_pass": round(ms_fused2, 5),
            "plain_leg": plain_leg,
            "plain_gemm_ms": round(ms_plain, 5),
            "plain_gemm_tflops": round(2.0 * w.M * w.N * w.K / (ms_plain * 1e-3) / 1e12, 2),
            "unfused_chain": chain,
            "unfused_chain_ms": round(ms_unfused, 5),
            "fused_vs_unfused_speedup": round(ms_unfused / ms, 3),
            "fused_algorithmic_GBps": round(algo_bytes / (ms * 1e-3) / 1e9, 1),
            **({"library_legs": "torch: hipBLASLt GEMM (matmul / addmm with the bias), torch "
                                "bias add and ReLU; context, same inputs",
                **{f"{k}_ms": round(v, 5) for k, v in ms_library.items()},
                "fused_vs_library_chain_speedup": round(ms_library["library_chain"] / ms, 3)}
               if ms_library else {}),
        },
    }
    if args.report:
        with open(args.report, "w") as f:
            json.dump(line, f, indent=1)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
