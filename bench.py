#!/usr/bin/env python3
"""Benchmark of the fused fp16 GEMM + bias + ReLU on one MI355X.

Default workload: M = N = K = 4096, A row-major, B column-major, fp16
uniform[-1,1] inputs, fp32 accumulation, bias + ReLU epilogue.  A step is one
call of the fused kernel; the metric is 2MNK / time in TFLOP/s.

Prints ONE JSON line.  `value` and `ms_per_step` come from K fused launches
back to back (HIP events around the K launches on the stream the library
launches on).  The comparison legs -- the fused kernel again, the plain GEMM,
the unfused three-launch chain (GEMM, bias add, ReLU), the two-launch chain
(GEMM, then bias add + ReLU in one pass) and torch's library path -- are then
timed interleaved: K rounds, one launch of every leg per round, each launch
between its own pair of events, so clock and power drift fall on every leg
alike; each leg reports its median and mean, and the speedups use medians.
The line also carries the fused kernel's roofline position and the CPU
oracle timed on a bounded sample of the same problem.

--workload prologue4096_RC times relu(A).B + bias -> ReLU (against a ReLU
pass over A followed by the fused GEMM), --workload sum4096_RC times
A.B + P.Q + bias -> ReLU with K2 = K (against two GEMMs, an add, a bias add
and a ReLU); their metric counts 2MN(K + K2) flops.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--tile ID]
                    [--report PATH] [--no-cpu]
    python bench.py --configs      # every workload configuration, one line each
    python bench.py --sweep [N]    # the paper's protocol: N random sizes
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


def strip_comments(src):
    """C++ source without its comments and with runs of whitespace collapsed
    (string and character literals are kept as they are)."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c in "\"'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            out.append(" ")
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_digest():
    """sha256 over the HIP sources with their comments removed, to tell
    whether stored counters were taken on the code that is built now."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2006_12645_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".hpp")):
            h.update(name.encode())
            h.update(strip_comments(open(os.path.join(csrc, name), encoding="utf-8").read()).encode())
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


def stored_clock_peak():
    """Observed shader clock (GHz) and the clock-adjusted fp16 MFMA peak
    (TFLOP/s: 256 CUs x 4096 flop per clock x that clock) of the headline
    kernel from the committed rocprofv3 MFMA-utilisation summary, or None
    when absent or taken on different kernel sources."""
    path = os.path.join(PROFILES, f"gemm_bias_act_{HEADLINE}_mfma_util.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_sha = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text)
    row = re.search(r"^\| `gemm_bias_act_fast16<256, 256[^`]*` \|([^\n]*)$", text, re.M)
    if not m_sha or not row or m_sha.group(1) != kernel_source_digest():
        return None
    cols = [c.strip() for c in row.group(1).split("|")]
    try:
        return float(cols[3]), float(cols[4])
    except (IndexError, ValueError):
        return None


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


def cpu_share():
    """Threads the oracle may use on this host: every CPU this process may run
    on, capped by OMP_NUM_THREADS when that is set (the CPU share of a GPU
    box), and the host facts reported beside the figure."""
    try:
        visible = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        visible = os.cpu_count() or 1
    cap = os.environ.get("OMP_NUM_THREADS")
    threads = min(visible, int(cap)) if cap and cap.isdigit() and int(cap) > 0 else visible
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return threads, visible, os.cpu_count(), model


def cpu_baseline(w, A, B, bias, P=None, Q=None, target_s=12.0):
    """The oracle on a bounded sample of output rows of the same problem, on
    every thread of this process's CPU share, plus a single-thread run on the
    1000^3 problem (rows of the ragged workload) for a per-core rate."""
    from oracle import oracle as O
    from paper_2006_12645_amd import datagen as D
    a_st, b_st = D.store(A, D.ROW), D.store(B, D.COL)
    K2 = w.extra.get("K2", 0) if P is not None else 0
    kw = dict(prologue_relu=w.extra.get("prologue") == "relu", bias=bias, act=O.ACT_RELU)
    if P is not None:
        kw.update(second=1, p_store=D.store(P, D.ROW), q_store=D.store(Q, D.COL), K2=K2)
    threads, visible, host_cpus, model = cpu_share()

    def run(rows, nthreads=threads):
        t0 = time.perf_counter()
        O.fused(a_st, D.ROW, b_st, D.COL, w.M, w.N, w.K, rows=rows, nthreads=nthreads, **kw)
        return time.perf_counter() - t0

    rows = list(range(min(w.M, 4 * threads)))
    dt = run(rows)
    # grow the sample to about target_s of work
    nrows = int(min(w.M, max(len(rows), len(rows) * target_s / max(dt, 1e-3))))
    dt = run(list(range(nrows)))
    flops = 2.0 * nrows * w.N * (w.K + K2)
    # one thread on the ragged 1000^3 problem: a per-core rate
    r = D.WORKLOADS["ragged1000"]
    rA, rB, rbias = D.logical_inputs(r)
    r_rows = list(range(r.M))
    t0 = time.perf_counter()
    O.gemm_bias_act(D.store(rA, D.ROW), D.ROW, D.store(rB, D.COL), D.COL, r.M, r.N, r.K, bias=rbias,
                    act=O.ACT_RELU, rows=r_rows, nthreads=1)
    dt1 = time.perf_counter() - t0
    per_core = 2.0 * len(r_rows) * r.N * r.K / dt1 / 1e9
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{nrows} of {w.M} output rows (all {w.N} columns, full reduction "
                      f"K={w.K}{f' + K2={K2}' if K2 else ''}) of the same {w.name} problem, "
                      f"fp64, {dt:.1f} s on {threads} threads",
            "threads": threads, "host_cpus_visible": visible, "host_cpus": host_cpus,
            "cpu_model": model,
            "single_thread": {"GFLOP/s": round(per_core, 3),
                              "sample": f"{len(r_rows)} of 1000 output rows of the 1000^3 ragged "
                                        f"problem, 1 thread, {dt1:.2f} s"}}


def time_interleaved(legs, rounds, warmup, torch):
    """Per-launch times (ms) of every leg, interleaved: `rounds` rounds, each
    launching every leg once in turn, each launch between its own pair of
    events on the current stream (where the library launches).  Returns
    {name: {"median_ms", "mean_ms"}}."""
    names = list(legs)
    for _ in range(warmup):
        for n in names:
            legs[n]()
    torch.cuda.synchronize()
    ev = {n: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(rounds)] for n in names}
    for r in range(rounds):
        for n in names:
            a, b = ev[n][r]
            a.record()
            legs[n]()
            b.record()
    torch.cuda.synchronize()
    out = {}
    for n in names:
        t = sorted(a.elapsed_time(b) for a, b in ev[n])
        mid = len(t) // 2
        med = t[mid] if len(t) % 2 else 0.5 * (t[mid - 1] + t[mid])
        out[n] = {"median_ms": round(med, 5), "mean_ms": round(sum(t) / len(t), 5)}
    return out


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


def graph_legs(legs, launches, rounds, torch):
    """Median ms per launch of every leg: each leg's `launches` calls (cycling
    through its list of callables) captured in one HIP graph, then `rounds`
    rounds replaying every leg's graph once in turn, each replay between its
    own pair of events (interleaved, so drift falls on every leg alike)."""
    graphs = {}
    for name, fns in legs.items():
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
        graphs[name] = g
    torch.cuda.synchronize()
    ev = {n: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(rounds)] for n in graphs}
    for r in range(rounds):
        for n, g in graphs.items():
            a, b = ev[n][r]
            a.record()
            g.replay()
            b.record()
    torch.cuda.synchronize()
    out = {}
    for n in graphs:
        t = sorted(a.elapsed_time(b) / launches for a, b in ev[n])
        mid = len(t) // 2
        out[n] = t[mid] if len(t) % 2 else 0.5 * (t[mid - 1] + t[mid])
    del graphs
    return out


def chain_legs(gba, dA, dB, dbias, out, acc="f32", tile=None):
    """The fused call and the two unfused chains on the same operands."""
    return {
        "fused": lambda: gba.gemm_bias_act(dA, dB, dbias, act="relu", accum=acc, out=out, tile=tile),
        "chain3": lambda: (gba.gemm_bias_act(dA, dB, None, act="none", accum=acc, out=out, tile=tile),
                           gba.bias_add_(out, dbias), gba.relu_(out)),
        "chain2": lambda: (gba.gemm_bias_act(dA, dB, None, act="none", accum=acc, out=out, tile=tile),
                           gba.bias_act_(out, dbias, "relu")),
    }


def configs(args, np, torch, D, gba):
    """Every single-product workload configuration: layouts x accumulations,
    the library's tile choice.  `us` is device time per launch from a
    captured graph of back-to-back launches on the same (cache-resident)
    operands, timed interleaved with the two unfused chains on the same
    operands (`chain3_us`: GEMM, bias add, ReLU; `chain2_us`: GEMM, then bias
    add and ReLU in one pass) and their speedups; `us_eager` the fused
    launches issued one by one from Python.  The roofline bound is HBM below
    the ridge point (peak flops / peak bytes) and MFMA above it; HBM-bound
    rows also give cold-cache figures (`cold`), rotating through at least
    1 GiB of operand copies, for the fused kernel and both chains."""
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
                legs = chain_legs(gba, dA, dB, dbias, out, acc)
                ms_eager = time_launches(legs["fused"], args.steps, args.warmup, torch)
                if args.fused_only:
                    # eager fused launches only (for counter runs of the profiler)
                    print(json.dumps({"workload": w.name, "M": w.M, "N": w.N, "K": w.K, "layout": layout,
                                      "accum": acc, "tile": gba.select_tile(w.M, w.N, w.K, la, lb, acc),
                                      "us_eager": round(ms_eager * 1e3, 2)}), flush=True)
                    continue
                t = graph_legs({k: [f] for k, f in legs.items()}, args.steps, 10, torch)
                ms = t["fused"]
                tf = flops / (ms * 1e-3) / 1e12
                gbs = nbytes / (ms * 1e-3) / 1e9
                line = {
                    "workload": w.name, "M": w.M, "N": w.N, "K": w.K, "layout": layout, "accum": acc,
                    "tile": gba.select_tile(w.M, w.N, w.K, la, lb, acc), "us": round(ms * 1e3, 2),
                    "us_eager": round(ms_eager * 1e3, 2), "TFLOP/s": round(tf, 1), "GB/s": round(gbs, 1),
                    "roofline": {"bound": "hbm" if hbm else "mfma",
                                 "frac": round(gbs / PEAK_HBM_GBS if hbm else tf / PEAK_F16_TFLOPS, 4)},
                    "chain3_us": round(t["chain3"] * 1e3, 2), "chain2_us": round(t["chain2"] * 1e3, 2),
                    "speedup_vs_chain3": round(t["chain3"] / ms, 3),
                    "speedup_vs_chain2": round(t["chain2"] / ms, 3),
                }
                if hbm:
                    nsets = -(-COLD_POOL_BYTES // int(nbytes))
                    sets = cold_operands(torch, dA, dB, w.M, w.N, nsets)
                    cold_legs = {}
                    for k in ("fused", "chain3", "chain2"):
                        cold_legs[k] = [chain_legs(gba, a, b, dbias, c, acc)[k] for a, b, c in sets]
                    tc = graph_legs(cold_legs, nsets, 3, torch)
                    del sets, cold_legs
                    gbs_cold = nbytes / (tc["fused"] * 1e-3) / 1e9
                    line["cold"] = {"us": round(tc["fused"] * 1e3, 2), "GB/s": round(gbs_cold, 1),
                                    "frac": round(gbs_cold / PEAK_HBM_GBS, 4), "sets": nsets,
                                    "chain3_us": round(tc["chain3"] * 1e3, 2),
                                    "chain2_us": round(tc["chain2"] * 1e3, 2),
                                    "speedup_vs_chain3": round(tc["chain3"] / tc["fused"], 3),
                                    "speedup_vs_chain2": round(tc["chain2"] / tc["fused"], 3)}
                print(json.dumps(line), flush=True)


def sweep(args, np, torch, D, gba):
    """The paper's evaluation protocol on MI355X: random problem sizes, each a
    multiple of 128 up to 4096 (datagen.sweep_shapes), RC layout, fp32
    accumulation, uniform[-1,1] data; per size the fused kernel (library tile
    choice) against the unfused three-launch chain (the paper's baseline:
    GEMM, bias add, ReLU), the two-launch chain and, as context, torch's
    library path (hipBLASLt GEMM, then add and ReLU), all graph-timed and
    interleaved.  One JSON line per size, then a summary line: sizes where
    fused wins, peak, worst, geometric and arithmetic mean speedup."""
    import math
    shapes = D.sweep_shapes(count=args.sweep)
    rows = []
    for idx, (M, N, K) in enumerate(shapes):
        A, B, bias = D.random_problem(900000 + 10 * idx, M, N, K)
        dA = torch.from_numpy(A).cuda()
        dB = torch.from_numpy(np.ascontiguousarray(B.T)).cuda().t()
        dbias = torch.from_numpy(bias).cuda()
        out = torch.empty((M, N), dtype=torch.float16, device="cuda")
        legs = chain_legs(gba, dA, dB, dbias, out)
        legs["library_chain"] = lambda: (torch.matmul(dA, dB, out=out), out.add_(dbias), out.relu_())
        t = graph_legs({k: [f] for k, f in legs.items()}, 10, 5, torch)
        line = {"M": M, "N": N, "K": K, "tile": gba.select_tile(M, N, K),
                "fused_us": round(t["fused"] * 1e3, 2),
                "TFLOP/s": round(2.0 * M * N * K / (t["fused"] * 1e-3) / 1e12, 1),
                **{f"{k}_us": round(t[k] * 1e3, 2) for k in ("chain3", "chain2", "library_chain")},
                **{f"speedup_vs_{k}": round(t[k] / t["fused"], 3) for k in ("chain3", "chain2",
                                                                            "library_chain")}}
        rows.append(line)
        print(json.dumps(line), flush=True)
        del dA, dB, out
    summary = {"sweep": f"{len(rows)} random sizes, multiples of 128 up to 4096, RC, fp32 accumulation, "
                        "GEMM+bias+ReLU"}
    for k in ("chain3", "chain2", "library_chain"):
        sp = [r[f"speedup_vs_{k}"] for r in rows]
        summary[k] = {"wins": sum(1 for x in sp if x > 1.0), "of": len(sp), "peak": max(sp),
                      "worst": min(sp), "geomean": round(math.exp(sum(map(math.log, sp)) / len(sp)), 3),
                      "mean": round(sum(sp) / len(sp), 3)}
    print(json.dumps(summary), flush=True)


THIN_SHAPES = ([(M, N, K) for M in (32, 64, 128, 256) for N in (2048, 4096, 8192) for K in (512, 1024, 2048, 4096)] +
               [(4096, 128, 1024), (8192, 256, 2048), (2048, 64, 4096), (512, 2048, 1024), (1024, 1024, 4096)])


SHORTK_SHAPES = [(M, N, K) for (M, N) in ((1024, 2048), (2048, 2048), (2048, 3072), (3072, 2048), (2560, 3072),
                                           (3072, 3072), (2944, 3200), (3456, 3456), (3840, 3840), (4096, 4096),
                                           (4096, 2048), (1536, 4096)) for K in (64, 128, 192, 256)]


def rule_tile(gba, M, N, K, layout, accum, prologue):
    """The tile the library chooses for a one-product request of this shape,
    layout, accumulation and prologue (host-only)."""
    la = gba.GBA_ROW_MAJOR if layout[0] == "R" else gba.GBA_COL_MAJOR
    lb = gba.GBA_ROW_MAJOR if layout[1] == "R" else gba.GBA_COL_MAJOR
    return gba.select_tile(M, N, K, la, lb, accum=accum, prologue=prologue)


def tile_sweep(args, np, torch, D, gba):
    """Every tile against the library's choice: for each shape of a set (the
    thin set, or the workload shapes plus 40 random multiples of 128 for a
    seed), every tile that fits is graph-timed warm (the same operands each
    launch) and with operands from HBM (launches rotate over copies of the
    operands spanning at least 1 GiB).  One JSON line per shape, then a
    summary: the library's choice against the per-shape best tile, in total
    time over the set."""
    if args.tile_sweep == "thin":
        shapes = THIN_SHAPES
    elif args.tile_sweep == "shortk":
        shapes = SHORTK_SHAPES
    else:
        shapes = ([(4096, 4096, 4096), (8192, 4096, 1024), (8192, 1024, 4096), (1024, 1024, 1024),
                   (1000, 1000, 1000), (32, 4096, 1024), (128, 4096, 1024), (256, 4096, 1024),
                   (2048, 2048, 2048), (64, 512, 32768), (512, 512, 8192)] +
                  D.sweep_shapes(int(args.tile_sweep), 40))
    lay, acc, pro = args.layout, args.accum, args.prologue
    operand = lambda x, colmajor: x.t().contiguous().t() if colmajor else x

    def graph(fn, n):
        fn(0)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(n):
                fn(i)
        g.replay()
        torch.cuda.synchronize()
        return g, n

    def run(g, n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n * 1000

    tot = {"rule": [0.0, 0.0], "best": [0.0, 0.0]}
    for idx, (M, N, K) in enumerate(shapes):
        nc = max(2, min(64, (1 << 30) // ((M * K + N * K) * 2) + 1))
        gen = torch.Generator(device="cuda").manual_seed(770000 + idx)
        As = [operand(torch.rand(M, K, generator=gen, device="cuda").half() - 0.5, lay[0] == "C") for _ in range(nc)]
        Bs = [operand(torch.rand(K, N, generator=gen, device="cuda").half() - 0.5, lay[1] == "C") for _ in range(nc)]
        bias = torch.rand(N, generator=gen, device="cuda").half()
        out = torch.empty(M, N, dtype=torch.float16, device="cuda")
        kw = dict(bias=bias, out=out, accum=acc, prologue="relu" if pro else None, workspace=None)
        warm, cold = {}, {}
        for t in range(gba.num_tiles()):
            info = gba.tile_info(t)
            if info["bm"] > M or info["bn"] > N or (acc == "f16" and info["split_k"] > 1):
                continue
            gw = graph(lambda i, t=t: gba.fused_gemm(As[0], Bs[0], tile=t, **kw), 10)
            gc = graph(lambda i, t=t: gba.fused_gemm(As[i % nc], Bs[i % nc], tile=t, **kw), max(10, nc))
            warm[t] = round(min(run(*gw) for _ in range(5)), 2)
            cold[t] = round(min(run(*gc) for _ in range(3)), 2)
        rule = rule_tile(gba, M, N, K, lay, acc, pro)
        print(json.dumps({"M": M, "N": N, "K": K, "rule": rule, "warm": warm, "cold": cold}), flush=True)
        if rule in warm:
            tot["rule"][0] += warm[rule]
            tot["rule"][1] += cold[rule]
            tot["best"][0] += min(warm.values())
            tot["best"][1] += min(cold.values())
        del As, Bs, out
        torch.cuda.empty_cache()
    print(json.dumps({"tile_sweep": args.tile_sweep, "layout": lay, "accum": acc, "prologue": pro,
                      "shapes": len(shapes),
                      "rule_over_best_warm": round(tot["rule"][0] / tot["best"][0], 4),
                      "rule_over_best_cold": round(tot["rule"][1] / tot["best"][1], 4)}), flush=True)


def ksweep(args, np, torch, D, gba):
    """Fixed cost and cost per reduction step of the fused kernel: at fixed
    M x N (the two MLP shapes, 1024^2 and 4096^2, RC, fp32 accumulation,
    the library's tile choice) the reduction length K runs over 256..8192,
    each point graph-timed (median of interleaved replays), and a least
    squares line time = fixed + per_step * K/64 is fitted.  One JSON line per
    point and one per fit."""
    for (M, N) in [(8192, 4096), (8192, 1024), (1024, 1024), (4096, 4096)]:
        ks = [256, 512, 1024, 2048, 4096, 8192]
        legs, tiles = {}, {}
        keep = []
        for K in ks:
            A, B, bias = D.random_problem(880000 + K, M, N, K)
            dA = torch.from_numpy(A).cuda()
            dB = torch.from_numpy(np.ascontiguousarray(B.T)).cuda().t()
            dbias = torch.from_numpy(bias).cuda()
            out = torch.empty((M, N), dtype=torch.float16, device="cuda")
            keep.append((dA, dB, dbias, out))
            tiles[K] = gba.select_tile(M, N, K)
            legs[str(K)] = [lambda dA=dA, dB=dB, dbias=dbias, out=out, t=tiles[K]:
                            gba.gemm_bias_act(dA, dB, dbias, act="relu", out=out, tile=t)]
        t = graph_legs(legs, 20, 7, torch)
        xs = [K / 64.0 for K in ks]
        ys = [t[str(K)] * 1e3 for K in ks]
        for K, y in zip(ks, ys):
            print(json.dumps({"M": M, "N": N, "K": K, "tile": tiles[K], "us": round(y, 2),
                              "TFLOP/s": round(2.0 * M * N * K / (y * 1e-6) / 1e12, 1)}), flush=True)
        # the fit uses the points that share the K = 4096 point's tile
        sel = [(x, y) for K, x, y in zip(ks, xs, ys) if tiles[K] == tiles[4096]]
        n = len(sel)
        mx = sum(x for x, _ in sel) / n
        my = sum(y for _, y in sel) / n
        slope = sum((x - mx) * (y - my) for x, y in sel) / sum((x - mx) ** 2 for x, _ in sel)
        print(json.dumps({"fit": f"{M}x{N}", "tile": tiles[4096], "points": n,
                          "fixed_us": round(my - slope * mx, 2), "per_step_us": round(slope, 4),
                          "step_TFLOP/s": round(2.0 * M * N * 64 / (slope * 1e-6) / 1e12, 1)}), flush=True)
        if (M, N) == (4096, 4096):
            # context: the same sweep through torch's library GEMM (hipBLASLt,
            # no epilogue) on the same operands
            lib = {str(K): [lambda dA=dA, dB=dB, out=out: torch.matmul(dA, dB, out=out)]
                   for K, (dA, dB, _, out) in zip(ks, keep)}
            tl = graph_legs(lib, 20, 7, torch)
            ly = [tl[str(K)] * 1e3 for K in ks]
            lmy = sum(ly) / len(ly)
            lmx = sum(xs) / len(xs)
            ls = sum((x - lmx) * (y - lmy) for x, y in zip(xs, ly)) / sum((x - lmx) ** 2 for x in xs)
            print(json.dumps({"fit": f"{M}x{N} library GEMM (hipBLASLt, context)", "points": len(ks),
                              "us": {str(K): round(y, 2) for K, y in zip(ks, ly)},
                              "fixed_us": round(lmy - ls * lmx, 2), "per_step_us": round(ls, 4),
                              "step_TFLOP/s": round(2.0 * M * N * 64 / (ls * 1e-6) / 1e12, 1)}), flush=True)
        del keep


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
                         "roofline position and fused-vs-unfused speedups")
    ap.add_argument("--ksweep", action="store_true",
                    help="instead of the headline line: fixed cost and cost per reduction step "
                         "of the fused kernel from a sweep of K at fixed M x N")
    ap.add_argument("--sweep", type=int, nargs="?", const=100, default=0, metavar="N",
                    help="instead of the headline line: the paper's protocol over N random "
                         "sizes (default 100), one line per size and a summary line")
    ap.add_argument("--tile-sweep", default=None, metavar="SET",
                    help="instead of the headline line: every tile against the library's choice "
                         "over a shape set ('thin', 'shortk', or a seed for the workload shapes "
                         "plus 40 random ones), warm and with operands from HBM")
    ap.add_argument("--layout", default="RC", choices=["RR", "RC", "CR", "CC"], help="with --tile-sweep")
    ap.add_argument("--accum", default="f32", choices=["f32", "f16"], help="with --tile-sweep")
    ap.add_argument("--prologue", action="store_true", help="with --tile-sweep: ReLU prologue on A")
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
    if args.sweep:
        sweep(args, np, torch, D, gba)
        return
    if args.ksweep:
        ksweep(args, np, torch, D, gba)
        return
    if args.tile_sweep:
        tile_sweep(args, np, torch, D, gba)
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

    # the comparison legs, timed interleaved after the headline window
    legs = {}
    if prologue is None and P is None:
        # the headline: gemm_bias_act, the plain GEMM, the paper's unfused
        # three-launch chain and the two-launch variant
        fused = lambda: gba.gemm_bias_act(dA, dB, dbias, act="relu", out=out, tile=tile)
        legs["plain"] = lambda: gba.gemm_bias_act(dA, dB, None, act="none", out=out, tile=tile)
        legs["unfused_chain"] = lambda: gba.unfused_gemm_bias_relu(dA, dB, dbias, out=out, tile=tile)
        legs["unfused_chain2"] = lambda: gba.unfused_gemm_bias_relu_2(dA, dB, dbias, out=out, tile=tile)
        idiom = "GEMM+bias+ReLU"
        chain = "GEMM, bias add, ReLU"
        chain2 = "GEMM, then bias add and ReLU in one pass"
        plain_leg = "GEMM only (no bias, no activation)"
        # context: the same problem through torch's library path (hipBLASLt
        # GEMM, torch's elementwise kernels), the counterpart of the paper's
        # library baseline
        legs["library_gemm"] = lambda: torch.matmul(dA, dB, out=out)
        legs["library_chain"] = lambda: (torch.matmul(dA, dB, out=out), out.add_(dbias), out.relu_())
        legs["library_addmm_relu"] = lambda: (torch.addmm(dbias, dA, dB, out=out), out.relu_())
    elif P is None:
        # relu(A).B + bias -> ReLU; unfused: ReLU pass over A, then the fused GEMM
        a_relu = dA.clone()
        fused = lambda: gba.fused_gemm(dA, dB, prologue="relu", bias=dbias, act="relu", out=out,
                                       tile=tile)
        legs["plain"] = lambda: gba.gemm_bias_act(dA, dB, dbias, act="relu", out=out, tile=tile)

        def unfused():
            gba.relu_(a_relu)
            gba.gemm_bias_act(a_relu, dB, dbias, act="relu", out=out, tile=tile)
        legs["unfused_chain"] = unfused
        idiom = "ReLU-prologue GEMM+bias+ReLU"
        chain = "ReLU over A, GEMM+bias+ReLU"
        chain2 = None
        plain_leg = "GEMM+bias+ReLU without the prologue"
    else:
        # A.B + P.Q + bias -> ReLU; unfused: two GEMMs, add, bias add, ReLU
        tmp = torch.empty_like(out)
        fused = lambda: gba.fused_gemm(dA, dB, P=dP, Q=dQ, bias=dbias, act="relu", out=out,
                                       tile=tile)
        legs["plain"] = lambda: gba.gemm_bias_act(dA, dB, dbias, act="relu", out=out, tile=tile)

        def unfused():
            gba.gemm_bias_act(dA, dB, None, act="none", out=out, tile=tile)
            gba.gemm_bias_act(dP, dQ, None, act="none", out=tmp, tile=tile)
            gba.add_(out, tmp)
            gba.bias_add_(out, dbias)
            gba.relu_(out)

        def unfused2():
            gba.gemm_bias_act(dA, dB, None, act="none", out=out, tile=tile)
            gba.gemm_bias_act(dP, dQ, None, act="none", out=tmp, tile=tile)
            gba.add_(out, tmp)
            gba.bias_act_(out, dbias, "relu")
        legs["unfused_chain"] = unfused
        legs["unfused_chain2"] = unfused2
        idiom = "Add(GEMM,GEMM)+bias+ReLU"
        chain = "GEMM, GEMM, add, bias add, ReLU"
        chain2 = "GEMM, GEMM, add, then bias add and ReLU in one pass"
        plain_leg = "GEMM+bias+ReLU of A.B alone"

    # The comparison legs first (interleaved), then the headline window:
    # `warmup` untimed and `steps` timed fused launches back to back, on a
    # GPU that is already running (not ramping up from idle).
    inter = {}
    if args.fused_only:
        args.no_cpu = True
    else:
        inter = time_interleaved({"fused": fused, **legs}, args.steps, args.warmup, torch)
    torch.cuda.synchronize()
    ms = time_launches(fused, args.steps, args.warmup, torch)
    torch.cuda.synchronize()

    flops = 2.0 * w.M * w.N * (w.K + K2)
    tflops = flops / (ms * 1e-3) / 1e12
    algo_bytes = 2.0 * (w.M * w.K + w.K * w.N + w.M * K2 + K2 * w.N + w.M * w.N + w.N)
    info = gba.tile_info(tile)

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(w, A, B, bias, P, Q)

    traffic = stored_traffic(w.name)
    clk = stored_clock_peak()
    metric = METRIC if w.name == HEADLINE else (
        f"fused {idiom} TFLOP/s (2MN(K+K2)/t) fp16 on 1 MI355X; % of MFMA peak")
    extra = None
    if inter:
        f_med = inter["fused"]["median_ms"]
        extra = {
            "frac_of_fp16_peak": round(tflops / PEAK_F16_TFLOPS, 4),
            "interleaved": "per-launch event pairs, one launch of every leg per round, "
                           f"{args.steps} rounds; speedups are ratios of medians",
            "legs": inter,
            "plain_leg": plain_leg,
            "plain_gemm_tflops": round(2.0 * w.M * w.N * w.K / (inter["plain"]["median_ms"] * 1e-3) / 1e12, 2),
            "unfused_chain": chain,
            "fused_vs_unfused_speedup": round(inter["unfused_chain"]["median_ms"] / f_med, 3),
            **({"unfused_chain2": chain2,
                "fused_vs_unfused2_speedup": round(inter["unfused_chain2"]["median_ms"] / f_med, 3)}
               if chain2 else {}),
            "fused_algorithmic_GBps": round(algo_bytes / (ms * 1e-3) / 1e9, 1),
            **({"clock_adjusted_peak": {
                    "sclk_GHz": clk[0], "peak_TFLOPs": clk[1], "frac": round(tflops / clk[1], 4),
                    "source": f"profiles/gemm_bias_act_{HEADLINE}_mfma_util.md (GRBM_GUI_ACTIVE over "
                              "the dispatch time, another run on another box)"}}
               if clk and w.name == HEADLINE else {}),
            **({"library_legs": "torch: hipBLASLt GEMM (matmul / addmm with the bias), torch "
                                "bias add and ReLU; context, same inputs",
                "fused_vs_library_chain_speedup": round(inter["library_chain"]["median_ms"] / f_med, 3),
                "fused_vs_library_gemm": round(inter["library_gemm"]["median_ms"] / f_med, 3)}
               if "library_chain" in inter else {}),
        }
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
        "extra": extra,
    }
    if args.report:
        with open(args.report, "w") as f:
            json.dump(line, f, indent=1)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
