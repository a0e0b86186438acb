#!/usr/bin/env python3
"""Benchmark: one per-rank training step of SBP linear layers on one MI355X.

Workload (the step): the 96 linear layers of a 24-layer Transformer (hidden
1024, ffn 4096, 16 heads, 8192 global tokens, p = 8 devices), each with its
own seeded SBP signature from {DP (S(0),B)->S(0), COL (B,S(1))->S(1),
KS (S(1),S(0))->P}; rank 0's share runs: every forward in layer order, then
the backward-data and backward-weight products of each linear in reverse
order, 288 local products on one HIP stream. Inputs are seeded
synthetic tensors resident in HBM (the global X, W and dY of every linear;
the library reads rank 0's shares in place).

`value` is whole-step TFLOP/s (sum of 2 m n k over the 288 local products,
divided by the measured step time); the step is replayed from a HIP graph
captured once after warm-up. The backward products of each linear go
through one sbp_linear_bwd call (they are independent and share one
launch). Per-kernel durations come from HIP events that the library records
with each kernel dispatch, in a separate eager pass over the same steps.

Prints one JSON line. Only one GPU: --gpus above 1 exits with a message.
"""
from __future__ import annotations

import argparse
import collections
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

BF16_PEAK_TFLOPS = 2516.6      # 256 CU x 2.4 GHz x 4096 flop/clk (dense)
HBM_PEAK_GBS = 8000.0
RIDGE = BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)

OPS = ("fwd", "bwd_data", "bwd_weight")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """sha256 over the library's kernel and host sources (sorted by name)."""
    import hashlib
    d = os.path.join(ROOT, "paper_2301_06813_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(d)):
        if f.endswith((".h", ".hip", ".cpp")):
            h.update(f.encode())
            with open(os.path.join(d, f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()


def counted_traffic(kernel: str):
    """HBM bytes per dispatch of `kernel` from the committed rocprofv3 counter
    summary (FETCH_SIZE and WRITE_SIZE, scaled by a plain copy), or None if
    the summary is missing, lacks this kernel, or was taken from other
    kernel sources."""
    path = os.path.join(ROOT, "profiles", "gemm_bf16_transformer_step_hbm_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    if "Kernel sources sha256: " + kernel_source_hash() not in text:
        return None
    for line in text.splitlines():
        cells = [c.strip().strip("`") for c in line.split("|")]
        if len(cells) > 5 and cells[1].replace("sbpk::", "") == kernel:
            return float(cells[5]) * 1e6
    return None


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, seconds):
    """The oracle's plain fp32 triple loop (fp32 accumulator, increasing
    reduction index) on a bounded sample of the same step: leading output
    rows of every product of the first four layers' 16 linears, timed on the
    host cores; plus workload 1 (every signature, rank and product of the
    tiny fp32 linear) on one thread."""
    import oracle
    from paper_2301_06813_amd import inputs, workloads
    sig_id = {"DP": oracle.DP, "COL": oracle.COL, "KS": oracle.KS}
    op_id = {"fwd": oracle.FWD, "bwd_data": oracle.BWD_DATA, "bwd_weight": oracle.BWD_WEIGHT}
    oracle.build()
    threads = oracle.threads()
    lins = wl.linears[:16]
    host = []
    for lin in lins:
        X, W, dY = workloads.make_tensors(lin, wl.dtype, "cuda")
        host.append(tuple(inputs.host_bits(t) for t in (X, W, dY)))
        del X, W, dY

    def run(nrows):
        fl, t0 = 0.0, time.perf_counter()
        for lin, (Xh, Wh, dYh) in zip(lins, host):
            for op in OPS:
                rows, cols, _, _ = oracle.out_shape(sig_id[lin.sig], op_id[op], lin.M, lin.K,
                                                    lin.N, wl.p, 0)
                nr = min(nrows, rows)
                oracle.linear_f32(sig_id[lin.sig], op_id[op], Xh, Wh, dYh, wl.p, 0,
                                  rows=range(0, nr))
                # every local product of a linear is 2 M K N / p flops
                fl += lin.flops_per_op(wl.p) * nr / rows
        return fl, time.perf_counter() - t0

    # calibrate: double the row sample until it takes a measurable time, then
    # scale it to the requested duration
    nrows, t1 = 1, 0.0
    while True:
        _, t1 = run(nrows)
        if t1 >= min(1.0, seconds / 4) or nrows >= 8192:
            break
        nrows *= 2
    nrows = max(1, min(8192, int(nrows * seconds / max(t1, 1e-6))))
    fl, t = run(nrows)

    # workload 1 on one thread: 3 signatures x 4 ranks x 3 products
    oracle.set_threads(1)
    try:
        fl1, t_1 = 0.0, time.perf_counter()
        for w1 in workloads.tiny_fp32():
            (lin,) = w1.linears
            Xh, Wh, dYh = (inputs.host_bits(t_) for t_ in workloads.make_tensors(
                lin, torch_float32(), "cpu"))
            for r in w1.ranks:
                for op in OPS:
                    oracle.linear_f32(sig_id[lin.sig], op_id[op], Xh, Wh, dYh, w1.p, r)
                    fl1 += lin.flops_per_op(w1.p)
        t_1 = time.perf_counter() - t_1
    finally:
        oracle.set_threads(threads)
    return {"value": fl / t / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": "first %d output rows of each of the 48 local products of layers 0-3 "
                      "(qkv/out/fc1/fc2 x fwd/bwd_data/bwd_weight), rank 0, plain fp32 "
                      "triple loop; %.3g GFLOP in %.1f s" % (nrows, fl / 1e9, t),
            "cpu_model": cpu_model(), "threads_available": len(os.sched_getaffinity(0)),
            "workload1_single_thread": {"ms": t_1 * 1e3, "gflops": fl1 / t_1 / 1e9,
                                        "products": 36, "threads": 1}}


def torch_float32():
    import torch
    return torch.float32


TIMED_REPLAYS = 10


def time_replays(torch, g, reps, n=TIMED_REPLAYS):
    """Per-call time of a graph of `reps` calls: the mean over n replays from
    one event pair around them all, and each replay's own (events between
    consecutive replays), in us per call."""
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    ev[0].record()
    for i in range(n):
        g.replay()
        ev[i + 1].record()
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) * 1e3 / reps for i in range(n)]
    return ev[0].elapsed_time(ev[n]) * 1e3 / (n * reps), per


def report_workload(cid, ranks, reps):
    """Per-call throughput of workload cid (2: Transformer FFN shard, 3: attention
    projections, 4: VGG head, 6: a Transformer layer under the 3-D rule on a
    2 x 2 x 2 mesh; its ranks are mesh coordinates) on the given ranks: each call (the forward product,
    or both backward products in one sbp_linear_bwd call) is replayed from a HIP
    graph over three rotating sets of its global inputs (more than the 256 MB
    Infinity Cache for the larger workloads). Returns one dict for the JSON line."""
    import torch
    from paper_2301_06813_amd import linear, sbp, workloads
    wl = {2: workloads.ffn_shard, 3: workloads.attention_dp, 4: workloads.vgg_head,
          6: workloads.transformer_3d}[cid]()
    stream = torch.cuda.Stream()
    rows = []
    for lin in wl.linears:
        sets = []
        for _ in range(3):
            X, W, dY = workloads.make_tensors(lin, wl.dtype, "cuda")
            sets.append((X, W, dY))
        for r in ranks:
            L = linear.layouts_for(lin, wl, r)
            outs = [{op: linear.alloc_out_L(op, L, lin.M, lin.K, lin.N, wl.dtype, "cuda")
                     for op in OPS} for _ in sets]
            for kind in ("fwd", "bwd"):
                it = [0]

                def call():
                    i = it[0] % len(sets)
                    it[0] += 1
                    X, W, dY = sets[i]
                    o = outs[i]
                    if kind == "fwd":
                        linear.run_L("fwd", L, X, W, dY, o["fwd"], stream.cuda_stream)
                    else:
                        linear.run_bwd_L(L, X, W, dY, o["bwd_data"], o["bwd_weight"],
                                         stream.cuda_stream)
                with torch.cuda.stream(stream):
                    call()
                    torch.cuda.synchronize()
                    g = torch.cuda.CUDAGraph()
                    with torch.cuda.graph(g, stream=stream):
                        for _ in range(reps):
                            call()
                g.replay()
                torch.cuda.synchronize()
                us, per = time_replays(torch, g, reps)
                ops = ("fwd",) if kind == "fwd" else ("bwd_data", "bwd_weight")
                prods, fl, by = [], 0.0, 0.0
                for op in ops:
                    m, n = outs[0][op].shape
                    k = {"fwd": linear.shard(L["x"], lin.M, lin.K).cols,
                         "bwd_data": linear.shard(L["dy"], lin.M, lin.N).cols,
                         "bwd_weight": linear.shard(L["x"], lin.M, lin.K).rows}[op]
                    ob = 4 if outs[0][op].dtype == torch.float32 else 2
                    prods.append("%s %dx%dx%d%s" % (op, m, n, k, " fp32" if ob == 4 else ""))
                    fl += 2.0 * m * n * k
                    by += 2.0 * (m * k + k * n) + ob * m * n
                rank = list(r) if wl.mesh else r
                rows.append({"linear": lin.name, "sig": lin.sig, "rank": rank, "call": kind,
                             "products": prods, "us": us, "us_stats": step_stats(per),
                             "tflops": fl / us / 1e6,
                             "pct_of_bf16_peak": 100.0 * fl / us / 1e6 / BF16_PEAK_TFLOPS,
                             "algorithmic_gbs": by / us / 1e3,
                             "roofline_min_us": max(fl / BF16_PEAK_TFLOPS / 1e6,
                                                    by / HBM_PEAK_GBS / 1e3)})
                log("%-4s %-4s r%s %-3s %7.1f us %6.0f TFLOP/s %s" % (
                    lin.name, lin.sig, r, kind, us, fl / us / 1e6, ", ".join(prods)))
        del sets
        torch.cuda.empty_cache()
    first = list(ranks[0]) if wl.mesh else ranks[0]
    tot_us = sum(x["us"] for x in rows if x["rank"] == first)
    tot_fl = sum(x["tflops"] * x["us"] * 1e6 for x in rows if x["rank"] == first)
    return {"metric": "local-shard GEMM TFLOP/s (fwd+bwd) per SBP signature; % of bf16 MFMA peak",
            "value": tot_fl / tot_us / 1e6, "unit": "TFLOP/s", "n_gpus": 1,
            "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": wl.name, "p": wl.p,
                       "ranks": [list(r) for r in ranks] if wl.mesh else list(ranks),
                       **({"mesh": list(wl.mesh),
                           "factors": list(wl.linears[0].factors)} if wl.mesh else {}),
                       "mode": "per-call hip_graph replay"},
            "calls": rows}


def report_attention(r, reps):
    """Per-call throughput of workload 7 (the attention core under a head
    split) on device r: the four attention calls, each replayed from a HIP
    graph over three rotating input sets. Returns one dict for the JSON line."""
    import torch
    from paper_2301_06813_amd import inputs, sbp, workloads
    wc = workloads.attention_core()
    B, H, S, D, p = wc.batch, wc.heads, wc.seq, wc.head_dim, wc.p
    h0, hr = sbp_split(H, p, r)
    stream = torch.cuda.Stream()
    sets = []
    for i in range(3):
        sd = wc.seed_base + 10 * i
        act = inputs.randn((B, S, 3, H, D), 1.0, sd + 1, torch.bfloat16, "cuda")
        logits = inputs.randn((B, hr, S, S), 1.0, sd + 2, torch.float32, "cuda")
        t = dict(Q=act[:, :, 0].permute(0, 2, 1, 3), K=act[:, :, 1].permute(0, 2, 1, 3),
                 V=act[:, :, 2].permute(0, 2, 1, 3), act=act,
                 P=torch.softmax(logits, -1).to(torch.bfloat16),
                 dS=inputs.randn((B, hr, S, S), 1.0, sd + 3, torch.bfloat16, "cuda"),
                 dO=inputs.randn((B, hr, S, D), 1.0, sd + 4, torch.bfloat16, "cuda"))
        del logits
        for k, shp in (("S", (B, hr, S, S)), ("O", (B, hr, S, D)), ("dQ", (B, hr, S, D)),
                       ("dK", (B, hr, S, D)), ("dP", (B, hr, S, S)), ("dV", (B, hr, S, D))):
            t["o_" + k] = torch.empty(shp, dtype=torch.bfloat16, device="cuda")
        sets.append(t)
    G = lambda x: sbp.view4(x, sbp.SBP_GLOBAL)
    L = lambda x: sbp.view4(x, sbp.SBP_LOCAL)
    calls = {
        "scores": (lambda t, s: sbp.sbp_attn_scores(G(t["Q"]), G(t["K"]), L(t["o_S"]), p, r, s),
                   [("S = Q K^T", S, S, D)]),
        "context": (lambda t, s: sbp.sbp_attn_context(L(t["P"]), G(t["V"]), L(t["o_O"]), p, r, s),
                    [("O = P V", S, D, S)]),
        "scores_bwd": (lambda t, s: sbp.sbp_attn_scores_bwd(L(t["dS"]), G(t["Q"]), G(t["K"]),
                                                            L(t["o_dQ"]), L(t["o_dK"]), p, r, s),
                       [("dQ = dS K", S, D, S), ("dK = dS^T Q", S, D, S)]),
        "context_bwd": (lambda t, s: sbp.sbp_attn_context_bwd(L(t["dO"]), L(t["P"]), G(t["V"]),
                                                              L(t["o_dP"]), L(t["o_dV"]), p, r, s),
                        [("dP = dO V^T", S, S, D), ("dV = P^T dO", S, D, S)]),
    }
    rows = []
    for name, (fn, prods) in calls.items():
        it = [0]

        def call():
            t = sets[it[0] % len(sets)]
            it[0] += 1
            fn(t, stream.cuda_stream)
        with torch.cuda.stream(stream):
            call()
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                for _ in range(reps):
                    call()
        g.replay()
        torch.cuda.synchronize()
        us, per = time_replays(torch, g, reps)
        fl = sum(2.0 * B * hr * m * n * k for _, m, n, k in prods)
        by = sum(2.0 * B * hr * (m * k + k * n + m * n) for _, m, n, k in prods)
        rows.append({"call": name, "us_stats": step_stats(per),
                     "products": ["%s %dx%dx%d x%d" % (d, m, n, k, B * hr)
                                                for d, m, n, k in prods],
                     "us": us, "tflops": fl / us / 1e6,
                     "pct_of_bf16_peak": 100.0 * fl / us / 1e6 / BF16_PEAK_TFLOPS,
                     "algorithmic_gbs": by / us / 1e3,
                     "roofline_min_us": max(fl / BF16_PEAK_TFLOPS / 1e6, by / HBM_PEAK_GBS / 1e3)})
        log("%-12s %7.1f us %6.0f TFLOP/s %6.0f GB/s %s" % (name, us, fl / us / 1e6, by / us / 1e3,
                                                           ", ".join(rows[-1]["products"])))
    tot_us = sum(x["us"] for x in rows)
    tot_fl = sum(x["tflops"] * x["us"] * 1e6 for x in rows)
    return {"metric": "local-shard GEMM TFLOP/s (fwd+bwd) per SBP signature; % of bf16 MFMA peak",
            "value": tot_fl / tot_us / 1e6, "unit": "TFLOP/s", "n_gpus": 1,
            "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": wc.name, "batch": B, "heads": H, "seq": S, "head_dim": D,
                       "p": p, "rank": r, "local_heads": hr,
                       "mode": "per-call hip_graph replay"},
            "calls": rows}


def describe(label, sh):
    """Shapes (m x n x k) of the products one kernel launch of a call computes."""
    if "data" in sh:   # a grouped backward pair
        return "bwd_data %dx%dx%d + bwd_weight %dx%dx%d" % (
            sh["data"]["m"], sh["data"]["n"], sh["data"]["k"], sh["weight"]["m"],
            sh["weight"]["n"], sh["weight"]["k"])
    return "%s %dx%dx%d" % (label, sh["m"], sh["n"], sh["k"])


def step_stats(xs):
    """Mean with its 99 % confidence interval (Student t), and median with a
    distribution-free 99 % interval from order statistics, of per-step times
    (ms)."""
    import math
    import statistics
    n = len(xs)
    out = {"n": n, "mean": statistics.fmean(xs), "median": statistics.median(xs),
           "min": min(xs), "max": max(xs)}
    if n >= 2:
        from scipy import stats as st
        sd = statistics.stdev(xs)
        half = st.t.ppf(0.995, n - 1) * sd / math.sqrt(n)
        out["mean_ci99"] = [float(out["mean"] - half), float(out["mean"] + half)]
        # ranks j < k with P(x_(j) <= median <= x_(k)) >= 0.99 (binomial)
        ys = sorted(xs)
        j = int(st.binom.ppf(0.005, n, 0.5))
        k = n - j
        if j >= 1 and k <= n:
            out["median_ci99"] = [ys[j - 1], ys[k - 1]]
    return out


def sbp_split(D, p, r):
    """(offset, length) of rank r's balanced block of D over p (the library's rule)."""
    from paper_2301_06813_amd import sbp
    s = sbp.sbp_shard_index(sbp.split(0, p, r), D, 1)
    return s.row_off, s.rows


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true", help="time eager launches, not a graph")
    ap.add_argument("--dump", default=None, help="write per-launch shapes and durations (JSON)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy 5 times (scale for HBM counters)")
    ap.add_argument("--workload", type=int, default=5, choices=(2, 3, 4, 5, 6, 7, 8),
                    help="5 (default): the 24-layer step; 8: the same step with searched "
                         "signatures; 2-4, 6: per-call report of that workload's local "
                         "products; 7: the attention core")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this build measures rank r's local products on a "
              "single MI355X and has no multi-GPU path (--gpus %d requested)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2301_06813_amd import sbp, workloads
    from paper_2301_06813_amd.step import Step
    torch.cuda.set_device(0)
    if args.copy_calibration:
        src = torch.ones(1 << 29, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": src.numel() * 2, "copy_bytes_written": dst.numel() * 2,
                          "copies": 5}))
        return
    sbp.lib()
    if args.workload == 7:
        print(json.dumps(report_attention(0, reps=10)))
        return
    if args.workload not in (5, 8):
        ranks = {4: (0, 1), 6: ((0, 0, 0),)}.get(args.workload, (0,))
        print(json.dumps(report_workload(args.workload, ranks, reps=10)))
        return
    wl = workloads.transformer_step() if args.workload == 5 else \
        workloads.transformer_step_searched()
    log("building step: %d linears, p=%d, rank 0" % (len(wl.linears), wl.p))
    step = Step(wl, 0)
    stream = torch.cuda.Stream()
    sid = stream.cuda_stream
    torch.cuda.synchronize()
    log("warmup %d" % args.warmup)
    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            step.launch_all(sid)
    torch.cuda.synchronize()

    graph = None
    if not args.eager:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=stream):
            step.launch_all(torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        for _ in range(2):
            graph.replay()
        torch.cuda.synchronize()

    log("timing %d steps (%s)" % (args.steps, "eager" if args.eager else "graph"))
    # an event before the first step and after every step: the pair around
    # all K steps gives the step time, consecutive pairs each step's own
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        ev[0].record()
        for i in range(args.steps):
            if graph is not None:
                graph.replay()
            else:
                step.launch_all(sid)
            ev[i + 1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[-1]) / args.steps
    per_step = [ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]
    tflops = step.flops / (ms * 1e-3) / 1e12

    # per-kernel durations: the library records a HIP event pair with every
    # kernel dispatch (sbp_profile_begin/end), so host time between launches
    # is not counted
    log("per-kernel profile pass")
    n = len(step.calls)
    ksteps = max(1, min(args.steps, 5))
    per_call = [None] * n          # per call: [[name, us], ...] in launch order
    with torch.cuda.stream(stream):
        for _ in range(ksteps):
            for i, ks in enumerate(step.profile(sid)):
                if per_call[i] is None:
                    per_call[i] = [[name, 0.0] for name, _ in ks]
                for j, (name, us) in enumerate(ks):
                    per_call[i][j][1] += us / ksteps
    by_kernel = collections.defaultdict(lambda: [0.0, 0.0, 0.0, 0])
    by_sig = collections.defaultdict(lambda: [0.0, 0.0])
    launches = []
    for m, ks in zip(step.meta, per_call):
        t_call = sum(us for _, us in ks) * 1e-6
        by_sig[m["sig"]][0] += t_call
        by_sig[m["sig"]][1] += m["flops"]
        gemm_ks = [name for name, _ in ks if name.startswith("gemm")]
        # the call's product(s) belong to its GEMM kernel(s): one kernel (a
        # single product, or both backward products grouped) takes them all;
        # two kernels are the backward-data then the backward-weight product
        if len(gemm_ks) == 2:
            shares = {0: m["data"], 1: m["weight"]}
        else:
            shares = {0: m}
        g = 0
        kd = collections.OrderedDict()
        for name, us in ks:
            b = by_kernel[name]
            b[0] += us * 1e-6
            b[3] += 1
            if name.startswith("gemm"):
                sh = shares.get(g, {"flops": 0.0, "bytes": 0.0})
                b[1] += sh["flops"]
                b[2] += sh["bytes"]
                g += 1
            kd[name] = kd.get(name, 0.0) + us
        launches.append(dict({k_: v_ for k_, v_ in m.items() if k_ not in ("lin", "layouts")},
                             kernels=kd, us=sum(us for _, us in ks)))
    if args.dump:
        with open(args.dump, "w") as f:
            json.dump(launches, f)
    gemms = {k: v for k, v in by_kernel.items() if k.startswith("gemm")}
    dom, (kt, kf, kb, kn) = max(gemms.items(), key=lambda kv: kv[1][0])
    intensity = kf / kb
    if intensity >= RIDGE:
        roof = {"bound": "mfma", "achieved": kf / kn / (kt / kn) / 1e12,
                "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": kb / kn / (kt / kn) / 1e9, "peak": HBM_PEAK_GBS,
                "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    # HBM bytes per launch of the dominant kernel, from the committed counter
    # summary (null if it was taken from other kernel sources)
    roof["traffic"] = counted_traffic(dom)
    roof["traffic_source"] = ("profiles/gemm_bf16_transformer_step_hbm_counters.md"
                              if roof["traffic"] is not None else None)
    roof["algorithmic_bytes_per_launch"] = kb / kn
    roof["algorithmic_flops_per_launch"] = kf / kn
    roof["kernel"] = dom
    roof["launches_per_step"] = kn
    roof["avg_launch_us"] = kt / kn * 1e6
    roof["algorithmic_intensity_flop_per_byte"] = intensity
    # the dominant kernel serves several calls (product shapes): each one's
    # own fraction of the same bound
    per = collections.OrderedDict()
    for m, ks in zip(step.meta, per_call):
        for j, (name, us) in enumerate(ks):
            if name != dom:
                continue
            gemm_ks = [n_ for n_, _ in ks if n_.startswith("gemm")]
            if len(gemm_ks) == 2:
                first = gemm_ks.index(name) == 0
                sh, label = (m["data"], "bwd_data") if first else (m["weight"], "bwd_weight")
            else:
                sh, label = m, m["ops"][0]
            key = "%s %s: %s" % (m["linear"].split("_", 1)[1], m["sig"], describe(label, sh))
            e = per.setdefault(key, [0, 0.0, sh["flops"], sh["bytes"]])
            e[0] += 1
            e[1] += us
    # each call's products against their own roofline, min(peak, I x 8 TB/s):
    # frac = roofline-minimum time / measured time
    roof["per_product"] = []
    for key, (n_, us_tot, fl_, by_) in per.items():
        us_ = us_tot / n_
        t_f, t_b = fl_ / (BF16_PEAK_TFLOPS * 1e6), by_ / (HBM_PEAK_GBS * 1e3)
        roof["per_product"].append({"products": key, "launches": n_, "avg_us": us_,
                                    "bound": "mfma" if t_f >= t_b else "hbm",
                                    "tflops": fl_ / us_ / 1e6, "gbs": by_ / us_ / 1e3,
                                    "roofline_min_us": max(t_f, t_b),
                                    "frac": max(t_f, t_b) / us_})

    out = {
        "metric": "local-shard GEMM TFLOP/s (fwd+bwd) per SBP signature; % of bf16 MFMA peak",
        "value": tflops,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) activations/gradients, N(0,1/K) weights)",
        "config": {"workload": wl.name, "layers": 24, "hidden": 1024, "ffn": 4096,
                   "heads": 16, "tokens": 8192, "p": wl.p, "rank": 0,
                   "local_products_per_step": 3 * len(wl.linears),
                   "calls_per_step": n, "gflop_per_step": step.flops / 1e9,
                   "signatures": dict(collections.Counter(l.sig for l in wl.linears)),
                   "mode": "eager" if args.eager else "hip_graph",
                   **({"signature_choice": "coordinate-descent search, modelled communication "
                       "%.2f ms per step (alpha %g s, beta %g s/B)" % (
                           1e3 * workloads.searched_signatures()[1], workloads.XGMI_ALPHA,
                           workloads.XGMI_BETA)} if args.workload == 8 else {})},
        "pct_of_bf16_peak": 100.0 * tflops / BF16_PEAK_TFLOPS,
        "step_ms_stats": step_stats(per_step),
        "per_signature_tflops": {s: v[1] / v[0] / 1e12 for s, v in sorted(by_sig.items())},
        "kernel_time_sum_ms": sum(v[0] for v in by_kernel.values()) * 1e3,
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle), ~%.0f s" % args.cpu_seconds)
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
