"""Plan tuner: times every kernel plan the library can run for each local
product shape of the workloads on this GPU, and writes the fastest as the
library's tuned plan table (csrc/tuned_plans.inc).

    python -m paper_2301_06813_amd.tune [--out PATH] [--workloads 2,3,4,5]
    python -m paper_2301_06813_amd.tune --bwd [--out PATH]
    python -m paper_2301_06813_amd.tune --step [--out PATH]

The second form tunes the backward pair of each linear (sbp_linear_bwd):
one grouped launch of both products on a shared instance, against the two
separate launches of their tuned plans, and writes csrc/tuned_bwd_plans.inc
with the pairs whose grouped launch was faster (run it on a library built
with the single-product table).

The third form chooses plans inside the 24-layer step (workload 5): for each
distinct call, largest share of the step first, the whole step is captured
and replayed with that call's fastest isolated candidates and with its
current plan, and a candidate is kept when the step is faster (coordinate
descent). In the step a product runs with warm caches, throttled clocks and
its neighbours' traffic, so the isolated winner is not always the step's.
It writes the changed plans as JSON lines for merging into the tables.

A plan is (output tile, kernel instance, reduction splits, persistent
workgroups per compute unit); candidates are set with sbp_set_plan_override
and timed through the C ABI on the real shard views of every rank (so operand
alignment, and with it the eligible kernels, is that of the real calls),
replayed from a HIP graph over rotating input sets larger than the 256 MB
Infinity Cache. The table is keyed the way the planner looks plans up:
(orientation, output dtype, m, n, k, pipelined-kernel eligibility). Products
of other shapes keep the planner's analytic model. Rebuild the library after
writing a new table.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))

TILES = [(256, 256), (256, 192), (256, 128), (128, 256), (128, 128), (128, 64), (64, 128), (64, 64)]
CODES = (1, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13)   # pipelined instances; 2 (generic) for the rest
SPLITS = (1, 2, 3, 4, 6, 8, 12, 16, 24, 32)
ORIENT = {"fwd": 0, "bwd_data": 1, "bwd_weight": 2}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def product_cases(wl_ids):
    """{key: (workload, linear, op, rank)} for every distinct local product."""
    import torch
    from . import linear, sbp, workloads
    wls = {2: workloads.ffn_shard, 3: workloads.attention_dp, 4: workloads.vgg_head,
           5: workloads.transformer_step, 6: workloads.transformer_3d}
    cases = {}
    for c in wl_ids:
        wl = wls[c]()
        for lin in wl.linears:
            for r in wl.ranks:
                L = linear.layouts_for(lin, wl, r)
                for op in ("fwd", "bwd_data", "bwd_weight"):
                    rows, cols = linear.out_shape(op, L, lin.M, lin.K, lin.N)
                    k = {"fwd": linear.shard(L["x"], lin.M, lin.K).cols,
                         "bwd_data": linear.shard(L["dy"], lin.M, lin.N).cols,
                         "bwd_weight": linear.shard(L["x"], lin.M, lin.K).rows}[op]
                    f32 = linear.out_dtype(op, L, wl.dtype) == torch.float32
                    key = (ORIENT[op], int(f32), rows, cols, k, _eligible(op, L, lin))
                    cases.setdefault(key, (wl, lin, op, r))
    return cases


def _eligible(op, L, lin):
    """The library's pipelined-kernel mode for rank r's operand views (the
    key the plan table is looked up by): 0 the generic kernel; 1 the
    pipelined kernel (every operand 16-byte aligned, leading dimensions and
    contiguous extents multiples of 8); 2 its shifted form (leading
    dimensions multiples of 8, a shard that starts inside a 16-byte block
    only along an output dimension, or along the reduction when both
    operands are k-major with the same offset)."""
    from . import linear

    def view(layout, rows, cols):
        s = linear.shard(layout, rows, cols)
        return (s.row_off * cols + s.col_off) % 8, s.cols

    M, K, N = lin.M, lin.K, lin.N
    if op == "fwd":
        (oa, ca), (ob, cb) = view(L["x"], M, K), view(L["w"], K, N)
        ok = K % 8 == 0 and N % 8 == 0 and oa == 0
    elif op == "bwd_data":
        (oa, ca), (ob, cb) = view(L["dy"], M, N), view(L["w"], K, N)
        ok = N % 8 == 0 and oa == ob
    else:
        (oa, ca), (ob, cb) = view(L["x"], M, K), view(L["dy"], M, N)
        ok = K % 8 == 0 and N % 8 == 0
    if not ok:
        return 0
    return 1 if (oa == 0 and ob == 0 and ca % 8 == 0 and cb % 8 == 0) else 2


# the instances with a shifted form (mode 2 products): tile, kernel code
SHIFT_CODES = {((64, 64), 1), ((128, 128), 4), ((64, 64), 12), ((128, 64), 12), ((64, 128), 12),
               ((128, 128), 12)}


def valid_candidates(sbp, key, tiles_n_items, max_splits=None, nbatch=1):
    """(tile_m, tile_n, splits, kernel, wgs_per_cu) plans to time for key (the
    argument order of sbp_set_plan_override)."""
    orient, f32, m, n, k, dma = key
    kblocks = max(1, (k + 63) // 64)
    out = []
    # shifted-form products: the instances that have that form, and the
    # generic kernel
    codes = (CODES + (2,)) if dma == 2 else (CODES if dma else (2,))
    for (bm, bn) in TILES:
        tiles = ((m + bm - 1) // bm) * ((n + bn - 1) // bn)
        for code in codes:
            if dma == 2 and code != 2 and ((bm, bn), code) not in SHIFT_CODES:
                continue
            try:
                sbp.sbp_set_plan_override(bm, bn, 1, code, 0)
            except sbp.SbpError:
                continue
            last = 0
            for s in SPLITS:
                if max_splits is not None and s > max_splits:
                    continue
                per = -(-kblocks // min(s, kblocks))
                eff = -(-kblocks // per)
                if eff == last or (eff > 1 and per < 2):
                    continue
                last = eff
                items = tiles * eff * nbatch
                if (items > 8192 and nbatch == 1) or (eff > 1 and items > 4096):
                    continue
                # the library clamps splits whose partials exceed the workspace
                if eff > 1 and eff * m * (-(-n // 4) * 4) * 4 > sbp.SBP_WORKSPACE_BYTES:
                    continue
                occs = (0,) if (code == 2 or items <= 256) else (0, 1, 2)
                for occ in occs:
                    out.append((bm, bn, eff, code, occ))
    sbp.sbp_set_plan_override(0, 0, 1)
    return out


def time_plan(torch, sbp, fn, plan, reps, stream, keep=False):
    """Mean time of fn under plan (set here, and cleared after, unless keep:
    then the caller has set the overrides)."""
    if not keep:
        sbp.sbp_set_plan_override(*plan)
    try:
        with torch.cuda.stream(stream):
            fn()           # first call on this stream may allocate the workspace
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                for _ in range(reps):
                    fn()
        g.replay()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        # replay() runs on the current stream: bracket it there
        e0.record()
        for _ in range(3):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / (3 * reps)
    finally:
        if not keep:
            sbp.sbp_set_plan_override(0, 0, 1)


GROUP_INSTANCES = [((128, 128), 1), ((256, 192), 1), ((128, 128), 4), ((128, 128), 5), ((256, 128), 5),
                   ((128, 256), 5), ((64, 64), 1), ((128, 64), 1), ((64, 128), 1),
                   ((256, 256), 1), ((128, 128), 7), ((128, 128), 10), ((64, 64), 5),
                   ((64, 64), 7), ((128, 64), 5), ((64, 128), 5), ((128, 128), 12),
                   ((128, 64), 12), ((64, 128), 12), ((64, 64), 12), ((128, 128), 13),
                   ((64, 64), 13), ((128, 128), 6), ((256, 256), 6), ((256, 128), 7),
                   ((128, 256), 7), ((128, 64), 7), ((64, 128), 7), ((128, 64), 13),
                   ((64, 128), 13), ((128, 64), 4), ((64, 128), 4), ((64, 64), 4),
                   ((256, 256), 8), ((128, 128), 9), ((256, 128), 9), ((128, 256), 9),
                   ((128, 64), 11), ((64, 128), 11), ((64, 64), 11)]


def bwd_pairs(wl_ids):
    """{(key_d, key_w): (workload, linear, rank)} for every distinct backward pair."""
    import torch
    from . import linear, sbp, workloads
    pairs = {}
    for c in wl_ids:
        wl = {2: workloads.ffn_shard, 3: workloads.attention_dp, 4: workloads.vgg_head,
              5: workloads.transformer_step, 6: workloads.transformer_3d}[c]()
        for lin in wl.linears:
            for r in wl.ranks:
                L = linear.layouts_for(lin, wl, r)
                keys = []
                for op in ("bwd_data", "bwd_weight"):
                    rows, cols = linear.out_shape(op, L, lin.M, lin.K, lin.N)
                    k = (linear.shard(L["dy"], lin.M, lin.N).cols if op == "bwd_data"
                         else linear.shard(L["x"], lin.M, lin.K).rows)
                    f32 = linear.out_dtype(op, L, wl.dtype) == torch.float32
                    keys.append((ORIENT[op], int(f32), rows, cols, k, _eligible(op, L, lin)))
                if keys[0][5] and keys[1][5]:
                    pairs.setdefault(tuple(keys), (wl, lin, r))
    return pairs


def tune_bwd(args, torch, sbp, linear, workloads, stream, single_best=None):
    """Grouped launch of each backward pair against its two products run
    separately: the sum of their tuned times (single_best, from the same run),
    else a measured pair of launches of the compiled-in plans."""
    pairs = bwd_pairs([int(c) for c in args.workloads.split(",") if int(c) != 7])
    log("%d distinct backward pairs" % len(pairs))
    rows = []
    for (kd, kw), (wl, lin, r) in sorted(pairs.items()):
        per_set = 2 * (2 * lin.M * lin.K + lin.K * lin.N + 2 * lin.M * lin.N)
        nsets = max(2, min(6, -(-600 * 2 ** 20 // per_set)))
        sets = []
        for i in range(nsets):
            X, W, dY = workloads.make_tensors(lin, wl.dtype, "cuda")
            Lr = linear.layouts_for(lin, wl, r)
            dX = linear.alloc_out_L("bwd_data", Lr, lin.M, lin.K, lin.N, wl.dtype, "cuda")
            dW = linear.alloc_out_L("bwd_weight", Lr, lin.M, lin.K, lin.N, wl.dtype, "cuda")
            sets.append((X, W, dY, dX, dW))
        it = [0]

        def fn():
            X, W, dY, dX, dW = sets[it[0] % nsets]
            it[0] += 1
            linear.run_bwd_L(Lr, X, W, dY, dX, dW, stream.cuda_stream)

        def timed(plan, mode, sw):
            sbp.sbp_set_plan_override(*plan)
            sbp.sbp_set_bwd_override(mode, sw)
            try:
                return time_plan(torch, sbp, fn, plan, args.reps, stream, keep=True)
            finally:
                sbp.sbp_set_plan_override(0, 0, 1)

        if single_best and kd in single_best and kw in single_best:
            sep = single_best[kd] + single_best[kw]
        else:
            sbp.sbp_set_bwd_override(1, 1)
            try:
                sep = time_plan(torch, sbp, fn, (0, 0, 1, 0, 0), 3 * args.reps, stream,
                                keep=True)
            finally:
                sbp.sbp_set_bwd_override(0, 1)
        timings = []
        kbd, kbw = max(1, (kd[4] + 63) // 64), max(1, (kw[4] + 63) // 64)
        for (bm, bn), code in GROUP_INSTANCES:
            if 2 in (kd[5], kw[5]) and ((bm, bn), code) not in SHIFT_CODES:
                continue   # grouped launches of shifted-form products
            for sd in (1, 2, 3, 4, 8, 16):
                if sd > 1 and kbd // sd < 2:
                    continue
                for sw in (1, 2, 3, 4, 8, 16):
                    if sw > 1 and kbw // sw < 2:
                        continue
                    try:
                        timings.append((timed((bm, bn, sd, code, 0), 2, sw),
                                        (bm, bn, code, sd, sw)))
                    except sbp.SbpError:
                        continue

        def retime(pl):
            bm, bn, code, sd, sw = pl
            sbp.sbp_set_plan_override(bm, bn, sd, code, 0)
            sbp.sbp_set_bwd_override(2, sw)
            try:
                return time_plan(torch, sbp, fn, None, 3 * args.reps, stream, keep=True)
            finally:
                sbp.sbp_set_plan_override(0, 0, 1)
        best = pick(timings, retime) if timings else None
        log("%s %s d %s w %s: separate %6.1f us, best grouped %6.1f us %s"
            % (lin.sig, lin.name, kd[2:5], kw[2:5], sep, best[0] if best else -1,
               best[1] if best else None))
        if best and best[0] < 0.97 * sep:
            rows.append((kd, kw, best[1], best[0], sep))
        del sets
        torch.cuda.empty_cache()
    with open(args.out, "w") as f:
        f.write("// Tuned grouped backward pairs: generated by paper_2301_06813_amd/tune.py --bwd.\n")
        f.write("// dX m, n, k, fp32, dW m, n, k, fp32 -> tile_m, tile_n, kernel, splits dX, "
                "splits dW; grouped us (separate us)\n")
        for kd, kw, (bm, bn, code, sd, sw), us, sep in rows:
            f.write("{%d, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d},  // %.1f (%.1f)\n"
                    % (kd[2], kd[3], kd[4], kd[1], kw[2], kw[3], kw[4], kw[1], bm, bn, code,
                       sd, sw, us, sep))
    log("wrote %s" % args.out)


def tune_attention(args, torch, sbp, stream):
    """Plans of the attention core's batched products (workload 7): one row per
    distinct product, keyed with its batch count. Each product is tuned through
    the call that holds it, with the plan override restricted to its
    orientation (the call's other product keeps its own plan)."""
    from . import inputs, workloads
    wc = workloads.attention_core()
    B, H, S, D, p = wc.batch, wc.heads, wc.seq, wc.head_dim, wc.p
    hr = -(-H // p) if H % p else H // p      # rank 0's heads (balanced split)
    nb = B * hr
    sets = []
    for i in range(3):
        sd = wc.seed_base + 10 * i
        act = inputs.randn((B, S, 3, H, D), 1.0, sd + 1, torch.bfloat16, "cuda")
        t = dict(act=act, Q=act[:, :, 0].permute(0, 2, 1, 3), K=act[:, :, 1].permute(0, 2, 1, 3),
                 V=act[:, :, 2].permute(0, 2, 1, 3),
                 P=inputs.randn((B, hr, S, S), 1.0, sd + 2, torch.bfloat16, "cuda"),
                 dS=inputs.randn((B, hr, S, S), 1.0, sd + 3, torch.bfloat16, "cuda"))
        for k_, shp in (("S", (B, hr, S, S)), ("O", (B, hr, S, D)), ("dQ", (B, hr, S, D)),
                        ("dK", (B, hr, S, D))):
            t[k_] = torch.empty(shp, dtype=torch.bfloat16, device="cuda")
        sets.append(t)
    G = lambda x: sbp.view4(x, sbp.SBP_GLOBAL)
    L = lambda x: sbp.view4(x, sbp.SBP_LOCAL)
    calls = [  # (call, orientation mask, product key)
        (lambda t, s: sbp.sbp_attn_scores(G(t["Q"]), G(t["K"]), L(t["S"]), p, 0, s), 2,
         (ORIENT["bwd_data"], 0, S, S, D, 1)),
        (lambda t, s: sbp.sbp_attn_context(L(t["P"]), G(t["V"]), L(t["O"]), p, 0, s), 1,
         (ORIENT["fwd"], 0, S, D, S, 1)),
        (lambda t, s: sbp.sbp_attn_scores_bwd(L(t["dS"]), G(t["Q"]), G(t["K"]), L(t["dQ"]),
                                              L(t["dK"]), p, 0, s), 4,
         (ORIENT["bwd_weight"], 0, S, D, S, 1)),
    ]
    rows = []
    for call, mask, key in calls:
        it = [0]

        def fn():
            t = sets[it[0] % len(sets)]
            it[0] += 1
            call(t, stream.cuda_stream)

        def timed(plan, reps):
            sbp.sbp_set_plan_override(*plan)
            sbp.sbp_set_override_orients(mask)
            try:
                return time_plan(torch, sbp, fn, plan, reps, stream, keep=True)
            finally:
                sbp.sbp_set_plan_override(0, 0, 1)

        cands = valid_candidates(sbp, key, None, max_splits=1, nbatch=nb)
        timings = []
        for plan in cands:
            try:
                timings.append((timed(plan, args.reps), plan))
            except sbp.SbpError as e:
                log("  plan %s failed: %s" % (plan, e))
        best = pick(timings, lambda pl: timed(pl, 3 * args.reps))
        auto = time_plan(torch, sbp, fn, (0, 0, 1, 0, 0), 3 * args.reps, stream)
        log("attention %s m %d n %d k %d x%d: best %6.1f us %s (model plan %6.1f us), %d candidates"
            % (list(ORIENT)[key[0]], key[2], key[3], key[4], nb, best[0], best[1], auto,
               len(cands)))
        rows.append((key, best[1], best[0], auto, nb))
    del sets
    torch.cuda.empty_cache()
    return rows


def pick(timings, retime, top=5, rounds=3):
    """Best plan of [(us, plan)]: the `top` fastest of the sweep are timed again
    `rounds` times at higher repetition and ranked by their median."""
    cands = [p for _, p in sorted(timings)[:top]]
    med = []
    for p in cands:
        ts = sorted(retime(p) for _ in range(rounds))
        med.append((ts[len(ts) // 2], p))
    return min(med)


# ------------------------------------------------------------ in-step tuning
def _call_key(torch, linear, meta, dtype):
    """Plan-table key of a step call: ("fwd", product key) or ("bwd", data key,
    weight key), product keys as in product_cases."""
    lin, L = meta["lin"], meta["layouts"]

    def pkey(op):
        rows, cols = linear.out_shape(op, L, lin.M, lin.K, lin.N)
        k = {"fwd": linear.shard(L["x"], lin.M, lin.K).cols,
             "bwd_data": linear.shard(L["dy"], lin.M, lin.N).cols,
             "bwd_weight": linear.shard(L["x"], lin.M, lin.K).rows}[op]
        f32 = linear.out_dtype(op, L, dtype) == torch.float32
        return (ORIENT[op], int(f32), rows, cols, k, _eligible(op, L, lin))
    if meta["ops"] == ("fwd",):
        return ("fwd", pkey("fwd"))
    return ("bwd", pkey("bwd_data"), pkey("bwd_weight"))


def _isolated_top(args, torch, sbp, linear, workloads, stream, key, wl, lin, r, top, diverse=0):
    """The `top` fastest candidate plans of one step call, timed in isolation
    (graph replays over rotating input sets, as the table tuner does), and
    up to `diverse` more: the fastest plan of each instance not yet among
    them."""
    per_set = 2 * (2 * lin.M * lin.K + lin.K * lin.N + 2 * lin.M * lin.N)
    nsets = max(2, min(6, -(-600 * 2 ** 20 // per_set)))
    Lr = linear.layouts_for(lin, wl, r)
    sets = []
    for _ in range(nsets):
        X, W, dY = workloads.make_tensors(lin, wl.dtype, "cuda")
        outs = {op: linear.alloc_out_L(op, Lr, lin.M, lin.K, lin.N, wl.dtype, "cuda")
                for op in ("fwd", "bwd_data", "bwd_weight")}
        sets.append((X, W, dY, outs))
    it = [0]
    timings = []
    if key[0] == "fwd":
        def fn():
            X, W, dY, o = sets[it[0] % nsets]
            it[0] += 1
            linear.run_L("fwd", Lr, X, W, dY, o["fwd"], stream.cuda_stream)
        for plan in valid_candidates(sbp, key[1], None):
            try:
                timings.append((time_plan(torch, sbp, fn, plan, args.reps, stream), ("fwd",) + plan))
            except sbp.SbpError:
                pass
    else:
        def fn():
            X, W, dY, o = sets[it[0] % nsets]
            it[0] += 1
            linear.run_bwd_L(Lr, X, W, dY, o["bwd_data"], o["bwd_weight"], stream.cuda_stream)
        kd, kw = key[1], key[2]
        kbd, kbw = max(1, (kd[4] + 63) // 64), max(1, (kw[4] + 63) // 64)
        for (bm, bn), code in GROUP_INSTANCES:
            if 2 in (kd[5], kw[5]) and ((bm, bn), code) not in SHIFT_CODES:
                continue
            for sd in (1, 2, 3, 4, 8, 16):
                if sd > 1 and kbd // sd < 2:
                    continue
                for sw in (1, 2, 3, 4, 8, 16):
                    if sw > 1 and kbw // sw < 2:
                        continue
                    sbp.sbp_set_plan_override(bm, bn, sd, code, 0)
                    sbp.sbp_set_bwd_override(2, sw)
                    try:
                        timings.append((time_plan(torch, sbp, fn, None, args.reps, stream,
                                                  keep=True), ("grp", bm, bn, code, sd, sw)))
                    except sbp.SbpError:
                        pass
                    finally:
                        sbp.sbp_set_plan_override(0, 0, 1)
        sbp.sbp_set_bwd_override(1, 1)
        try:
            timings.append((time_plan(torch, sbp, fn, None, args.reps, stream, keep=True),
                            ("sep",)))
        finally:
            sbp.sbp_set_plan_override(0, 0, 1)
    del sets
    torch.cuda.empty_cache()
    ranked = [p for _, p in sorted(timings)]
    out = ranked[:top]
    if diverse:
        # plus the fastest plan of every other (tile, kernel) instance, in order
        def inst(p):
            return None if p[0] == "sep" else (p[1], p[2], p[4] if p[0] == "fwd" else p[3])
        seen = {inst(p) for p in out}
        for p in ranked[top:]:
            if len(out) >= top + diverse:
                break
            if inst(p) is not None and inst(p) not in seen:
                seen.add(inst(p))
                out.append(p)
    return out


def _apply(sbp, cand, on):
    """Set (on) or clear the overrides that make one call run candidate cand."""
    if not on:
        sbp.sbp_set_plan_override(0, 0, 1)
        return
    if cand[0] == "fwd":
        _, bm, bn, splits, code, occ = cand
        sbp.sbp_set_plan_override(bm, bn, splits, code, occ)
    elif cand[0] == "grp":
        _, bm, bn, code, sd, sw = cand
        sbp.sbp_set_plan_override(bm, bn, sd, code, 0)
        sbp.sbp_set_bwd_override(2, sw)
    else:
        sbp.sbp_set_bwd_override(1, 1)


def tune_step(args, torch, sbp, linear, workloads, stream):
    """Plans of the 24-layer step's calls chosen inside the step: for each
    distinct call (largest share of the step first) the step graph is
    captured with that call's candidate plans -- the fastest few in isolation
    and the library's current plan -- and replayed; a candidate replaces the
    current plan when the whole step is faster by more than the noise, with
    earlier choices kept (coordinate descent). Writes the changed table rows
    to args.out (one line per key: fwd or bwd, key, plan, step ms)."""
    from .step import Step
    wl = workloads.transformer_step() if args.step_workload == 5 else \
        workloads.transformer_step_searched()
    step = Step(wl, 0)
    keys = [_call_key(torch, linear, m, wl.dtype) for m in step.meta]
    calls_of = {}
    for i, k in enumerate(keys):
        calls_of.setdefault(k, []).append(i)
    chosen = {}

    def hook(i, before):
        c = chosen.get(keys[i]) if trial[0] is None or keys[i] != trial[0][0] else trial[0][1]
        if c is not None:
            _apply(sbp, c, before)

    trial = [None]

    def measure(reps=args.step_reps):
        sid = stream.cuda_stream
        with torch.cuda.stream(stream):
            step.launch_all(sid, hook)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                step.launch_all(torch.cuda.current_stream().cuda_stream, hook)
        torch.cuda.synchronize()
        g.replay()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        del g
        return e0.elapsed_time(e1) / reps

    # per-call step time of the current plans orders the keys
    prof = [0.0] * len(keys)
    with torch.cuda.stream(stream):
        step.launch_all(stream.cuda_stream)
        for _ in range(2):
            for i, ks in enumerate(step.profile(stream.cuda_stream)):
                prof[i] += sum(us for _, us in ks)
    share = {k: sum(prof[i] for i in idx) for k, idx in calls_of.items()}
    order = sorted(share, key=lambda k: -share[k])
    base = min(measure() for _ in range(3))
    log("step %.4f ms with the current plans; %d distinct calls" % (base, len(order)))
    rows = []
    for k in order:
        i0 = calls_of[k][0]
        m = step.meta[i0]
        cands = _isolated_top(args, torch, sbp, linear, workloads, stream, k, wl, m["lin"], 0,
                              args.step_top, args.step_diverse)
        res = {}
        for rnd in range(2):
            trial[0] = None
            res.setdefault(None, []).append(measure())
            for c in cands:
                trial[0] = (k, c)
                try:
                    res.setdefault(c, []).append(measure())
                except sbp.SbpError as e:
                    log("  %s failed: %s" % (c, e))
                    res[c] = [1e9]
                finally:
                    trial[0] = None
        best = min(res, key=lambda c: min(res[c]))
        cur = min(res[None])
        log("%s x%d (%.0f us/step): current %.4f ms, best %s %.4f ms" % (
            k, len(calls_of[k]), share[k] / 2, cur, best, min(res[best])))
        if best is not None and min(res[best]) < cur * (1 - args.step_gain):
            chosen[k] = best
            rows.append((k, best, min(res[best]), cur))
    trial[0] = None
    final = min(measure() for _ in range(3))
    log("step %.4f -> %.4f ms" % (base, final))
    with open(args.out, "w") as f:
        for k, c, t, t0 in rows:
            f.write(json.dumps({"key": k, "plan": c, "step_ms": t, "was_ms": t0}) + "\n")
    log("wrote %s" % args.out)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--out", default=None)
    ap.add_argument("--workloads", default="2,3,4,5,6,7")
    ap.add_argument("--reps", type=int, default=10)
    ap.add_argument("--bwd", action="store_true", help="tune grouped backward pairs only")
    ap.add_argument("--all", action="store_true",
                    help="tune single products, then backward pairs against their sums")
    ap.add_argument("--out-bwd", default=os.path.join(HERE, "csrc", "tuned_bwd_plans.inc"))
    ap.add_argument("--step", action="store_true",
                    help="choose the 24-layer step's plans inside the step (writes JSON lines "
                         "of changed plans to --out)")
    ap.add_argument("--step-workload", type=int, default=5, choices=(5, 8))
    ap.add_argument("--step-top", type=int, default=5)
    ap.add_argument("--step-diverse", type=int, default=0,
                    help="also try the fastest plan of up to this many more instances")
    ap.add_argument("--step-reps", type=int, default=30)
    ap.add_argument("--step-gain", type=float, default=0.002)
    args = ap.parse_args()
    if args.out is None:
        args.out = args.out_bwd if args.bwd else os.path.join(HERE, "csrc", "tuned_plans.inc")

    import torch
    from . import linear, sbp, workloads
    torch.cuda.set_device(0)
    sbp.lib()
    stream = torch.cuda.Stream()
    if args.bwd:
        tune_bwd(args, torch, sbp, linear, workloads, stream)
        return
    if args.step:
        tune_step(args, torch, sbp, linear, workloads, stream)
        return
    cases = product_cases([int(c) for c in args.workloads.split(",") if int(c) != 7])
    log("%d distinct local products" % len(cases))
    single_best = {}
    rows = []
    t_start = time.time()
    for key, (wl, lin, op, r) in sorted(cases.items()):
        orient, f32, m, n, k, dma = key
        per_set = 2 * (lin.M * lin.K + lin.K * lin.N + lin.M * lin.N)
        nsets = max(2, min(6, -(-600 * 2 ** 20 // per_set)))
        sets = []
        for i in range(nsets):
            X, W, dY = workloads.make_tensors(lin, wl.dtype, "cuda")
            Lr = linear.layouts_for(lin, wl, r)
            out = linear.alloc_out_L(op, Lr, lin.M, lin.K, lin.N, wl.dtype, "cuda")
            sets.append((X, W, dY, out))
        it = [0]

        def fn():
            X, W, dY, out = sets[it[0] % nsets]
            it[0] += 1
            linear.run_L(op, Lr, X, W, dY, out, stream.cuda_stream)

        cands = valid_candidates(sbp, key, None)
        timings = []
        for plan in cands:
            try:
                timings.append((time_plan(torch, sbp, fn, plan, args.reps, stream), plan))
            except sbp.SbpError as e:
                log("  plan %s failed: %s" % (plan, e))
        best = pick(timings, lambda p: time_plan(torch, sbp, fn, p, 3 * args.reps, stream))
        auto = time_plan(torch, sbp, fn, (0, 0, 1, 0, 0), 3 * args.reps, stream)
        single_best[key] = best[0]
        bm, bn, splits, code, occ = best[1]
        log("%s %-10s m %5d n %5d k %5d f32 %d dma %d: best %6.1f us %s (model plan %6.1f us), "
            "%d candidates" % (lin.sig, op, m, n, k, f32, dma, best[0], best[1], auto, len(cands)))
        rows.append((key, best[1], best[0], auto))
        del sets
        torch.cuda.empty_cache()
    wl_ids = [int(c) for c in args.workloads.split(",")]
    if 7 in wl_ids:
        rows += [(key, plan, us, auto) + (nb,) for key, plan, us, auto, nb in
                 tune_attention(args, torch, sbp, stream)]
    log("tuned in %.0f s" % (time.time() - t_start))
    dev = torch.cuda.get_device_properties(0)
    with open(args.out, "w") as f:
        f.write("// Tuned bf16 plans: generated by paper_2301_06813_amd/tune.py on %s (%d CUs).\n"
                % (dev.name, dev.multi_processor_count))
        f.write("// orient, out_f32, m, n, k, pipelined-eligible -> tile_m, tile_n, kernel, "
                "splits, persistent workgroups per CU; fastest measured, us (model's plan, us)\n")
        for row in rows:
            (orient, f32, m, n, k, dma), (bm, bn, splits, code, occ), us, auto = row[:4]
            nb = row[4] if len(row) > 4 else 1
            batch = ", %d" % nb if nb > 1 else ""
            f.write("{%d, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d%s},  // %.1f (%.1f)\n"
                    % (orient, f32, m, n, k, dma, bm, bn, code, splits, occ, batch, us, auto))
    log("wrote %s" % args.out)
    if args.all:
        args.out = args.out_bwd
        tune_bwd(args, torch, sbp, linear, workloads, stream, single_best)


if __name__ == "__main__":
    main()
