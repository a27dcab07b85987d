"""Offline plan sweep (the auto-tuning step): time every compiled kernel
variant and split count on the shapes of interest on one MI355X, keep the
fastest per shape, and write the table the library compiles in.

    python -m paper_1909_02765_amd.tune --out tuned.json          # on the GPU
    python -m paper_1909_02765_amd.tune --emit tuned.json         # rewrite csrc/tuned_plans.inc

The table maps an exact shape (C_in, H, W, C_out, K, stride, pad) to a variant
name and a split count; shapes not in it fall back to the cost model.  With
--prepacked the sweep times every plan on weights prepacked for it, and
--emit --prepacked writes csrc/tuned_plans_prepacked.inc, the table behind
ilpm_conv2d_plan_prepacked.  With --pooled the calls carry the ReLU + 2x2
max-pool epilogue (tables tuned_plans_pooled*.inc, behind
ilpm_conv2d_plan_for and the epilogue call's default plan).
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
INC = os.path.join(PKG, "csrc", "tuned_plans.inc")
INC_PREPACKED = os.path.join(PKG, "csrc", "tuned_plans_prepacked.inc")
INC_POOLED = os.path.join(PKG, "csrc", "tuned_plans_pooled.inc")
INC_POOLED_PREPACKED = os.path.join(PKG, "csrc", "tuned_plans_pooled_prepacked.inc")
EPI_POOL = 3  # ReLU + 2x2 max-pool


def table_path(prepacked, pooled):
    if pooled:
        return INC_POOLED_PREPACKED if prepacked else INC_POOLED
    return INC_PREPACKED if prepacked else INC

SPLITS = (1, 2, 3, 4, 6, 8, 12, 16, 24, 32, 48, 64)
FINALISTS = 4


def default_shapes():
    sys.path.insert(0, ROOT)
    import workloads
    shapes = [tuple(c.dims()[k] for k in ("c_in", "h", "w", "c_out", "k", "stride", "pad"))
              for c in workloads.ALL_CASES]
    for _, ci, co, hw, _, _ in workloads.vgg16_layers():
        shapes.append((ci, hw, hw, co, 3, 1, 1))
    # The 3x3 layers of ResNet (Table 2 of the paper): conv2.x .. conv5.x.
    shapes += [(64, 56, 56, 64, 3, 1, 1), (128, 28, 28, 128, 3, 1, 1),
               (256, 14, 14, 256, 3, 1, 1), (512, 7, 7, 512, 3, 1, 1)]
    out = []
    for s in shapes:
        if s not in out:
            out.append(s)
    return out


def candidate_plans(ilpm, shape):
    c_in, h, w, c_out, k, s, p = shape
    plans, seen = [], set()
    for path in (ilpm.PATH_DIRECT, ilpm.PATH_IGEMM):
        for v in range(ilpm.num_variants(path)):
            for sp in (SPLITS if path == ilpm.PATH_IGEMM else (1,)):
                try:
                    pl = ilpm.plan_variant(c_in, h, w, c_out, k, s, p, path, v, sp)
                except ilpm.IlpmError:
                    continue
                key = (pl.path, pl.variant, pl.splits)
                if key not in seen:
                    seen.add(key)
                    plans.append(pl)
    return plans


def call_args(ilpm, bufs, shape, plan, stream, epilogue=0):
    """(entry point, arguments) of one call of `plan`: ilpm_conv2d_fwd_plan on
    the OIHW weights, or ilpm_conv2d_fwd_prepacked when bufs carries packed
    weights (x, w, out, packed); with an epilogue, the epilogue entry points
    (out then has the epilogue's shape)."""
    c_in, h, w, c_out, k, s, p = shape
    x, wt, out = bufs[:3]
    packed = bufs[3] if len(bufs) > 3 else None
    if epilogue:
        src = packed if packed is not None else wt
        fn = ilpm.lib.ilpm_conv2d_fwd_prepacked_epilogue if packed is not None else ilpm.lib.ilpm_conv2d_fwd_epilogue
        return fn, (ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(src.data_ptr()), None, c_in, h, w, c_out, k, s, p,
                    epilogue, ctypes.byref(plan), ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(stream))
    if packed is None:
        return ilpm.lib.ilpm_conv2d_fwd_plan, (
            ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(wt.data_ptr()), None, c_in, h, w, c_out, k, s, p,
            ctypes.c_void_p(out.data_ptr()), ctypes.byref(plan), ctypes.c_void_p(stream))
    return ilpm.lib.ilpm_conv2d_fwd_prepacked, (
        ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(packed.data_ptr()), None, c_in, h, w, c_out, k, s, p,
        ctypes.byref(plan), ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(stream))


def time_plan(torch, ilpm, bufs, shape, plan, reps, epilogue=0):
    f, args = call_args(ilpm, bufs, shape, plan, torch.cuda.current_stream().cuda_stream, epilogue)
    for _ in range(3):
        rc = f(*args)
        if rc != 0:
            raise ilpm.IlpmError(rc, f.__name__)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        f(*args)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1000.0 / reps


def time_plan_graph(torch, ilpm, bufs, shape, plan, reps, epilogue=0, per_graph=20):
    """Mean us per call with the calls replayed from a captured HIP graph:
    the kernels' own rate, without the host's launch cost between calls
    (which bounds eager timing of the smallest layers)."""
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    f, args = call_args(ilpm, bufs, shape, plan, stream.cuda_stream, epilogue)
    with torch.cuda.stream(stream):
        for _ in range(3):
            rc = f(*args)
            if rc != 0:
                raise ilpm.IlpmError(rc, f.__name__)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for _ in range(per_graph):
                f(*args)
    torch.cuda.synchronize()
    n = max(1, reps // per_graph)
    for _ in range(max(1, n // 4)):
        g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(n):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1000.0 / (n * per_graph)


def spin_up(torch, ms=300.0):
    """Untimed matrix work for `ms` milliseconds of wall clock, so that the
    first shape is not timed while the GPU is still ramping up."""
    import time
    a = torch.randn((2048, 2048), device="cuda")
    t0 = time.perf_counter()
    while (time.perf_counter() - t0) * 1e3 < ms:
        for _ in range(10):
            a = a @ a * 1e-3
        torch.cuda.synchronize()


def sweep(shapes, reps=100, graph=False, prepacked=False, pooled=False):
    import torch
    import paper_1909_02765_amd as ilpm
    torch.cuda.set_device(0)
    spin_up(torch)
    timer = time_plan_graph if graph else time_plan
    result = {}
    for shape in shapes:
        c_in, h, w, c_out, k, s, p = shape
        ho, wo = ilpm.out_size(h, k, s, p), ilpm.out_size(w, k, s, p)
        x = torch.rand((1, c_in, h, w), device="cuda")
        wt = torch.randn((c_out, c_in, k, k), device="cuda") * 0.05
        epi = EPI_POOL if pooled else 0
        out = torch.empty(ilpm.epilogue_out_shape(c_out, h, w, k, s, p, epi) if pooled else (1, c_out, ho, wo),
                          device="cuda")
        rows = []
        packs = {}
        for plan in candidate_plans(ilpm, shape):
            if plan.path == ilpm.PATH_DIRECT and plan.variant == 1 and c_in * c_out * ho * wo * k * k > 3e8:
                continue  # the plain fallback is far too slow to matter here
            bufs = (x, wt, out)
            if prepacked:
                packs[id(plan)] = ilpm.prepack_weights(wt, plan)
                bufs = (x, wt, out, packs[id(plan)])
            us = timer(torch, ilpm, bufs, shape, plan, reps, epi)
            rows.append(({"variant": ilpm.variant_name(plan.path, plan.variant), "path": plan.path,
                          "splits": plan.splits, "us": round(us, 3)}, plan))
        rows.sort(key=lambda r: r[0]["us"])
        # The close finishers are re-timed with ten times the calls, three
        # rounds interleaved, each keeping its best round: the first pass is
        # short and the top few often lie within its noise.
        finalists = rows[:FINALISTS]
        for row, _ in finalists:
            row["us_refined"] = float("inf")
        for _ in range(3):
            for row, plan in finalists:
                bufs = (x, wt, out, packs[id(plan)]) if prepacked else (x, wt, out)
                us = timer(torch, ilpm, bufs, shape, plan, reps * 10, epi)
                row["us_refined"] = round(min(row["us_refined"], us), 3)
        finalists.sort(key=lambda r: r[0]["us_refined"])
        ranked = [row for row, _ in finalists + rows[FINALISTS:]]
        key = ",".join(str(v) for v in shape)
        result[key] = {"best": ranked[0], "top": ranked[:8], "prepacked": prepacked, "pooled": pooled}
        print(key, ranked[0], flush=True)
        del packs
    return result


KEEP_MARGIN = 0.01  # a new plan must beat the table's current one by 1% to replace it


def read_table(path=INC):
    """The plan table as {"C_in,H,W,C_out,K,stride,pad": (variant, splits)}."""
    table = {}
    if not os.path.exists(path):
        return table
    for line in open(path):
        line = line.strip()
        if not line.startswith("{"):
            continue
        body = line[1:line.index("}")]
        parts = [t.strip() for t in body.split(",")]
        table[",".join(parts[:7])] = (parts[7].strip('"'), int(parts[8]))
    return table


def choose(entry, incumbent):
    """The best refined row, unless the incumbent plan was a finalist within KEEP_MARGIN of it."""
    best = entry["best"]
    if incumbent is None:
        return best
    t_best = best.get("us_refined", best["us"])
    for row in entry["top"]:
        if "us_refined" in row and (row["variant"], row["splits"]) == incumbent:
            if row["us_refined"] <= t_best * (1.0 + KEEP_MARGIN):
                return row
    return best


def read_comments(path=INC):
    """The timing comment of each table line, by shape key."""
    out = {}
    if not os.path.exists(path):
        return out
    for line in open(path):
        line = line.strip()
        if line.startswith("{") and "//" in line:
            body = line[1:line.index("}")]
            out[",".join(t.strip() for t in body.split(",")[:7])] = line[line.index("//"):]
    return out


def emit(table, path=INC):
    """Rewrite the table: shapes in `table` (a sweep) get their chosen plan;
    every other shape keeps its current line."""
    current = read_table(path)
    comments = read_comments(path)
    rows = {}
    for key, (variant, splits) in current.items():
        rows[key] = "{%s, \"%s\", %d},  %s" % (key.replace(",", ", "), variant, splits, comments.get(key, ""))
    for key, v in table.items():
        b = choose(v, current.get(key))
        us = b.get("us_refined", b["us"])
        rows[key] = "{%s, \"%s\", %d},  // %.2f us" % (key.replace(",", ", "), b["variant"], b["splits"], us)
    what = {INC_PREPACKED: "with prepacked weights (written by tune.py --emit --prepacked)",
            INC_POOLED: "with the ReLU + 2x2 max-pool epilogue (written by tune.py --emit --pooled)",
            INC_POOLED_PREPACKED: "with prepacked weights and the ReLU + 2x2 max-pool epilogue "
                                  "(written by tune.py --emit --pooled --prepacked)"}.get(
        path, "(written by tune.py --emit)")
    lines = ["// {C_in, H, W, C_out, K, stride, pad, \"variant\", splits}",
             "// Fastest measured plan per shape on one MI355X " + what + "."]
    for key in sorted(rows, key=lambda k: [int(t) for t in k.split(",")]):
        lines.append(rows[key].rstrip())
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=None, help="write the sweep as JSON")
    ap.add_argument("--emit", default=None, help="JSON from a sweep -> csrc/tuned_plans.inc")
    ap.add_argument("--reps", type=int, default=100)
    ap.add_argument("--shapes", nargs="*", default=None, metavar="C_in,H,W,C_out,K,stride,pad",
                    help="sweep only these shapes (default: every workload and VGG-16 / ResNet layer)")
    ap.add_argument("--graph", action="store_true",
                    help="time calls replayed from a HIP graph (for launch-bound layers)")
    ap.add_argument("--prepacked", action="store_true",
                    help="time plans on prepacked weights / emit the prepacked table")
    ap.add_argument("--pooled", action="store_true",
                    help="time plans with the ReLU + 2x2 max-pool epilogue / emit the pooled table")
    args = ap.parse_args()
    if args.emit:
        with open(args.emit) as f:
            table = json.load(f)
        if any(v.get("prepacked", False) != args.prepacked or v.get("pooled", False) != args.pooled
               for v in table.values()):
            raise SystemExit("the sweep's weight layout or epilogue does not match --prepacked / --pooled")
        emit(table, table_path(args.prepacked, args.pooled))
        return
    shapes = ([tuple(int(t) for t in sh.split(",")) for sh in args.shapes] if args.shapes
              else default_shapes())
    table = sweep(shapes, args.reps, args.graph, args.prepacked, args.pooled)
    if args.out:
        with open(args.out, "w") as f:
            json.dump(table, f, indent=1)


if __name__ == "__main__":
    main()
