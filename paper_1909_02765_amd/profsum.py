"""Summaries of rocprofv3 runs of bench.py, as kept under profiles/.

Counter runs use `bench.py --counter-run --workload W --copy-calib MIB`, which
prints one JSON line naming the plan, the dispatch counts (untimed spin-up,
counted warm-up, timed, cold) and the bytes each calibration copy moves:

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d F -o run -- python3 bench.py --counter-run ... > F.log
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d W -o run -- python3 bench.py --counter-run ... > W.log
    python -m paper_1909_02765_amd.profsum traffic F W --update profiles/traffic.json

FETCH_SIZE and WRITE_SIZE read in KiB per dispatch, in units that are not
exactly bytes on this chip, so each is scaled by what it reads for a plain
copy kernel (`copy_f4`) whose bytes are known.  The per-launch figure is the
mean over the timed dispatches of the convolution kernel (back to back, so
its operands are warm in the last-level cache); the cold figures are the
mean over the dispatches that each follow a 512 MiB scrub.

    python -m paper_1909_02765_amd.profsum trace D --log L  # kernel-trace table (markdown)
    python -m paper_1909_02765_amd.profsum counters D LOG   # mean of each counter, timed dispatches
    python -m paper_1909_02765_amd.profsum layers D W...     # per-layer table from <D>/<W>_{FETCH_SIZE,
                                                            # WRITE_SIZE,sqa,sqb,kt} runs (markdown)
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import statistics


def _one(d, suffix):
    f = glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True)
    if not f:
        raise SystemExit(f"no *{suffix} under {d}")
    return f[0]


def _bench_line(log):
    lines = [l for l in open(log) if l.startswith("{")]
    if not lines:
        raise SystemExit(f"no JSON line in {log}")
    return json.loads(lines[-1])


def is_conv_kernel(name):
    """The convolution kernels proper (not the weight packing or the split sum)."""
    return ("conv_igemm" in name or "conv_direct" in name) and "pack_weights" not in name


def dispatch_counters(d):
    """{dispatch id: (kernel name, {counter: summed value})} of a --pmc run
    (rows of one dispatch are summed over the counter's instances)."""
    rows = {}
    for r in csv.DictReader(open(_one(d, "counter_collection.csv"))):
        e = rows.setdefault(int(r["Dispatch_Id"]), (r["Kernel_Name"], {}))
        e[1][r["Counter_Name"]] = e[1].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return [rows[i] for i in sorted(rows)]


def timed_conv(rows, line, cold=False):
    """(kernel name, counter dicts of the timed dispatches -- or with `cold`,
    of the cold ones that end a --counter-run) of the run's most frequent
    convolution kernel."""
    names = {}
    for n, _ in rows:
        if is_conv_kernel(n):
            names[n] = names.get(n, 0) + 1
    if not names:
        raise SystemExit("no convolution dispatches")
    name = max(names, key=names.get)
    conv = [c for n, c in rows if n == name]
    dsp = line["dispatches"]
    if cold:
        return name, conv[len(conv) - dsp["cold"]:]
    s0 = dsp["spinup"] + dsp["warmup"]
    return name, conv[s0:s0 + dsp["timed"]]


def counter_mean(group, counter):
    return statistics.mean(c[counter] for c in group)


def traffic(fetch_dir, write_dir):
    out = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        line = _bench_line(d.rstrip("/") + ".log")
        rows = dispatch_counters(d)
        name, timed = timed_conv(rows, line)
        copies = [c[counter] for n, c in rows if "copy_f4" in n]
        if not copies or not line.get("copy_calib_bytes_each_way"):
            raise SystemExit(f"{d}: no calibration copies (run bench.py with --copy-calib)")
        factor = line["copy_calib_bytes_each_way"] / 1024.0 / statistics.mean(copies)
        raw = counter_mean(timed, counter)
        _, cold = timed_conv(rows, line, cold=True)
        out[counter] = dict(kernel=name, line=line, n=len(timed), raw_kib=raw, factor=factor,
                            bytes=raw * 1024.0 * factor, cold=counter_mean(cold, counter) * 1024.0 * factor)
    f, w = out["FETCH_SIZE"], out["WRITE_SIZE"]
    if f["line"]["kernel_digest"] != w["line"]["kernel_digest"] or f["kernel"] != w["kernel"]:
        raise SystemExit("the two counter runs were taken on different kernels")
    return f["line"]["workload"], {
        "kernel_digest": f["line"]["kernel_digest"],
        "kernel": f["kernel"],
        "plan": f["line"]["plan"],
        "fetch_bytes_per_launch": round(f["bytes"]), "write_bytes_per_launch": round(w["bytes"]),
        "hbm_bytes_per_launch": round(f["bytes"]) + round(w["bytes"]),
        "fetch_factor": round(f["factor"], 4), "write_factor": round(w["factor"], 4),
        "raw_fetch_kib": round(f["raw_kib"], 2), "raw_write_kib": round(w["raw_kib"], 2),
        "timed_dispatches": f["n"],
        "cold_fetch_bytes": round(f["cold"]), "cold_write_bytes": round(w["cold"]),
        "us_per_layer_under_counters": [f["line"]["us_per_layer"], w["line"]["us_per_layer"]]}


def timed_trace_ns(d, line):
    """Durations (ns) of the timed dispatches of the run's most frequent
    convolution kernel, from a kernel trace and the run's bench line (either
    a --counter-run line or the default one)."""
    durs = trace_durations(d)
    name = max((n for n in durs if is_conv_kernel(n)), key=lambda n: len(durs[n]))
    if "dispatches" in line:
        dsp = line["dispatches"]
        skip, n = dsp["spinup"] + dsp["warmup"], dsp["timed"]
    else:
        skip, n = line["spinup_calls"] + line["warmup"], line["steps"]
    return name, durs[name][skip:skip + n]


def layers_table(root, workloads):
    """One row per workload: plan, median kernel duration, counters per
    dispatch and derived shares, HBM bytes (calibrated)."""
    out = ["| layer | plan | kernel µs (median) | waves | VALU inst | MFMA inst | SALU inst | LDS inst | "
           "bank-conflict cycles / LDS inst | MFMA busy | TA busy | fetch MB | write MB |",
           "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for w in workloads:
        base = os.path.join(root, w)
        _, t = traffic(base + "_FETCH_SIZE", base + "_WRITE_SIZE")
        la = _bench_line(base + "_sqa.log")
        _, ca = timed_conv(dispatch_counters(base + "_sqa"), la)
        lb = _bench_line(base + "_sqb.log")
        _, cb = timed_conv(dispatch_counters(base + "_sqb"), lb)
        lk = _bench_line(base + "_kt.log")
        _, d = timed_trace_ns(base + "_kt", lk)
        med = statistics.median(d)
        m = {k: counter_mean(ca, k) for k in ca[0]}
        m.update({k: counter_mean(cb, k) for k in cb[0]})
        # Shares over the kernel's own duration at the measured clock: the
        # matrix-pipe cycles per SIMD (1024 SIMDs) and the address-unit busy
        # cycles per CU (256 TAs), against median duration x 2.4 GHz.
        cyc = med * 2.4
        mfma = m["SQ_VALU_MFMA_BUSY_CYCLES"] / 1024.0 / cyc
        ta = m["TA_TA_BUSY"] / 256.0 / cyc
        bank = m["SQ_LDS_BANK_CONFLICT"] / m["SQ_INSTS_LDS"] if m["SQ_INSTS_LDS"] else 0.0
        out.append(f"| {w} | {la['plan']} | {med / 1e3:.2f} | {m['SQ_WAVES']:.0f} | {m['SQ_INSTS_VALU']:.0f} | "
                   f"{m['SQ_INSTS_MFMA']:.0f} | {m['SQ_INSTS_SALU']:.0f} | {m['SQ_INSTS_LDS']:.0f} | {bank:.2f} | "
                   f"{100 * mfma:.1f}% | {100 * ta:.1f}% | {t['fetch_bytes_per_launch'] / 1e6:.3f} | "
                   f"{t['write_bytes_per_launch'] / 1e6:.3f} |")
    return "\n".join(out)


def trace_table(d):
    rows = list(csv.DictReader(open(_one(d, "kernel_stats.csv"))))
    out = ["| Kernel | Calls | Average ns | Min ns | Max ns |", "|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| `{r['Name'][:160]}` | {r['Calls']} | {float(r['AverageNs']):.0f} | {r['MinNs']} | {r['MaxNs']} |")
    return "\n".join(out)


def trace_durations(d):
    """{kernel name: [ns per dispatch in order]} from the kernel trace."""
    durs = {}
    for r in csv.DictReader(open(_one(d, "kernel_trace.csv"))):
        durs.setdefault(r["Kernel_Name"], []).append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    return durs


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("fetch_dir")
    t.add_argument("write_dir")
    t.add_argument("--update", default=None, help="merge the entry into this JSON file")
    k = sub.add_parser("trace")
    k.add_argument("dir")
    k.add_argument("--log", default=None, help="the bench.py output of the traced run (its JSON line gives "
                   "the spin-up, warm-up and timed call counts)")
    c = sub.add_parser("counters")
    c.add_argument("dir")
    c.add_argument("log")
    y = sub.add_parser("layers")
    y.add_argument("dir")
    y.add_argument("workloads", nargs="+")
    a = ap.parse_args()
    if a.cmd == "traffic":
        wl, e = traffic(a.fetch_dir, a.write_dir)
        print(json.dumps({wl: e}, indent=1))
        if a.update:
            try:
                cur = json.load(open(a.update))
            except (OSError, ValueError):
                cur = {}
            cur[wl] = e
            with open(a.update, "w") as f:
                json.dump(cur, f, indent=1)
                f.write("\n")
    elif a.cmd == "trace":
        print(trace_table(a.dir))
        if a.log:
            name, v = timed_trace_ns(a.dir, _bench_line(a.log))
            print(f"\n`{name[:120]}`: {len(v)} timed dispatches, median {statistics.median(v):.0f} ns, "
                  f"mean {statistics.mean(v):.0f} ns, min {min(v)} ns")
    elif a.cmd == "layers":
        print(layers_table(a.dir, a.workloads))
    else:
        line = _bench_line(a.log)
        name, timed = timed_conv(dispatch_counters(a.dir), line)
        print(json.dumps({"kernel": name[:200], "plan": line.get("plan"), "timed_dispatches": len(timed),
                          "mean": {k: round(counter_mean(timed, k), 1) for k in timed[0]}}, indent=1))


if __name__ == "__main__":
    main()
