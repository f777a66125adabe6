"""Summarise rocprofv3 output of bench.py into short text notes under profiles/.

Inputs (directories written by rocprofv3 ``--output-format csv``):
  --trace DIR   a ``--kernel-trace --stats`` run (uses *_kernel_stats.csv);
                alone (with --trace-bench), only the per-kernel table of the
                store's own kernels is written
  --fetch DIR   a ``--pmc FETCH_SIZE`` run (uses *_counter_collection.csv)
  --write DIR   a ``--pmc WRITE_SIZE`` run
  --bench FILE  the JSON line bench.py printed in the counter runs
  --window NAME:FIRST:COUNT  (repeatable, with --trace alone) the average
                duration of dispatches FIRST .. FIRST+COUNT-1, in start order,
                of the kernel whose name contains NAME (*_kernel_trace.csv):
                the launches a bench phase timed, apart from other launches
                of the same kernel in the run
  --pmc DIR     (repeatable, instead of --fetch/--write) any ``--pmc`` runs:
                the average per dispatch of every counter collected, for
                every store kernel, plus the L2 hit rate where TCC_HIT and
                TCC_MISS were both collected

HBM traffic of a kernel = FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each
scaled by the factor that maps the same counter onto the known byte count of
a plain device-to-device copy in the same run (the copy bench.py times for
its ceiling, a ``__amd_rocclr_copyBuffer`` dispatch of ``hbm_ceiling.bytes``
bytes as that run's JSON line states). The record
carries the SHA-256 of the copy kernel's source; bench.py reports the traffic
only while that source is unchanged.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
from collections import defaultdict

HERE = os.path.dirname(os.path.abspath(__file__))
COPY_SRC = os.path.join(HERE, "csrc", "copy.hip")
GATHER = "k_copy_pairs<true>"
SCATTER = "k_copy_pairs<false>"
PLAIN_COPY = "__amd_rocclr_copyBuffer"


def copy_source_sha() -> str:
    return hashlib.sha256(open(COPY_SRC, "rb").read()).hexdigest()


def _one(pattern: str) -> str:
    hits = glob.glob(pattern)
    if not hits:
        raise FileNotFoundError(pattern)
    return hits[0]


def kernel_stats(trace_dir: str):
    rows = list(csv.DictReader(open(_one(os.path.join(trace_dir, "*kernel_stats.csv")))))
    return [(r["Name"], int(r["Calls"]), float(r["AverageNs"]) / 1e6, float(r["Percentage"]))
            for r in rows]


def dispatch_window(trace_dir: str, spec: str):
    """(name, first, count, average ms) over a slice of one kernel's dispatches."""
    name, first, count = spec.rsplit(":", 2)
    first, count = int(first), int(count)
    rows = [r for r in csv.DictReader(open(_one(os.path.join(trace_dir, "*kernel_trace.csv"))))
            if name in r["Kernel_Name"]]
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    sel = rows[first:first + count]
    if len(sel) != count:
        raise ValueError(f"{spec}: the trace holds {len(rows)} dispatches of {name}")
    ms = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e6 for r in sel]
    return name, first, count, sum(ms) / count


def counter_per_dispatch(pmc_dir: str, counter: str):
    """{kernel short name: [value per dispatch]} for the gather, scatter and plain copy."""
    out = defaultdict(list)
    for r in csv.DictReader(open(_one(os.path.join(pmc_dir, "*counter_collection.csv")))):
        if r["Counter_Name"] != counter:
            continue
        name = r["Kernel_Name"]
        for key in (GATHER, SCATTER, PLAIN_COPY):
            if key in name:
                out[key].append(float(r["Counter_Value"]))
    return out


def plain_copy_value(vals):
    """The 8 GiB copy dispatches (the largest plain-copy dispatches of the run)."""
    top = max(vals)
    return [v for v in vals if v > 0.9 * top]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace", required=True)
    ap.add_argument("--fetch", default=None)
    ap.add_argument("--write", default=None)
    ap.add_argument("--bench", default=None, help="bench.py JSON line of a counter run")
    ap.add_argument("--trace-bench", default=None, help="bench.py JSON line of the trace run")
    ap.add_argument("--out", default=os.path.join(os.path.dirname(HERE), "profiles"))
    ap.add_argument("--name", default="gather_llama8b")
    ap.add_argument("--cmd", required=True, help="the command that produced the inputs")
    ap.add_argument("--pmc", action="append", default=[], help="a --pmc run directory")
    ap.add_argument("--window", action="append", default=[],
                    help="NAME:FIRST:COUNT, the average over a slice of one kernel's dispatches")
    a = ap.parse_args()
    if a.pmc:
        return store_counters(a)
    if not (a.fetch and a.write and a.bench):
        return store_kernels_only(a)

    bench = json.loads(open(a.bench).read().strip().splitlines()[-1])
    algo = bench["roofline"]["bytes_per_launch"]
    fetch = counter_per_dispatch(a.fetch, "FETCH_SIZE")
    write = counter_per_dispatch(a.write, "WRITE_SIZE")
    pf = plain_copy_value(fetch[PLAIN_COPY])
    pw = plain_copy_value(write[PLAIN_COPY])
    known_kib = bench["hbm_ceiling"]["bytes"] / 1024  # the plain copy's size in that run
    f_factor = known_kib / (sum(pf) / len(pf))
    w_factor = known_kib / (sum(pw) / len(pw))
    g_fetch = sum(fetch[GATHER]) / len(fetch[GATHER])
    g_write = sum(write[GATHER]) / len(write[GATHER])
    traffic = (g_fetch * f_factor + g_write * w_factor) * 1024
    stats = kernel_stats(a.trace)

    os.makedirs(a.out, exist_ok=True)
    rec = {
        "kernel": GATHER,
        "workload": bench["config"]["workload"],
        "copy_hip_sha256": copy_source_sha(),
        "fetch_kib_per_dispatch": round(g_fetch, 1),
        "write_kib_per_dispatch": round(g_write, 1),
        "fetch_factor": round(f_factor, 4),
        "write_factor": round(w_factor, 4),
        "traffic_bytes_per_launch": int(traffic),
        "algorithmic_bytes_per_launch": int(algo),
        "traffic_over_algorithmic": round(traffic / algo, 4),
        "dispatches": len(fetch[GATHER]),
    }
    with open(os.path.join(a.out, f"{a.name}_traffic.json"), "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")

    lines = [f"# Kernel trace: {a.name}", "", "Command (run from the repository root on the MI355X host):", "",
             "```", a.cmd.strip(), "```", "",
             "| kernel | calls | avg ms | % of GPU time |", "|---|---|---|---|"]
    for name, calls, avg, pct in stats[:12]:
        short = name if len(name) < 70 else name[:67] + "..."
        lines.append(f"| `{short}` | {calls} | {avg:.4f} | {pct:.2f} |")
    g = [s for s in stats if GATHER in s[0]]
    if g:
        lines += ["", f"Gather kernel average over {g[0][1]} dispatches: **{g[0][2]:.4f} ms**."]
    if a.trace_bench:
        tb = json.loads(open(a.trace_bench).read().strip().splitlines()[-1])["roofline"]
        lines += [f"bench.py's own HIP-event average in the same run: **{tb['avg_launch_ms']:.4f} ms** "
                  f"over {tb['launches']} timed launches ({tb['achieved']:.1f} GB/s, "
                  f"{100 * tb['frac']:.1f}% of 8 TB/s)."]
    with open(os.path.join(a.out, f"{a.name}_kernel_trace.md"), "w") as f:
        f.write("\n".join(lines) + "\n")

    lines = [f"# HBM traffic: {a.name}", "", "Commands (repository root, on the MI355X host):", "", "```",
             a.cmd.strip(), "```", "",
             "| quantity | value |", "|---|---|",
             f"| gather FETCH_SIZE per dispatch | {g_fetch:,.0f} KiB ({len(fetch[GATHER])} dispatches) |",
             f"| gather WRITE_SIZE per dispatch | {g_write:,.0f} KiB |",
             f"| plain {known_kib / 2**20:.0f} GiB copy FETCH_SIZE | {sum(pf) / len(pf):,.0f} KiB -> factor {f_factor:.4f} |",
             f"| plain {known_kib / 2**20:.0f} GiB copy WRITE_SIZE | {sum(pw) / len(pw):,.0f} KiB -> factor {w_factor:.4f} |",
             f"| traffic per gather launch (scaled) | {traffic / 1e9:.3f} GB |",
             f"| algorithmic bytes per launch | {algo / 1e9:.3f} GB |",
             f"| traffic / algorithmic | {traffic / algo:.4f} |",
             "", f"Copy kernel source SHA-256: `{rec['copy_hip_sha256']}`."]
    with open(os.path.join(a.out, f"{a.name}_hbm_counters.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print(json.dumps(rec))


def short_name(name: str) -> str:
    short = name.replace("ptsd::(anonymous namespace)::", "").replace("void ", "")
    return short.replace("(anonymous namespace)::", "").split("(")[0]


def store_counters(a):
    """Per-kernel averages of the counters of one or more --pmc runs."""
    vals = defaultdict(lambda: defaultdict(list))  # kernel -> counter -> values
    order = []
    for d in a.pmc:
        for r in csv.DictReader(open(_one(os.path.join(d, "*counter_collection.csv")))):
            if "ptsd::" not in r["Kernel_Name"]:
                continue
            c = r["Counter_Name"]
            if c not in order:
                order.append(c)
            vals[short_name(r["Kernel_Name"])][c].append(float(r["Counter_Value"]))
    hit = "TCC_HIT_sum" in order and "TCC_MISS_sum" in order
    head = ["kernel", "dispatches"] + [f"{c} / dispatch" for c in order] + (["L2 hit rate"] if hit else [])
    lines = [f"# Counters: {a.name}", "", "Commands (run from the repository root on the MI355X host):",
             "", "```", a.cmd.strip(), "```", "",
             "Averages per dispatch over every dispatch of the runs (FETCH_SIZE in KiB, "
             "unscaled).", "",
             "| " + " | ".join(head) + " |", "|" + "---|" * len(head)]
    rows = sorted(vals.items(), key=lambda kv: -sum(kv[1].get("FETCH_SIZE", [0])))
    for k, cs in rows:
        n = max(len(v) for v in cs.values())
        cells = [f"`{k}`", str(n)]
        for c in order:
            v = cs.get(c)
            cells.append(f"{sum(v) / len(v):,.1f}" if v else "")
        if hit:
            h, m = sum(cs.get("TCC_HIT_sum", [0])), sum(cs.get("TCC_MISS_sum", [0]))
            cells.append(f"{h / (h + m):.3f}" if h + m else "")
        lines.append("| " + " | ".join(cells) + " |")
    if a.bench:
        tb = json.loads(open(a.bench).read().strip().splitlines()[-1])
        extra = {k: tb[k] for k in ("lookup_only", "library_counters") if k in tb}
        if extra:
            lines += ["", "bench.py in the first counter run (its own library counters; its "
                      "timings are not the kernels' own, since counter collection serialises "
                      "and lengthens every dispatch):", "", "```",
                      json.dumps(extra, indent=1), "```"]
    os.makedirs(a.out, exist_ok=True)
    with open(os.path.join(a.out, f"{a.name}_counters.md"), "w") as f:
        f.write("\n".join(lines) + "\n")


def store_kernels_only(a):
    """Per-kernel table of every store kernel in a trace run, plus the
    per-round kernel times bench.py measured with HIP events in that run."""
    stats = kernel_stats(a.trace)
    lines = [f"# Kernel trace: {a.name}", "", "Command (run from the repository root on the MI355X host):", "",
             "```", a.cmd.strip(), "```", "",
             "| kernel | calls | avg us | % of GPU time |", "|---|---|---|---|"]
    for name, calls, avg, pct in stats:
        if "ptsd::" not in name:
            continue
        short = short_name(name)
        lines.append(f"| `{short}` | {calls} | {avg * 1e3:.2f} | {pct:.2f} |")
    if a.trace_bench:
        tb = json.loads(open(a.trace_bench).read().strip().splitlines()[-1])
        lines += ["", f"bench.py in the same run: {tb['value']} {tb['unit']}, "
                  f"{tb['ms_per_step']} ms per step; kernel time per step (HIP events, ms):", ""]
        for k, v in tb.get("kernel_ms_per_round", {}).items():
            lines.append(f"- {k}: {v}")
        if "evictions" in tb:
            lines.append(f"- evictions in the warm-up and timed steps: {tb['evictions']}; "
                         f"index rebuilds in the timed steps: {tb['index_rebuilds']}")
        if "lookup_only" in tb:
            lo = tb["lookup_only"]
            lines.append(f"- lookup only (counters off): {lo['kernel_avg_ms']} ms per call, "
                         f"{lo['lookups_per_s_kernel']:,.0f} lookups/s at the kernel")
        if "roofline" in tb and not tb.get("kernel_ms_per_round"):
            rf = tb["roofline"]
            lines.append(f"- gather: {rf['avg_launch_ms']} ms per launch over {rf['launches']} "
                         f"timed launches ({rf['achieved']} GB/s)")
    for spec in a.window:
        name, first, count, avg = dispatch_window(a.trace, spec)
        lines += ["", f"`{name}` dispatches {first}-{first + count - 1} (start order) in the trace: "
                  f"**{avg:.4f} ms** average."]
    os.makedirs(a.out, exist_ok=True)
    with open(os.path.join(a.out, f"{a.name}_kernel_trace.md"), "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
