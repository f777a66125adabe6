"""Summarise rocprofv3 output of bench.py into short text notes under profiles/.

Inputs (directories written by rocprofv3 ``--output-format csv``):
  --trace DIR   a ``--kernel-trace --stats`` run (uses *_kernel_stats.csv):
                the per-kernel table of the store's own kernels
  --window NAME:FIRST:COUNT  (repeatable, with --trace) the average
                duration of dispatches FIRST .. FIRST+COUNT-1, in start order,
                of the kernel whose name contains NAME (*_kernel_trace.csv):
                the launches a bench phase timed, apart from other launches
                of the same kernel in the run
  --fetch DIR, --write DIR  ``--pmc FETCH_SIZE`` and ``--pmc WRITE_SIZE`` runs,
                with --bench FILE, the JSON line bench.py printed in them:
                the gather's HBM traffic record (below)
  --reqs DIR    (optional, with --fetch) a ``--pmc TCC_EA0_RDREQ
                TCC_EA0_RDREQ_32B TCC_EA0_RDREQ_64B TCC_EA0_RDREQ_128B`` run,
  --wreqs DIR   and a ``--pmc TCC_EA0_WRREQ TCC_EA0_WRREQ_64B ...`` run: the
                same traffic counted from memory requests times their sizes
  --pmc DIR     (repeatable, instead of the above) any ``--pmc`` runs: the
                average per dispatch of every counter collected, for every
                store kernel, plus the L2 hit rate where TCC_HIT and TCC_MISS
                were both collected

HBM traffic of the gather. FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are
each scaled by the factor that maps the same counter onto the known byte
count of the bench's own bandwidth probes in the same run: a pure read
stream (ptstore_bandwidth_probe kind 0, ``k_read``) and a pure write stream
(kind 1, ``k_write``) of ``hbm_ceiling.bytes`` each, as the run's JSON line
states. The raw counts, the factors and, for comparison, the factors a plain
device-to-device copy (``__amd_rocclr_copyBuffer``) gives are all recorded.
Independently of any factor, the request counters give bytes as requests x
request size (32, 64 or 128 bytes; a write request is 64 bytes if counted as
such, else 32), checked against the probes' known bytes as well. Traffic
is compared with the algorithmic bytes summed over every gather dispatch of
the run (the JSON line's ``gather_all``). The record carries the SHA-256 of
the copy kernels' code (csrc/copy.hip and csrc/kernels.hpp); bench.py
reports the traffic only while that code is unchanged.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
from collections import defaultdict

HERE = os.path.dirname(os.path.abspath(__file__))
COPY_SRC = os.path.join(HERE, "csrc", "copy.hip")
COPY_HDR = os.path.join(HERE, "csrc", "kernels.hpp")  # the copy kernels' shared types and constants
GATHER = "k_copy_slices("
SCATTER = "k_copy_pairs("
PLAIN_COPY = "__amd_rocclr_copyBuffer"


def _code(path: str) -> str:
    """A source file with comments dropped and whitespace runs collapsed."""
    src = open(path).read()
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return " ".join(src.split())


def copy_source_sha() -> str:
    """SHA-256 of the copy kernels' code: csrc/copy.hip and the header of
    their shared types and constants (csrc/kernels.hpp), comments dropped and
    whitespace runs collapsed, so that editing a comment does not void the
    counter records taken on that code."""
    code = _code(COPY_SRC) + "\n" + _code(COPY_HDR)
    return hashlib.sha256(code.encode()).hexdigest()


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


PROBE_READ = "k_read("
PROBE_WRITE = "k_write("


def kernel_key(name: str):
    """The short key of a kernel this summary tracks, or None."""
    for key in (GATHER, "k_copy_spans<true>", SCATTER, PROBE_READ, PROBE_WRITE, PLAIN_COPY):
        if key in name:
            return key
    return None


def counters_by_kernel(pmc_dir: str):
    """{kernel key: {counter: [value per dispatch, in file order]}}."""
    out = defaultdict(lambda: defaultdict(list))
    for r in csv.DictReader(open(_one(os.path.join(pmc_dir, "*counter_collection.csv")))):
        key = kernel_key(r["Kernel_Name"])
        if key:
            c = r["Counter_Name"].replace("_sum", "")
            out[key][c].append(float(r["Counter_Value"]))
    return out


def plain_copy_value(vals):
    """The large plain-copy dispatches (the largest of the run)."""
    top = max(vals)
    return [v for v in vals if v > 0.9 * top]


def mean(v):
    return sum(v) / len(v)


def read_bytes(cs, k):
    """Read bytes of dispatch k from the request counters: requests x size."""
    r32, r64, r128 = (cs[c][k] for c in ("TCC_EA0_RDREQ_32B", "TCC_EA0_RDREQ_64B", "TCC_EA0_RDREQ_128B"))
    return 32 * r32 + 64 * r64 + 128 * r128


def write_bytes(cs, k):
    w, w64 = cs["TCC_EA0_WRREQ"][k], cs["TCC_EA0_WRREQ_64B"][k]
    return 64 * w64 + 32 * (w - w64)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace", default=None)
    ap.add_argument("--fetch", default=None)
    ap.add_argument("--write", default=None)
    ap.add_argument("--reqs", default=None, help="a --pmc run of the read request counters")
    ap.add_argument("--wreqs", default=None, help="a --pmc run of the write request counters")
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
    if a.fetch and a.write and a.bench:
        return gather_traffic(a)
    return store_kernels_only(a)


def gather_traffic(a):
    bench = json.loads(open(a.bench).read().strip().splitlines()[-1])
    known = bench["hbm_ceiling"]["bytes"]  # bytes of each probe dispatch
    fe, wr = counters_by_kernel(a.fetch), counters_by_kernel(a.write)
    gk = GATHER if GATHER in fe else "k_copy_spans<true>"
    f_factor = known / 1024 / mean(fe[PROBE_READ]["FETCH_SIZE"])
    w_factor = known / 1024 / mean(wr[PROBE_WRITE]["WRITE_SIZE"])
    cf = cw = None
    if PLAIN_COPY in fe and PLAIN_COPY in wr:
        cf = known / 1024 / mean(plain_copy_value(fe[PLAIN_COPY]["FETCH_SIZE"]))
        cw = known / 1024 / mean(plain_copy_value(wr[PLAIN_COPY]["WRITE_SIZE"]))
    g_fetch, g_write = fe[gk]["FETCH_SIZE"], wr[gk]["WRITE_SIZE"]
    n = len(g_fetch)
    ga = bench.get("gather_all")
    if ga:  # algorithmic bytes over every gather dispatch of the run
        if ga["dispatches"] != n:
            raise ValueError(f"the run holds {n} gather dispatches, bench.py counted {ga['dispatches']}")
        algo_total = ga["bytes"]
        algo_read = ga.get("read_bytes", algo_total / 2)
    else:
        algo_total = bench["roofline"]["bytes_per_launch"] * n
        algo_read = algo_total / 2
    algo_write = algo_total - algo_read
    traffic_total = (sum(g_fetch) * f_factor + sum(g_write) * w_factor) * 1024
    ratio = traffic_total / algo_total
    per_launch = bench["roofline"]["bytes_per_launch"]
    rec = {
        "kernel": gk,
        "workload": bench["config"]["workload"],
        "copy_code_sha256": copy_source_sha(),
        "dispatches": n,
        "raw_fetch_kib_per_dispatch": round(mean(g_fetch), 1),
        "raw_write_kib_per_dispatch": round(mean(g_write), 1),
        "fetch_factor": round(f_factor, 4),
        "write_factor": round(w_factor, 4),
        "factor_source": f"bandwidth probes of {known} bytes (read kind 0, write kind 1) in the same runs",
        "plain_copy_factors": [round(cf, 4), round(cw, 4)] if cf else None,
        "algorithmic_bytes_all_dispatches": int(algo_total),
        "traffic_bytes_all_dispatches": int(traffic_total),
        "traffic_over_algorithmic": round(ratio, 4),
        "algorithmic_bytes_per_launch": int(per_launch),
        "traffic_bytes_per_launch": int(round(ratio * per_launch)),
    }
    lines_req = []
    if a.reqs and a.wreqs:
        rq, wq = counters_by_kernel(a.reqs), counters_by_kernel(a.wreqs)
        if len(rq[gk]["TCC_EA0_RDREQ_32B"]) != n or len(wq[gk]["TCC_EA0_WRREQ"]) != n:
            raise ValueError("the request runs hold another number of gather dispatches")
        rd = sum(read_bytes(rq[gk], k) for k in range(n))
        wb = sum(write_bytes(wq[gk], k) for k in range(n))
        probe_rd = mean([read_bytes(rq[PROBE_READ], k) for k in range(len(rq[PROBE_READ]["TCC_EA0_RDREQ_32B"]))])
        probe_wr = mean([write_bytes(wq[PROBE_WRITE], k) for k in range(len(wq[PROBE_WRITE]["TCC_EA0_WRREQ"]))])
        cover = sum(rq[gk]["TCC_EA0_RDREQ_32B"][k] + rq[gk]["TCC_EA0_RDREQ_64B"][k] +
                    rq[gk]["TCC_EA0_RDREQ_128B"][k] for k in range(n)) / sum(rq[gk]["TCC_EA0_RDREQ"])
        rec.update({
            "request_read_bytes_all_dispatches": int(rd),
            "request_write_bytes_all_dispatches": int(wb),
            "request_traffic_over_algorithmic": round((rd + wb) / algo_total, 4),
            "request_read_over_algorithmic_read": round(rd / algo_read, 4),
            "request_write_over_algorithmic_write": round(wb / algo_write, 4),
            "probe_check": {"read_probe_bytes_from_requests_over_known": round(probe_rd / known, 4),
                            "write_probe_bytes_from_requests_over_known": round(probe_wr / known, 4),
                            "read_requests_covered_by_size_classes": round(cover, 4)},
        })
        if "TCC_EA0_WRREQ_DRAM_CREDIT_STALL" in wq[gk]:
            w_all = sum(wq[gk]["TCC_EA0_WRREQ"])
            rec["dram_credit_stalls_per_write_request"] = {
                "read": round(sum(wq[gk]["TCC_EA0_RDREQ_DRAM_CREDIT_STALL"]) / w_all, 4),
                "write": round(sum(wq[gk]["TCC_EA0_WRREQ_DRAM_CREDIT_STALL"]) / w_all, 4)}
        lines_req = [
            f"| gather read bytes from requests (32/64/128 B classes) | {rd / n / 1e9:.3f} GB per dispatch |",
            f"| gather write bytes from requests (64 B, else 32 B) | {wb / n / 1e9:.3f} GB per dispatch |",
            f"| request bytes / algorithmic | {(rd + wb) / algo_total:.4f} (read {rd / algo_read:.4f}, "
            f"write {wb / algo_write:.4f}) |",
            f"| check: read probe bytes from requests / known | {probe_rd / known:.4f} |",
            f"| check: write probe bytes from requests / known | {probe_wr / known:.4f} |",
            f"| read requests counted in a size class | {cover:.4f} |"]
        if "dram_credit_stalls_per_write_request" in rec:
            st = rec["dram_credit_stalls_per_write_request"]
            lines_req.append(f"| DRAM credit stalls per write request (read, write) | "
                             f"{st['read']:.4f}, {st['write']:.4f} |")
    os.makedirs(a.out, exist_ok=True)
    with open(os.path.join(a.out, f"{a.name}_traffic.json"), "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    lines = [f"# HBM traffic: {a.name}", "", "Commands (repository root, on the MI355X host):", "", "```",
             a.cmd.strip(), "```", "",
             "| quantity | value |", "|---|---|",
             f"| gather dispatches in the run | {n} |",
             f"| gather FETCH_SIZE, raw | {mean(g_fetch):,.0f} KiB per dispatch |",
             f"| gather WRITE_SIZE, raw | {mean(g_write):,.0f} KiB per dispatch |",
             f"| read probe ({known / 2**30:.0f} GiB) FETCH_SIZE | {mean(fe[PROBE_READ]['FETCH_SIZE']):,.0f} KiB -> factor {f_factor:.4f} |",
             f"| write probe ({known / 2**30:.0f} GiB) WRITE_SIZE | {mean(wr[PROBE_WRITE]['WRITE_SIZE']):,.0f} KiB -> factor {w_factor:.4f} |"]
    if cf:
        lines.append(f"| plain copy factors, for comparison | FETCH {cf:.4f}, WRITE {cw:.4f} |")
    lines += [f"| traffic, all gather dispatches (scaled) | {traffic_total / 1e9:.3f} GB |",
              f"| algorithmic bytes, all gather dispatches | {algo_total / 1e9:.3f} GB |",
              f"| traffic / algorithmic | {ratio:.4f} |"] + lines_req + [
              "", f"Copy kernel code SHA-256 (csrc/copy.hip and csrc/kernels.hpp without comments and whitespace): `{rec['copy_code_sha256']}`."]
    with open(os.path.join(a.out, f"{a.name}_hbm_counters.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print(json.dumps(rec))


def short_name(name: str) -> str:
    short = name.replace("ptsd::(anonymous namespace)::", "").replace("void ", "")
    return short.replace("(anonymous namespace)::", "").split("(")[0]


def store_counters(a):
    """Per-kernel averages of the counters of one or more --pmc runs."""
    vals = defaultdict(lambda: defaultdict(list))  # (kernel, grid) -> counter -> values
    order = []
    for d in a.pmc:
        for r in csv.DictReader(open(_one(os.path.join(d, "*counter_collection.csv")))):
            if "ptsd::" not in r["Kernel_Name"]:
                continue
            c = r["Counter_Name"]
            if c not in order:
                order.append(c)
            vals[(short_name(r["Kernel_Name"]), int(r.get("Grid_Size") or 0))][c].append(
                float(r["Counter_Value"]))
    # a kernel launched at several grid sizes (say a lookup of a timed batch and
    # the lookups inside the prefill's inserts) gets a row per grid size
    grids = defaultdict(set)
    for k, g in vals:
        grids[k].add(g)
    vals = {(f"{k} (grid {g:,})" if len(grids[k]) > 1 else k): v for (k, g), v in vals.items()}
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
            if "avg_launch_ms" in rf:
                lines.append(f"- gather: {rf['avg_launch_ms']} ms per launch over {rf['launches']} "
                             f"timed launches ({rf['achieved']} GB/s)")
            else:  # bound by the host link: bytes per step over the time the link carries them
                lines.append(f"- {rf['kernel']}: {rf['achieved']} {rf['unit']} over the {rf['bound']} "
                             f"({rf['frac']} of {rf['peak']} {rf['unit']})")
            ga = tb.get("gather_all_launches")
            if ga:
                lines.append(f"- every gather launch, host-tier and device rows: {ga['avg_launch_ms']} ms "
                             f"per launch over {ga['launches']} launches")
    for spec in a.window:
        name, first, count, avg = dispatch_window(a.trace, spec)
        lines += ["", f"`{name}` dispatches {first}-{first + count - 1} (start order) in the trace: "
                  f"**{avg:.4f} ms** average."]
    os.makedirs(a.out, exist_ok=True)
    with open(os.path.join(a.out, f"{a.name}_kernel_trace.md"), "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
