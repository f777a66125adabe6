"""Host-side tools: bench.py's argument contract and the rocprofv3 summariser (no GPU)."""
from __future__ import annotations

import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert p.returncode == 2
    line = json.loads(p.stdout.strip().splitlines()[-1])
    assert "one GPU" in line["error"]


def _write_trace(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_kernel_stats.csv"), "w") as f:
        f.write('"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs","StdDev"\n')
        for name, calls, avg, pct in rows:
            f.write(f'"{name}",{calls},{calls * avg},{avg},{pct},{avg},{avg},0\n')


def _write_pmc(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w") as f:
        f.write('"Kernel_Name","Counter_Name","Counter_Value"\n')
        for k, c, v in rows:
            f.write(f'"{k}","{c}",{v}\n')


def test_profile_summary_traffic(tmp_path):
    """Traffic = FETCH_SIZE and WRITE_SIZE scaled by what the bench's read and
    write probes of known size read for them in the same runs, against the
    algorithmic bytes summed over every gather dispatch; and, independently,
    memory requests times their sizes, checked on the probes too."""
    ns = "void ptsd::(anonymous namespace)::"
    gather = ns + "k_copy_slices(ptsd::(anonymous namespace)::CopyArgs)"
    rd = ns + "k_read(unsigned int __vector(4) const*, long, unsigned int __vector(4)*)"
    wrk = ns + "k_write(unsigned int __vector(4)*, long)"
    gib = 1 << 30
    fe, wr, rq, wq = (tmp_path / n for n in ("fetch", "write", "reqs", "wreqs"))
    # FETCH_SIZE reads half the KiB of a pure read (factor 2), WRITE_SIZE all of a
    # pure write (factor 1); four gathers of 3 GiB read + 3 GiB written, then a
    # fifth dispatch of 1 GiB + 1 GiB: 26 GiB algorithmic in all
    g_r = [3 * gib] * 4 + [gib]
    _write_pmc(str(fe), [(rd, "FETCH_SIZE", gib / 1024 / 2)] * 2 +
               [(gather, "FETCH_SIZE", b / 1024 / 2) for b in g_r])
    _write_pmc(str(wr), [(wrk, "WRITE_SIZE", gib / 1024)] * 2 +
               [(gather, "WRITE_SIZE", b / 1024) for b in g_r])
    # reads in 128-byte requests (a few 64 and 32 byte ones), writes in 64-byte ones
    req = []
    for k, b in [(rd, gib)] + [(gather, b) for b in g_r]:
        req += [(k, "TCC_EA0_RDREQ_sum", (b - 96) / 128 + 2), (k, "TCC_EA0_RDREQ_32B_sum", 1),
                (k, "TCC_EA0_RDREQ_64B_sum", 1), (k, "TCC_EA0_RDREQ_128B_sum", (b - 96) / 128)]
    _write_pmc(str(rq), req)
    _write_pmc(str(wq), [(k, c, v) for k, b in [(wrk, gib)] + [(gather, b) for b in g_r]
                         for c, v in (("TCC_EA0_WRREQ_sum", b / 64), ("TCC_EA0_WRREQ_64B_sum", b / 64))])
    bench = tmp_path / "bench.json"
    bench.write_text(json.dumps({"roofline": {"bytes_per_launch": 26 * gib / 5},
                                 "gather_all": {"dispatches": 5, "bytes": 26 * gib},
                                 "hbm_ceiling": {"bytes": gib},
                                 "config": {"workload": "synthetic"}}) + "\n")
    out = tmp_path / "profiles"
    args = [sys.executable, "-m", "paper_2607_22648_amd.profile_summary", "--fetch", str(fe),
            "--write", str(wr), "--reqs", str(rq), "--wreqs", str(wq), "--bench", str(bench),
            "--out", str(out), "--name", "t", "--cmd", "cmd"]
    p = subprocess.run(args, capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert p.returncode == 0, p.stderr
    rec = json.loads((out / "t_traffic.json").read_text())
    assert rec["fetch_factor"] == 2.0 and rec["write_factor"] == 1.0
    assert rec["dispatches"] == 5 and rec["traffic_over_algorithmic"] == 1.0
    assert rec["traffic_bytes_per_launch"] == round(26 * gib / 5)
    assert rec["raw_fetch_kib_per_dispatch"] == round(26 * gib / 2 / 1024 / 2 / 5, 1)
    assert rec["request_traffic_over_algorithmic"] == 1.0
    assert rec["probe_check"]["read_probe_bytes_from_requests_over_known"] == 1.0
    assert rec["probe_check"]["write_probe_bytes_from_requests_over_known"] == 1.0
    assert rec["probe_check"]["read_requests_covered_by_size_classes"] == 1.0
    assert "cmd" in (out / "t_hbm_counters.md").read_text()
    # a run whose gather dispatches differ from what bench.py counted is refused
    bench.write_text(json.dumps({"roofline": {"bytes_per_launch": 1}, "gather_all": {"dispatches": 4, "bytes": 1},
                                 "hbm_ceiling": {"bytes": gib}, "config": {"workload": "x"}}) + "\n")
    p = subprocess.run(args, capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert p.returncode != 0 and "gather dispatches" in p.stderr


def test_profile_summary_counters(tmp_path):
    """Per-kernel averages of any counters, and the L2 hit rate."""
    k = "void ptsd::(anonymous namespace)::k_lookup<16, false>(ptsd::IndexView, ptsd::Batch, int*, int*)"
    d = tmp_path / "pmc"
    _write_pmc(str(d), [(k, "TCC_HIT_sum", 30), (k, "TCC_MISS_sum", 10),
                        (k, "TCC_HIT_sum", 50), (k, "TCC_MISS_sum", 10),
                        ("void at::native::other", "TCC_HIT_sum", 1)])
    out = tmp_path / "profiles"
    p = subprocess.run([sys.executable, "-m", "paper_2607_22648_amd.profile_summary", "--trace", "x",
                        "--pmc", str(d), "--out", str(out), "--name", "c", "--cmd", "cmd"],
                       capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert p.returncode == 0, p.stderr
    text = (out / "c_counters.md").read_text()
    row = [l for l in text.splitlines() if "k_lookup<16, false>" in l][0]
    cells = [c.strip() for c in row.strip("|").split("|")]
    assert cells[1] == "2"                      # dispatches
    assert cells[2] == "40.0" and cells[3] == "10.0"  # averages of HIT and MISS
    assert cells[4] == "0.800"                  # 80 hits of 100
    assert "at::native" not in text


def test_profile_summary_dispatch_window(tmp_path):
    """--window averages one slice of a kernel's dispatches, in start order,
    from the per-dispatch trace; the other kernels and dispatches stay out."""
    look = "void ptsd::(anonymous namespace)::k_lookup<16, false>(ptsd::IndexView, ptsd::Batch, int*, int*)"
    other = "void ptsd::(anonymous namespace)::k_publish(ptsd::(anonymous namespace)::InsertArgs)"
    tr = tmp_path / "trace"
    _write_trace(str(tr), [(look, 6, 30_000, 80.0), (other, 2, 5_000, 20.0)])
    # dispatches in shuffled file order: start times 0..5 ms, durations 100, 10, 20, 30, 40, 100 us
    rows = [(look, 5, 100), (other, 1, 7), (look, 0, 100), (look, 3, 30), (look, 1, 10), (look, 4, 40),
            (look, 2, 20), (other, 2, 9)]
    with open(tr / "run_kernel_trace.csv", "w") as f:
        f.write('"Kernel_Name","Start_Timestamp","End_Timestamp"\n')
        for k, start_ms, dur_us in rows:
            s0 = start_ms * 1_000_000 + (500_000 if k == other else 0)
            f.write(f'"{k}",{s0},{s0 + dur_us * 1000}\n')
    out = tmp_path / "profiles"
    p = subprocess.run([sys.executable, "-m", "paper_2607_22648_amd.profile_summary", "--trace", str(tr),
                        "--window", "k_lookup<16, false>:1:4", "--out", str(out), "--name", "w",
                        "--cmd", "cmd"], capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert p.returncode == 0, p.stderr
    text = (out / "w_kernel_trace.md").read_text()
    assert "dispatches 1-4" in text and "**0.0250 ms** average" in text  # (10+20+30+40)/4 us
    p = subprocess.run([sys.executable, "-m", "paper_2607_22648_amd.profile_summary", "--trace", str(tr),
                        "--window", "k_lookup<16, false>:3:4", "--out", str(out), "--name", "w",
                        "--cmd", "cmd"], capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert p.returncode != 0 and "holds 6 dispatches" in p.stderr  # a slice past the end is refused


def test_profile_summary_trace_bench_lines(tmp_path):
    """The trace summary quotes the bench line of the same run: a gather's
    average launch against the HBM, or, for the tiered store, the host link's
    rate and the average over every gather launch."""
    gather = "void ptsd::(anonymous namespace)::k_copy_slices(ptsd::(anonymous namespace)::CopyArgs)"
    tr = tmp_path / "trace"
    _write_trace(str(tr), [(gather, 4, 12_500_000, 90.0)])
    out = tmp_path / "profiles"
    lines = {
        "hbm": {"value": 10.0, "unit": "requests/s", "ms_per_step": 25.0,
                "roofline": {"bound": "hbm", "kernel": "k_copy_slices (gather)", "achieved": 6500.0,
                             "peak": 8000.0, "unit": "GB/s", "frac": 0.8125, "avg_launch_ms": 12.5,
                             "launches": 40}},
        "link": {"value": 89.0, "unit": "requests/s", "ms_per_step": 719.0,
                 "roofline": {"bound": "host link", "kernel": "k_copy_slices (gather, host-tier rows)",
                              "achieved": 56.0, "peak": 64.0, "unit": "GB/s", "frac": 0.875},
                 "gather_all_launches": {"avg_launch_ms": 21.9, "launches": 128}},
    }
    for name, line in lines.items():
        b = tmp_path / f"{name}.json"
        b.write_text("[bench] log line\n" + json.dumps(line) + "\n")
        p = subprocess.run([sys.executable, "-m", "paper_2607_22648_amd.profile_summary", "--trace", str(tr),
                            "--trace-bench", str(b), "--out", str(out), "--name", name, "--cmd", "cmd"],
                           capture_output=True, text=True, cwd=ROOT, timeout=120)
        assert p.returncode == 0, p.stderr
    text = (out / "hbm_kernel_trace.md").read_text()
    assert "`k_copy_slices` | 4 | 12500.00" in text
    assert "- gather: 12.5 ms per launch over 40 timed launches (6500.0 GB/s)" in text
    text = (out / "link_kernel_trace.md").read_text()
    assert "56.0 GB/s over the host link (0.875 of 64.0 GB/s)" in text
    assert "21.9 ms per launch over 128 launches" in text


def test_copy_code_hash_ignores_comments_only(tmp_path, monkeypatch):
    """The counter records are keyed to the copy kernels' code: editing a
    comment or the spacing keeps the key, changing code changes it, and
    bench.py reports the recorded traffic only under the same key."""
    sys.path.insert(0, ROOT)
    from paper_2607_22648_amd import profile_summary as ps
    src = open(ps.COPY_SRC).read()
    base = ps.copy_source_sha()
    variants = {
        "comment": src.replace("#include", "// a new comment line\n#include", 1),
        "block comment": src.replace("#include", "/* a block\n   comment */ #include", 1),
        "spacing": src.replace("\n", "\n\n", 5),
        "code": src.replace("kUnroll = 8", "kUnroll = 4", 1),
    }
    keys = {}
    for name, text in variants.items():
        f = tmp_path / f"{name.replace(' ', '_')}.hip"
        f.write_text(text)
        monkeypatch.setattr(ps, "COPY_SRC", str(f))
        keys[name] = ps.copy_source_sha()
    assert keys["comment"] == base and keys["block comment"] == base and keys["spacing"] == base
    assert keys["code"] != base
    monkeypatch.undo()
    hdr = open(ps.COPY_HDR).read()
    f = tmp_path / "kernels.hpp"
    f.write_text(hdr.replace("kSliceDests = 64", "kSliceDests = 32", 1))
    monkeypatch.setattr(ps, "COPY_HDR", str(f))
    assert ps.copy_source_sha() != base  # the copy kernels' constants are part of the key
    monkeypatch.undo()
    import bench
    monkeypatch.setattr(ps, "COPY_SRC", str(tmp_path / "code.hip"))
    assert bench.recorded_traffic("llama8b", 1e9) is None
    monkeypatch.undo()
    rec = json.load(open(os.path.join(ROOT, "profiles", "gather_llama8b_traffic.json")))
    if rec.get("copy_code_sha256") == base:
        assert bench.recorded_traffic("llama8b", 1e9) == round(rec["traffic_over_algorithmic"] * 1e9)
