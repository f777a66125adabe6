#!/usr/bin/env python3
"""Prefix lookup + KV gather throughput on one MI355X.

A step is one pass of the hot path over the workload's request batch:
chained block hashing, index probing with parent verification, the
longest-common-prefix decision, and the gather of the matched KV blocks into
a paged cache (ptstore_lookup_gather, issued per sub-batch). The store is
built beforehand through the same library's insert + scatter (timed
separately and reported under "prefill").

Default workload: Llama-3-8B-shaped KV (32 layers x 8 KV heads x 128, bf16,
16-token blocks); 256 requests of 4096 tokens = one of 512 passages of 3584
tokens (Zipf s=1.1) + 512 fresh tokens; the store holds the 256 most
popular passages (57,344 blocks, 120 GB); two sub-batches of 128 requests
share one 68.7 GB paged cache.

Prints one JSON line. ``value`` = requests/s of the whole job, inputs resident
in HBM. ``roofline`` = the gather kernel's algorithmic bytes (one pool read of
each distinct stored block a call needs + one cache write of every matched
block) over its average duration, measured with HIP events the library
records on the launch stream. ``cpu_baseline`` = the
CPU oracle, single-threaded, on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
# the host link of the tiered store: PCIe 5.0 x16, 64 GB/s per direction
HOST_LINK_PEAK_GBPS = 64.0
METRIC = "prefix lookup+KV gather: requests/s and achieved HBM GB/s (% of peak), 1 GPU"

# bytes the lookup must touch per examined block with one probe: 64 B of the
# request's tokens, a 16 B index slot, 64 B of stored tokens, 4 B parent, 4 B id out
LOOKUP_BYTES_PER_BLOCK = 152
# a write this large leaves none of a small pool in the 256 MB Infinity Cache
FLUSH_BYTES = 1 << 30


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default: 100 for the llama8b fused load, about 2.5 s of "
                         "copies, 20 for the other workloads)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="llama8b",
                    choices=["llama8b", "tiny", "llama70b_shard", "trie", "stream", "stream_evict",
                             "llama70b_full", "hybrid8b"])
    ap.add_argument("--cpu-sample", type=int, default=-1,
                    help="requests the CPU oracle is timed on (0: skip; -1: the whole batch, "
                         "8 requests for the 70B-shaped shard)")
    ap.add_argument("--copy-shape", default="",
                    help="chunks_per_group,threads[,grid] of the copy kernels")
    ap.add_argument("--seed", type=int, default=1234)
    ap.add_argument("--per-layer", action="store_true",
                    help="passage configs: gather one layer per call (a pipelined load)")
    ap.add_argument("--tier-schedule", default="streams", choices=["streams", "serial"],
                    help="llama70b_full: 'streams' looks all requests up, then loads those read "
                         "from the host tier on one stream and the rest on another (two caches); "
                         "'serial' runs one lookup+gather per request on one stream")
    args = ap.parse_args()
    if args.steps is None:
        args.steps = 100 if args.config == "llama8b" and not args.per_layer else 20
    return args


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def recorded_traffic(config: str, bytes_per_launch: float):
    """HBM bytes per gather launch from the committed rocprofv3 counter record
    (its measured traffic over algorithmic bytes, times this run's
    algorithmic bytes per launch), or None if there is none for this workload
    or the copy kernel changed since."""
    from paper_2607_22648_amd.profile_summary import copy_source_sha
    path = os.path.join(ROOT, "profiles", f"gather_{config}_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("copy_code_sha256") != copy_source_sha():
        return None
    return int(round(rec["traffic_over_algorithmic"] * bytes_per_launch))


def prefill(store, w, dev, torch, batch_passages: int):
    """Insert the stored passages and scatter random KV for their blocks."""
    from paper_2607_22648_amd import ptstore as P
    sh = w.shape
    st_toks, st_offs = w.store_batch()
    nb = w.passage_blocks
    Rs = len(st_offs) - 1
    g = torch.Generator(device=dev)
    bytes_sc = 0
    cache = None
    for lo in range(0, Rs, batch_passages):
        hi = min(Rs, lo + batch_passages)
        R = hi - lo
        toks = torch.from_numpy(st_toks[st_offs[lo]:st_offs[hi]]).to(dev)
        offs = torch.from_numpy((st_offs[lo:hi + 1] - st_offs[lo]).astype(np.int64)).to(dev)
        n_cache = R * nb * sh.block_bytes
        if cache is None or cache.numel() != n_cache:
            cache = torch.empty(n_cache, dtype=torch.uint8, device=dev)
        g.manual_seed(1000 + lo)
        cache.random_(0, 256, generator=g)
        bt = torch.arange(R * nb, dtype=torch.int32, device=dev).view(R, nb)
        m, ids, created = store.insert(toks, offs, nb)
        store.scatter(ids, created, bt, cache)
        bytes_sc += int(created.sum().item()) * 2 * sh.block_bytes
    torch.cuda.synchronize()
    t_ins, n_ins = store.kernel_times(P.KIND_INSERT)
    t_sc, n_sc = store.kernel_times(P.KIND_SCATTER)
    del cache
    torch.cuda.empty_cache()
    return {"insert_ms": round(t_ins, 3), "insert_calls": n_ins, "scatter_ms": round(t_sc, 3),
            "scatter_GBps": round(bytes_sc / (t_sc * 1e6), 1) if t_sc else None,
            "blocks": int(store.stats()["blocks_stored"])}


def cpu_baseline(w, sample: int):
    """Time the CPU oracle (1 thread) on the first `sample` requests, sub-batched as on the GPU."""
    from oracle import OracleStore
    from workloads.synth import concat_requests
    sh = w.shape
    sample = min(sample, w.n_requests)
    # the oracle store holds the stored passages these requests reference
    used = set(int(x) for x in w.req_passage[:sample])
    need = [p for p in w.stored if int(p) in used]
    o = OracleStore.for_shape(sh, capacity=max(1, len(need) * w.passage_blocks))
    if need:
        st, so = concat_requests([w.passages[p] for p in need])
        o.insert(st, so, w.passage_blocks)
        o.pool()[:] = 0x5A  # resident payload (its content does not change the work)
    maxb = w.max_blocks
    subs = [(lo, min(hi, sample)) for lo, hi in w.sub_batches() if lo < sample]
    max_R = max(hi - lo for lo, hi in subs)
    cache_blocks = max_R * maxb
    cache = np.empty(cache_blocks * sh.block_bytes, dtype=np.uint8)
    cache[:] = 0xA5
    inputs = []
    for lo, hi in subs:
        toks, offs = w.request_slice(lo, hi)
        R = hi - lo
        inputs.append((toks, offs, np.arange(R * maxb, dtype=np.int32).reshape(R, maxb)))
    moved = 0
    dt = 0.0
    passes = 0
    # whole passes over the sample until about CPU_TARGET_S of oracle time
    while passes == 0 or (dt < CPU_TARGET_S and dt * (passes + 1) / passes <= CPU_CAP_S):
        for toks, offs, bt in inputs:
            t0 = time.perf_counter()
            m, ids = o.lookup(toks, offs, maxb)
            o.gather(ids, m, bt, cache, cache_blocks)
            dt += time.perf_counter() - t0
            moved += int(m.sum()) * 2 * sh.block_bytes
        passes += 1
    o.close()
    what = "all" if sample == w.n_requests else f"the first {sample} of"
    return {"value": round(sample * passes / dt, 3), "unit": "requests/s", "cores": 1,
            "kind": "oracle",
            "sample": f"{what} {w.n_requests} requests in sub-batches of {w.sub_batch}, "
                      f"{passes} pass(es) ({moved / 1e9:.1f} GB moved); the oracle store holds "
                      f"the {len(need)} stored passages they reference",
            "seconds": round(dt, 3), "GBps": round(moved / dt / 1e9, 2),
            "host_cpus": os.cpu_count(), "cpu_model": cpu_model()}


CPU_TARGET_S = 10.0  # oracle time the CPU baseline aims for
CPU_CAP_S = 30.0

SLOW_ALLOC_S = 1.0   # a settled device allocates the pool in well under 0.1 s
SETTLE_PAUSE_S = 15.0

# Placement note (measured on MI355X): a pool allocated while the driver is
# still reclaiming a large allocation another process just freed takes 2-3 s
# to allocate and keeps a slower physical placement for its whole lifetime
# (about 6% less gather bandwidth, three times the DRAM credit stalls);
# allocated 10 s or more later it takes 0.08 s and runs at full speed. A
# serving store allocates its pool once, long before it serves, so the bench
# measures that state: if the first allocation was slow, it frees the store,
# pauses, and allocates again, and reports both allocation times.
SETTLE = {}


COPY_SHAPE = ""  # --copy-shape, applied to every store the bench creates


def make_store(P, *args, **kw):
    t0 = time.perf_counter()
    store = P.PrefixStore(*args, **kw)
    first = time.perf_counter() - t0
    SETTLE.update({"first_alloc_s": round(first, 3), "reallocated": False})
    if first > SLOW_ALLOC_S:
        log(f"pool allocation took {first:.2f}s: the device is still reclaiming memory a previous "
            f"process freed; re-allocating after {SETTLE_PAUSE_S:.0f}s")
        store.close()
        time.sleep(SETTLE_PAUSE_S)
        t0 = time.perf_counter()
        store = P.PrefixStore(*args, **kw)
        SETTLE.update({"reallocated": True, "second_alloc_s": round(time.perf_counter() - t0, 3)})
    if COPY_SHAPE:
        store.set_copy_shape(*(int(x) for x in COPY_SHAPE.split(",")))
    return store


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def hbm_ceiling(torch, P, src, dst, nbytes: int) -> dict:
    """Practical HBM ceiling measured in this run on the very buffers the
    gather uses (its pool as the source, its paged cache as the destination),
    so that it sees the same physical placement: read-only, write-only and
    copy streams with the copy kernels' access pattern (16-byte non-temporal
    vectors), plus torch's device-to-device copy of the same bytes."""
    a, b = src.view(-1)[:nbytes], dst.view(-1)[:nbytes]
    out = {"bytes": nbytes}
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for name, kind, moved in (("read", 0, nbytes), ("write", 1, nbytes), ("copy", 2, 2 * nbytes)):
        P.ptstore_bandwidth_probe(kind, a, b, nbytes)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(5):
            P.ptstore_bandwidth_probe(kind, a, b, nbytes)
        e1.record()
        torch.cuda.synchronize()
        out[f"{name}_GBps"] = round(moved * 5 / (e0.elapsed_time(e1) * 1e6), 1)
    b.copy_(a)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(5):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    out["torch_d2d_GBps"] = round(2 * nbytes * 5 / (e0.elapsed_time(e1) * 1e6), 1)
    return out


def base_line(args, value, unit, ms_per_step, config):
    return {"metric": METRIC, "value": round(value, 2), "unit": unit, "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 3),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u8",
            "data": "synthetic", "config": config}


def gather_rows(torch, ids, m):
    """(distinct stored blocks, matched blocks) of one gather call. The copy
    reads each distinct stored block once and writes it to every cache block
    that needs it: (distinct + matched) blocks are its algorithmic bytes."""
    sel = torch.arange(ids.shape[1], device=ids.device)[None, :] < m[:, None]
    rows = ids[sel]
    return int(torch.unique(rows).numel()), int(rows.numel())


def roofline(kernel, bytes_per_launch, avg_ms, launches, traffic, ceiling=None):
    achieved = bytes_per_launch / (avg_ms * 1e6)
    out = {"bound": "hbm", "kernel": kernel, "achieved": round(achieved, 1),
           "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
           "traffic": traffic, "avg_launch_ms": round(avg_ms, 4), "launches": launches,
           "bytes_per_launch": int(bytes_per_launch)}
    if ceiling:
        # the practical ceiling on the same buffers: the faster of a pure read
        # and a pure write stream
        c = max(ceiling["read_GBps"], ceiling["write_GBps"])
        out["frac_of_measured_stream_ceiling"] = round(achieved / c, 4)
    return out


WORKLOAD_TEXT = {
    "tiny": "tiny fp16 KV (2 x 8 x 128), 64 req x 1024 tok (768-tok Zipf-1.0 passage of 32 + 256 "
            "fresh), store = top-16 passages",
    "llama8b": "llama8b-shaped KV, 256 req x 4096 tok (3584-tok Zipf-1.1 passage of 512 + 512 "
               "fresh), store = top-256 passages",
    "llama70b_shard": "llama70b-shaped KV (80 x 8 x 128 bf16), 64 req x 32768 tok (30720-tok "
                      "Zipf-1.2 passage of 64 + 2048 fresh), one GPU's shard = odd ranks 1..31 "
                      "(16 passages)",
    "llama70b_full": "llama70b-shaped KV, all 32 stored passages (322 GB) on one GPU: 48,640 "
                     "blocks in HBM + 1,920 HBM replica slots + 12,800 blocks in pinned host "
                     "memory (stored in a seeded random order); 64 req x 32768 tok, 1 per call",
    "hybrid8b": "hybrid 32-layer KV (layers alternate 8 and 2 KV heads of 128, bf16: 32 KiB and "
                "8 KiB slabs, 1.25 MiB blocks), 256 req x 4096 tok (3584-tok Zipf-1.1 passage of "
                "512 + 512 fresh), store = top-256 passages",
    "trie": "divergent trie, 8192 walks of a 64-level tree (4 children at p=0.1), 1M stored "
            "blocks, 1 x 8 x 128 fp16 KV",
    "stream": "llama8b-shaped store, rounds of 128 lookups+gathers and 128 dedup inserts + "
              "scatter, 160 GB pool",
    "stream_evict": "llama8b-shaped store, rounds of 128 lookups+gathers and 128 dedup inserts "
                    "of 512-token questions + scatter, 160 GB pool with frequency-based leaf "
                    "eviction",
}


def run_passage(args, torch, P, synth, dev):
    w = synth.build(args.config, seed=args.seed)
    log(f"workload {args.config}: {w.n_requests} requests, max_blocks {w.max_blocks}, "
        f"{len(w.stored)} stored passages")
    sh = w.shape
    shape = P.StoreShape(sh.layers, sh.kv_heads, sh.head_dim, sh.block_tokens, sh.elem_bytes,
                         sh.layer_chunk_bytes)
    pool_blocks = len(w.stored) * w.passage_blocks
    store = make_store(P, shape, pool_blocks, flags=P.PTSTORE_FLAG_TIMING)
    # one paged cache shared by the sub-batches, allocated before the
    # prefill's temporary caches: allocated after them (right after their
    # free) its gathers ran 13 % slower on hybrid8b, and on llama8b 9 %
    # slower when another process had just freed a large allocation
    subs = w.sub_batches()
    maxb = w.max_blocks
    max_R = max(hi - lo for lo, hi in subs)
    cache = torch.full((max_R * maxb * sh.block_bytes,), 0xA5, dtype=torch.uint8, device=dev)
    t0 = time.time()
    batch = max(1, (16 << 30) // (w.passage_blocks * sh.block_bytes))
    pre = prefill(store, w, dev, torch, batch_passages=min(64, batch))
    log(f"prefill: {pre} ({time.time() - t0:.1f}s)")

    # requests resident in HBM
    sub_inputs = []
    for lo, hi in subs:
        toks, offs = w.request_slice(lo, hi)
        R = hi - lo
        sub_inputs.append(dict(
            R=R,
            toks=torch.from_numpy(toks).to(dev),
            offs=torch.from_numpy(offs).to(dev),
            bt=torch.arange(R * maxb, dtype=torch.int32, device=dev).view(R, maxb),
            m=torch.empty(R, dtype=torch.int32, device=dev),
            ids=torch.empty((R, maxb), dtype=torch.int32, device=dev)))
    log(f"cache {cache.numel() / 1e9:.1f} GB, {len(subs)} sub-batches")

    def step():
        for s in sub_inputs:
            if args.per_layer:  # a pipelined load: the block list once, one copy per layer
                store.lookup(s["toks"], s["offs"], maxb, m=s["m"], ids=s["ids"])
                store.gather_prepare(s["ids"], s["m"], s["bt"], cache)
                for l in range(sh.layers):
                    store.gather_prepared(cache, (l, l + 1))
            else:
                store.lookup_gather(s["toks"], s["offs"], maxb, s["bt"], cache, m=s["m"],
                                    ids=s["ids"])

    # in the timed steps the library records events around its copy kernel
    # alone: events around the lookup and the list build too would add
    # microseconds to every call (a fifth of a step at the tiny shape); the
    # lookups are timed in a pass of their own afterwards
    store.set_timing_kinds(1 << P.KIND_GATHER)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    store.kernel_times(P.KIND_GATHER)
    rows = [gather_rows(torch, s["ids"], s["m"]) for s in sub_inputs]
    distinct = sum(d for d, _ in rows)
    matched = sum(n for _, n in rows)
    blocks_examined = sum(int(np.minimum(np.diff(w.request_slice(lo, hi)[1]) // sh.block_tokens,
                                         maxb).sum()) for lo, hi in subs)

    torch.cuda.synchronize()
    # per-step HIP events on the stream the store's kernels run on (torch's
    # current stream), for the median; the K steps are timed as a whole too
    cur = torch.cuda.current_stream()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    evs[0].record(cur)
    for k in range(args.steps):
        step()
        evs[k + 1].record(cur)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    per_step = sorted(evs[k].elapsed_time(evs[k + 1]) for k in range(args.steps))
    g_ms, g_n = store.kernel_times(P.KIND_GATHER)
    # the lookups of the same sub-batches back to back, the library's events
    # off, one event pair around them (an event pair around each short
    # launch would add its launch latency)
    store.set_timing_kinds(0)
    lk_reps = min(args.steps, 10)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(cur)
    for _ in range(lk_reps):
        for s in sub_inputs:
            store.lookup(s["toks"], s["offs"], maxb, m=s["m"], ids=s["ids"])
    ev1.record(cur)
    torch.cuda.synchronize()
    lookup_ms = ev0.elapsed_time(ev1) / (lk_reps * len(sub_inputs))
    store.set_timing_kinds(1 << P.KIND_GATHER)

    ms_per_step = elapsed * 1e3 / args.steps
    gather_bytes_step = (distinct + matched) * sh.block_bytes
    lookup_bytes_step = blocks_examined * LOOKUP_BYTES_PER_BLOCK
    step_GBps = (gather_bytes_step + lookup_bytes_step) / (ms_per_step * 1e6)
    st = store.stats()
    flushed = None
    if st["blocks_stored"] * sh.block_bytes <= FLUSH_BYTES // 2:
        # a pool this small stays in the 256 MB Infinity Cache between steps;
        # gathers that follow a 1 GiB write read it from HBM instead
        flush = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=dev)
        store.kernel_times(P.KIND_GATHER)
        for k in range(args.steps):
            flush.fill_(k & 0xFF)
            step()
        torch.cuda.synchronize()
        f_ms, f_n = store.kernel_times(P.KIND_GATHER)
        f_gbps = gather_bytes_step * args.steps / (f_ms * 1e6)
        flushed = {"gather_GBps": round(f_gbps, 1), "frac": round(f_gbps / HBM_PEAK_GBPS, 4),
                   "avg_launch_ms": round(f_ms / max(f_n, 1), 4), "launches": f_n,
                   "flush": f"{FLUSH_BYTES >> 30} GiB written before each step"}
        del flush
    nb = min(cache.numel(), st["blocks_stored"] * sh.block_bytes, 16 << 30) // 16 * 16
    ceiling = hbm_ceiling(torch, P, store.pool_tensor(), cache, nb)
    del cache
    store.close()
    torch.cuda.empty_cache()
    cpu = None
    if args.cpu_sample:
        n = args.cpu_sample if args.cpu_sample > 0 else (8 if sh.layers > 32 else w.n_requests)
        log("timing the CPU oracle ...")
        cpu = cpu_baseline(w, n)
        log(f"cpu baseline: {cpu}")
    out = base_line(args, w.n_requests * args.steps / elapsed, "requests/s", ms_per_step, {
        "workload": WORKLOAD_TEXT[args.config],
        "layers": sh.layers, "kv_heads": sh.kv_heads, "head_dim": sh.head_dim,
        "block_tokens": sh.block_tokens, "kv_dtype": sh.dtype,
        "requests": w.n_requests, "sub_batches": len(subs), "sub_batch": w.sub_batch,
        "stored_blocks": st["blocks_stored"], "block_bytes": sh.block_bytes,
        "gather_calls": "block list once, one copy per layer" if args.per_layer
        else "one per sub-batch"})
    out.update({
        "ms_per_step_median": round(per_step[len(per_step) // 2], 3),
        "ms_per_step_min_max": [round(per_step[0], 3), round(per_step[-1], 3)],
        "hbm_GBps": round(step_GBps, 1),
        "hbm_frac": round(step_GBps / HBM_PEAK_GBPS, 4),
        "matched_blocks_per_step": matched,
        "distinct_blocks_per_step": distinct,
        "roofline": roofline("k_copy_slices (gather)" if not sh.layer_chunk_bytes
                             else "k_copy_spans<true> (gather)",
                             gather_bytes_step * args.steps / max(g_n, 1),
                             g_ms / max(g_n, 1), g_n,
                             None if args.per_layer else
                             recorded_traffic(args.config, gather_bytes_step * args.steps / max(g_n, 1)),
                             ceiling),
        "lookup_ms_per_call": round(lookup_ms, 4),
        "gather_after_cache_flush": flushed,
        # every gather dispatch of this process (warm-up, timed and flushed
        # steps, each step the same blocks), for the rocprofv3 traffic record
        "gather_all": None if args.per_layer else {
            "dispatches": (args.warmup + args.steps + (args.steps if flushed else 0)) * len(subs),
            "bytes": (args.warmup + args.steps + (args.steps if flushed else 0)) * gather_bytes_step,
            "read_bytes": (args.warmup + args.steps + (args.steps if flushed else 0)) * distinct
            * sh.block_bytes},
        "hbm_ceiling": ceiling,
        "prefill": pre,
        "cpu_baseline": cpu,
    })
    return out


def host_link_ceiling(torch, P, host_ptr: int, sink: torch.Tensor, nbytes: int) -> dict:
    """Read-only stream over the host tier with the copy kernels' access
    pattern: the practical host-link rate the tier's gathers can reach."""
    st = torch.cuda.current_stream()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    best = 0.0
    for _ in range(3):
        a.record(st)
        P.ptstore_bandwidth_probe(0, host_ptr, sink, nbytes, st)
        b.record(st)
        b.synchronize()
        best = max(best, nbytes / (a.elapsed_time(b) * 1e6))
    return {"read_GBps": round(best, 1), "bytes": nbytes}


def run_tiered(args, torch, P, synth, dev):
    """All of a too-large store on one GPU: device tier, replica slots, host tier.
    Steps are timed before and after one ptstore_replicate."""
    w = synth.build(args.config, seed=args.seed)
    sh = w.shape
    tiers = w.tiers
    owned, R_rep, H_blocks = tiers["device_blocks"], tiers["replica_blocks"], tiers["host_blocks"]
    shape = P.StoreShape(sh.layers, sh.kv_heads, sh.head_dim, sh.block_tokens, sh.elem_bytes,
                         sh.layer_chunk_bytes)
    t0 = time.time()
    log(f"allocating {(owned + R_rep) * sh.block_bytes / 2**30:.0f} GiB device + "
        f"{H_blocks * sh.block_bytes / 2**30:.0f} GiB pinned host ...")
    store = make_store(P, shape, owned + R_rep, host_blocks=H_blocks, replica_blocks=R_rep,
                          flags=P.PTSTORE_FLAG_TIMING | P.PTSTORE_FLAG_EVICT)
    log(f"store: {owned} device + {R_rep} replica rows, {H_blocks} host blocks "
        f"({time.time() - t0:.1f}s to allocate)")
    t0 = time.time()
    pre = prefill(store, w, dev, torch, batch_passages=1)
    log(f"prefill: {pre} ({time.time() - t0:.1f}s)")
    subs = w.sub_batches()
    maxb = w.max_blocks
    sub_inputs = []
    for lo, hi in subs:
        toks, offs = w.request_slice(lo, hi)
        R = hi - lo
        sub_inputs.append(dict(
            R=R, toks=torch.from_numpy(toks).to(dev), offs=torch.from_numpy(offs).to(dev),
            bt=torch.arange(R * maxb, dtype=torch.int32, device=dev).view(R, maxb),
            m=torch.empty(R, dtype=torch.int32, device=dev),
            ids=torch.empty((R, maxb), dtype=torch.int32, device=dev)))
    max_R = max(s["R"] for s in sub_inputs)
    cache = torch.full((sh.layers * 2 * max_R * maxb * sh.chunk_bytes,), 0xA5, dtype=torch.uint8,
                       device=dev)
    host_ptr = store.buffers().host_pool
    link = host_link_ceiling(torch, P, host_ptr, cache, min(16 << 30, H_blocks * sh.block_bytes))
    log(f"host link: {link}")
    streams = args.tier_schedule == "streams"
    if streams:
        # all requests in one lookup; then loads of requests that read the host
        # tier on one stream, of the others on a second stream, each into a
        # cache of its own, so the host-link copies and the HBM copies overlap
        toks_all, offs_all = w.request_slice(0, w.n_requests)
        R_all = w.n_requests
        look = dict(toks=torch.from_numpy(toks_all).to(dev), offs=torch.from_numpy(offs_all).to(dev),
                    m=torch.empty(R_all, dtype=torch.int32, device=dev),
                    ids=torch.empty((R_all, maxb), dtype=torch.int32, device=dev))
        cache_h = torch.full_like(cache, 0xA5)
        s_host, s_dev = torch.cuda.Stream(), torch.cuda.Stream()
        bt1 = torch.arange(maxb, dtype=torch.int32, device=dev).view(1, maxb)
        rep_map = [None]  # host-tier block -> replica slot, read after each replicate
        host_span = []

    def route():
        """Requests that read at least one block from the host tier, and the rest."""
        m = look["m"].cpu().numpy()
        ids = look["ids"].cpu().numpy()
        rep = rep_map[0]
        on_host = []
        for r in range(len(m)):
            row = ids[r, :m[r]]
            hr = row[row >= owned] - owned
            on_host.append(bool(len(hr)) and bool((rep[hr] < 0).any()))
        return [r for r in range(len(m)) if on_host[r]], [r for r in range(len(m)) if not on_host[r]]

    def step():
        if not streams:
            for s in sub_inputs:
                store.lookup_gather(s["toks"], s["offs"], maxb, s["bt"], cache, m=s["m"], ids=s["ids"])
            return
        main = torch.cuda.current_stream()
        store.lookup(look["toks"], look["offs"], maxb, m=look["m"], ids=look["ids"])
        host_r, dev_r = route()  # waits for the lookup (a 0.5 MB read back)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        s_host.wait_stream(main)  # both wait for the lookup, then run side by side
        s_dev.wait_stream(main)
        e0.record(s_host)
        for st_, reqs, c in ((s_host, host_r, cache_h), (s_dev, dev_r, cache)):
            for r in reqs:
                store.gather(look["ids"][r:r + 1], look["m"][r:r + 1], bt1, c, stream=st_)
        e1.record(s_host)
        main.wait_stream(s_host)
        main.wait_stream(s_dev)
        host_span.append((e0, e1))

    def where_blocks():
        """(device-resident, host-resident) gathered blocks per step."""
        rep = store.replica_map().cpu().numpy()
        dev_n = host_n = 0
        for s in ([look] if streams else sub_inputs):
            m = s["m"].cpu().numpy()
            ids = s["ids"].cpu().numpy()
            for r in range(len(m)):
                row = ids[r, :m[r]]
                hr = row[row >= owned] - owned
                on_host = int((rep[hr] < 0).sum())
                host_n += on_host
                dev_n += len(row) - on_host
        return dev_n, host_n

    def phase(n_steps, n_warm):
        if streams:
            rep_map[0] = store.replica_map().cpu().numpy()
        for _ in range(n_warm):
            step()
        torch.cuda.synchronize()
        store.kernel_times(P.KIND_GATHER)
        store.kernel_times(P.KIND_LOOKUP)
        if streams:
            host_span.clear()
        t = time.perf_counter()
        for _ in range(n_steps):
            step()
        torch.cuda.synchronize()
        el = time.perf_counter() - t
        g_ms, g_n = store.kernel_times(P.KIND_GATHER)
        d_n, h_n = where_blocks()
        host_bytes = h_n * sh.block_bytes  # read over the host link per step
        # time the host link carries them: the host stream's span with two
        # streams, else the sum of the gather kernels (all host-bound but a
        # small HBM share)
        h_ms = (sum(a.elapsed_time(b) for a, b in host_span) / n_steps if streams
                else g_ms / n_steps)
        out = {"requests_per_s": round(w.n_requests * n_steps / el, 2),
               "ms_per_step": round(el * 1e3 / n_steps, 2),
               "gather_kernel_ms_per_step": round(g_ms / n_steps, 2),
               "blocks_from_device": d_n, "blocks_from_host": h_n,
               "host_GB_per_step": round(host_bytes / 1e9, 2),
               "host_link_GBps": round(host_bytes / (h_ms * 1e6), 1) if h_ms else None,
               "gather_launches": g_n, "_elapsed": el, "_g_ms": g_ms, "_matched": d_n + h_n}
        if streams:
            out["host_stream_ms_per_step"] = round(h_ms, 2)
            out["schedule"] = ("lookup of all requests, then loads reading the host tier on one "
                               "stream and the others on a second, two caches")
        return out

    steps = max(1, min(args.steps, 4))
    a = phase(steps, args.warmup)
    log(f"without replicas: {a}")
    store.kernel_times(P.KIND_REPLICATE)
    store.replicate()
    torch.cuda.synchronize()
    r_ms, _ = store.kernel_times(P.KIND_REPLICATE)
    st = store.stats()
    rep = {"replicate_ms": round(r_ms, 2), "blocks_copied": st["replica_copies"],
           "GBps": round(st["replica_copies"] * sh.block_bytes / (r_ms * 1e6), 1) if r_ms else None}
    log(f"replicate: {rep}")
    b = phase(steps, 0)
    log(f"with replicas: {b}")
    del cache
    if streams:
        del cache_h
    store.close()
    torch.cuda.empty_cache()
    # one request per gather call, and a request's blocks are distinct: each
    # matched block is read once and written once
    gather_bytes_step = b["_matched"] * 2 * sh.block_bytes
    out = base_line(args, w.n_requests * steps / b["_elapsed"], "requests/s",
                    b["_elapsed"] * 1e3 / steps, {
        "workload": WORKLOAD_TEXT[args.config],
        "layers": sh.layers, "kv_heads": sh.kv_heads, "head_dim": sh.head_dim,
        "block_tokens": sh.block_tokens, "kv_dtype": sh.dtype, "requests": w.n_requests,
        "sub_batch": w.sub_batch, "schedule": args.tier_schedule,
        "device_blocks": owned, "replica_blocks": R_rep,
        "host_blocks": H_blocks, "block_bytes": sh.block_bytes})
    out["steps"] = steps
    clean = lambda d: {k: v for k, v in d.items() if not k.startswith("_")}
    hl = b["host_link_GBps"]
    out.update({
        # the path is bound by the host link: the copy kernel's reads of
        # host-tier rows, their bytes per step over the time the link carries
        # them, against the link's published peak
        "roofline": {"bound": "host link", "kernel": "k_copy_slices (gather, host-tier rows)",
                     "achieved": hl, "peak": HOST_LINK_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(hl / HOST_LINK_PEAK_GBPS, 4) if hl else None, "traffic": None,
                     "bytes_per_step": b["host_GB_per_step"] * 1e9,
                     "frac_of_measured_link_ceiling": round(hl / link["read_GBps"], 4) if hl else None},
        # every gather launch of a step (host-tier and device rows) against HBM
        "gather_all_launches": roofline("k_copy_slices (gather)", gather_bytes_step / len(subs),
                                        b["_g_ms"] / max(b["gather_launches"], 1),
                                        b["gather_launches"], None),
        "host_link": {"achieved": hl, "ceiling": link["read_GBps"],
                      "frac_of_ceiling": round(hl / link["read_GBps"], 4) if hl else None,
                      "unit": "GB/s",
                      "spec": "PCIe 5.0 x16, 64 GB/s per direction"},
        "with_replicas": clean(b), "without_replicas": clean(a), "replicate": rep,
        "host_link_ceiling": link, "prefill": pre, "cpu_baseline": None,
    })
    return out


def run_trie(args, torch, P, synth, dev):
    t0 = time.time()
    w = synth.build("trie", seed=args.seed)
    log(f"trie workload: {len(w.store_offsets) - 1} store walks, {w.n_requests} requests "
        f"({time.time() - t0:.1f}s)")
    sh = w.shape
    shape = P.StoreShape(sh.layers, sh.kv_heads, sh.head_dim, sh.block_tokens, sh.elem_bytes,
                         sh.layer_chunk_bytes)
    store = make_store(P, shape, w.capacity, flags=P.PTSTORE_FLAG_TIMING | P.PTSTORE_FLAG_COUNTERS)
    W = len(w.store_offsets) - 1
    g = torch.Generator(device=dev)
    created_total = 0
    for lo in range(0, W, 32768):
        hi = min(W, lo + 32768)
        toks = torch.from_numpy(w.store_tokens[w.store_offsets[lo]:w.store_offsets[hi]]).to(dev)
        offs = torch.from_numpy((w.store_offsets[lo:hi + 1] - w.store_offsets[lo])
                                .astype(np.int64)).to(dev)
        m, ids, cr = store.insert(toks, offs, w.depth)
        flat = cr.view(-1).to(torch.int64)
        n_new = int(flat.sum().item())
        created_total += n_new
        if n_new == 0:
            continue
        bt = torch.where(flat != 0, torch.cumsum(flat, 0) - 1, -1).to(torch.int32).view_as(cr)
        cache = torch.empty(sh.layers * 2 * n_new * sh.chunk_bytes, dtype=torch.uint8, device=dev)
        g.manual_seed(lo)
        cache.random_(0, 256, generator=g)
        store.scatter(ids, cr, bt, cache)
        del cache
    torch.cuda.synchronize()
    ins_ms, ins_n = store.kernel_times(P.KIND_INSERT)
    sc_ms, sc_n = store.kernel_times(P.KIND_SCATTER)
    torch.cuda.empty_cache()
    R = w.n_requests
    toks = torch.from_numpy(w.tokens).to(dev)
    offs = torch.from_numpy(w.offsets).to(dev)
    m = torch.empty(R, dtype=torch.int32, device=dev)
    ids = torch.empty((R, w.depth), dtype=torch.int32, device=dev)
    bt = torch.arange(R * w.depth, dtype=torch.int32, device=dev).view(R, w.depth)
    cache = torch.full((sh.layers * 2 * R * w.depth * sh.chunk_bytes,), 0xA5, dtype=torch.uint8,
                       device=dev)
    # lookup only (the probe-bound headline of this workload), timed with the
    # event counters off. First back to back, with the library's per-launch
    # events off too and one event pair around all K calls on the stream
    # they run on (two events around every launch add microseconds to a
    # 25-microsecond kernel); then K more, each bracketed by the library's
    # own events. One more lookup with the counters on counts its probes.
    store.set_counters(False)
    store.set_timing(False)
    for _ in range(args.warmup):
        store.lookup(toks, offs, w.depth, m=m, ids=ids)
    torch.cuda.synchronize()
    store.kernel_times(P.KIND_LOOKUP)
    cur = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(cur)
    for _ in range(args.steps):
        store.lookup(toks, offs, w.depth, m=m, ids=ids)
    ev1.record(cur)
    torch.cuda.synchronize()
    lk_elapsed = time.perf_counter() - t0
    lk_stream = ev0.elapsed_time(ev1) / args.steps
    store.set_timing(True)
    for _ in range(args.steps):
        store.lookup(toks, offs, w.depth, m=m, ids=ids)
    torch.cuda.synchronize()
    lk_ms, lk_n = store.kernel_times(P.KIND_LOOKUP)
    store.set_counters(True)
    store.reset_counters()
    store.lookup(toks, offs, w.depth, m=m, ids=ids)
    stt = store.stats()
    probes = stt["probes"]
    compares = stt["token_compares"]
    store.kernel_times(P.KIND_LOOKUP)
    store.set_counters(False)
    distinct, matched = gather_rows(torch, ids, m)
    trie_bytes = (distinct + matched) * sh.block_bytes
    # fused lookup + gather, with events around the copy kernel alone
    store.set_timing_kinds(1 << P.KIND_GATHER)
    for _ in range(args.warmup):
        store.lookup_gather(toks, offs, w.depth, bt, cache, m=m, ids=ids)
    torch.cuda.synchronize()
    store.kernel_times(P.KIND_GATHER)
    store.kernel_times(P.KIND_LOOKUP)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        store.lookup_gather(toks, offs, w.depth, bt, cache, m=m, ids=ids)
    torch.cuda.synchronize()
    fu_elapsed = time.perf_counter() - t0
    g_ms, g_n = store.kernel_times(P.KIND_GATHER)
    nb = min(cache.numel(), int(stt["blocks_stored"]) * sh.block_bytes, 16 << 30) // 16 * 16
    ceiling = hbm_ceiling(torch, P, store.pool_tensor(), cache, nb)
    store.close()
    del cache
    torch.cuda.empty_cache()
    cpu = None
    if args.cpu_sample:
        from oracle import OracleStore
        o = OracleStore.for_shape(sh, w.capacity, with_payload=False)
        o.insert(w.store_tokens, w.store_offsets, w.depth)
        reps, t_cpu = 0, 0.0
        while t_cpu < CPU_TARGET_S:
            t1 = time.perf_counter()
            o.lookup(w.tokens, w.offsets, w.depth)
            t_cpu += time.perf_counter() - t1
            reps += 1
        o.close()
        cpu = {"value": round(R * reps / t_cpu, 1), "unit": "lookups/s", "cores": 1,
               "kind": "oracle", "sample": f"lookup only (pointer trie, no payload) of all {R} "
                                           f"walks, {reps} repetitions", "seconds": round(t_cpu, 3)}
    lk_avg = lk_ms / max(lk_n, 1)
    out = base_line(args, R * args.steps / fu_elapsed, "requests/s", fu_elapsed * 1e3 / args.steps, {
        "workload": WORKLOAD_TEXT["trie"], "requests": R, "depth": w.depth,
        "stored_blocks": int(stt["blocks_stored"]), "block_bytes": sh.block_bytes})
    out.update({
        "lookup_only": {"lookups_per_s": round(R * args.steps / lk_elapsed, 1),
                        "stream_ms_per_call": round(lk_stream, 4),
                        "lookups_per_s_stream": round(R / (lk_stream / 1e3), 1),
                        "kernel_avg_ms": round(lk_avg, 4),
                        "lookups_per_s_kernel": round(R / (lk_avg / 1e3), 1),
                        "timing": "lookups_per_s (wall) and *_stream: K calls back to back, the "
                                  "library's per-launch events off, one event pair around them; "
                                  "kernel_*: K more calls, each between the library's own events",
                        "counters": "off in the timed lookups; probes and compares from one "
                                    "more lookup with them on",
                        "probes_per_call": int(probes), "token_compares_per_call": int(compares),
                        "probes_per_s_kernel": round(probes / (lk_avg / 1e3), 1),
                        "blocks_examined": int(R * w.depth),
                        "algorithmic_GBps": round(R * w.depth * LOOKUP_BYTES_PER_BLOCK
                                                  / (lk_avg * 1e6), 1)},
        "matched_blocks": matched, "distinct_blocks": distinct,
        "roofline": roofline("k_copy_slices (gather)", trie_bytes, g_ms / max(g_n, 1),
                             g_n, recorded_traffic("trie", trie_bytes), ceiling),
        "hbm_ceiling": ceiling,
        "gather_all": {"dispatches": args.warmup + args.steps,
                       "bytes": (args.warmup + args.steps) * trie_bytes,
                       "read_bytes": (args.warmup + args.steps) * distinct * sh.block_bytes},
        "prefill": {"insert_ms": round(ins_ms, 3), "insert_calls": ins_n,
                    "scatter_ms": round(sc_ms, 3), "blocks": created_total},
        "cpu_baseline": cpu,
    })
    return out


def run_stream(args, torch, P, synth, dev):
    sw = synth.build(args.config, seed=args.seed)
    base = sw.base
    sh = base.shape
    shape = P.StoreShape(sh.layers, sh.kv_heads, sh.head_dim, sh.block_tokens, sh.elem_bytes,
                         sh.layer_chunk_bytes)
    evict = args.config == "stream_evict"
    flags = P.PTSTORE_FLAG_TIMING | P.PTSTORE_FLAG_COUNTERS | (P.PTSTORE_FLAG_EVICT if evict else 0)
    store = make_store(P, shape, sw.pool_blocks, flags=flags)
    maxb = base.max_blocks
    per = len(sw.rounds[0].lookup_offsets) - 1
    # the paged cache before the prefill's temporary caches: allocated after
    # them (right after their free) its gathers ran 3.7 % slower
    cache = torch.full((sh.layers * 2 * per * maxb * sh.chunk_bytes,), 0xA5, dtype=torch.uint8,
                       device=dev)
    pre = prefill(store, base, dev, torch, batch_passages=32)
    bt = torch.arange(per * maxb, dtype=torch.int32, device=dev).view(per, maxb)
    m = torch.empty(per, dtype=torch.int32, device=dev)
    ids = torch.empty((per, maxb), dtype=torch.int32, device=dev)
    rounds = [(torch.from_numpy(r.lookup_tokens).to(dev), torch.from_numpy(r.lookup_offsets).to(dev),
               torch.from_numpy(r.insert_tokens).to(dev), torch.from_numpy(r.insert_offsets).to(dev))
              for r in sw.rounds]
    n_timed = min(args.steps, len(rounds) - args.warmup)

    def one_round(i):
        """The round's gather list (ids, m; kept for its distinct blocks) and
        the created flags of its insert."""
        lt, lo, it, io = rounds[i]
        store.lookup_gather(lt, lo, maxb, bt, cache, m=m, ids=ids)
        got = (ids.clone(), m.clone())
        _, iids, icr = store.insert(it, io, maxb)
        store.scatter(iids, icr, bt[:io.numel() - 1], cache)
        return got, icr

    warm = [gather_rows(torch, *one_round(i)[0]) for i in range(args.warmup)]
    torch.cuda.synchronize()
    distinct_warm = sum(d for d, _ in warm)
    matched_warm = sum(n for _, n in warm)
    for k in (P.KIND_GATHER, P.KIND_LOOKUP, P.KIND_INSERT, P.KIND_SCATTER, P.KIND_EVICT):
        store.kernel_times(k)
    blocks0 = store.stats()["blocks_stored"]
    evictions0 = store.stats()["evictions"]
    store.reset_counters()
    keep = []
    t0 = time.perf_counter()
    for i in range(args.warmup, args.warmup + n_timed):
        got, cr = one_round(i)
        keep.append((got, cr.to(torch.int64).sum()))
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    rows = [gather_rows(torch, *a) for a, _ in keep]
    distinct = sum(d for d, _ in rows)
    matched = sum(n for _, n in rows)
    created = int(sum(int(b.item()) for _, b in keep))
    kinds = [("gather", P.KIND_GATHER), ("lookup", P.KIND_LOOKUP), ("insert", P.KIND_INSERT),
             ("scatter", P.KIND_SCATTER)] + ([("evict (part of insert)", P.KIND_EVICT)] if evict else [])
    t = {k: store.kernel_times(v) for k, v in kinds}
    st = store.stats()
    nb = min(cache.numel(), st["blocks_stored"] * sh.block_bytes, 16 << 30) // 16 * 16
    ceiling = hbm_ceiling(torch, P, store.pool_tensor(), cache, nb)
    store.close()
    del cache
    torch.cuda.empty_cache()
    g_ms, g_n = t["gather"]
    g_bytes = (distinct + matched) * sh.block_bytes
    ms_round = elapsed * 1e3 / n_timed
    out = base_line(args, per * n_timed / elapsed, "requests/s", ms_round, {
        "workload": WORKLOAD_TEXT[args.config], "lookups_per_round": per, "inserts_per_round": per,
        "timed_rounds": n_timed, "pool_blocks": sw.pool_blocks, "block_bytes": sh.block_bytes})
    out["steps"] = n_timed
    out.update({
        "inserts_per_s": round(per * n_timed / elapsed, 2),
        "matched_blocks": matched, "distinct_blocks": distinct, "created_blocks": created,
        "blocks_stored": {"before": blocks0, "after": st["blocks_stored"]},
        "roofline": roofline("k_copy_slices (gather)", g_bytes / max(g_n, 1),
                             g_ms / max(g_n, 1), g_n,
                             recorded_traffic(args.config, g_bytes / max(g_n, 1)), ceiling),
        "hbm_ceiling": ceiling,
        "gather_all": {"dispatches": args.warmup + n_timed,
                       "bytes": (distinct_warm + matched_warm + distinct + matched) * sh.block_bytes,
                       "read_bytes": (distinct_warm + distinct) * sh.block_bytes},
        "evictions": st["evictions"], "index_rebuilds": st["index_rebuilds"],
        "full_events": st["full_events"],
        "library_counters": {
            "timed_rounds": n_timed,
            "evictions_per_round": round((st["evictions"] - evictions0) / n_timed, 1),
            "index_rebuilds": st["index_rebuilds"],
            "probes_per_round": round(st["probes"] / n_timed, 1),
            "token_compares_per_round": round(st["token_compares"] / n_timed, 1),
            "cas_attempts_per_round": round(st["cas_attempts"] / n_timed, 1),
            "cas_failures_per_round": round(st["cas_failures"] / n_timed, 1)},
        "kernel_ms_per_round": {k: round(v[0] / n_timed, 4) for k, v in t.items()},
        "scatter_GBps": round(created * 2 * sh.block_bytes / (t["scatter"][0] * 1e6), 1)
        if t["scatter"][0] else None,
        "prefill": pre,
        "cpu_baseline": None,
    })
    return out


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(json.dumps({"error": "the store runs on one GPU only; sharding it over several "
                                   "GPUs is a design, not code (--gpus 1)"}))
        sys.exit(2)
    global COPY_SHAPE
    COPY_SHAPE = args.copy_shape
    import torch
    from paper_2607_22648_amd import ptstore as P
    from workloads import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.config == "trie":
        out = run_trie(args, torch, P, synth, dev)
    elif args.config in ("stream", "stream_evict"):
        out = run_stream(args, torch, P, synth, dev)
    elif args.config == "llama70b_full":
        out = run_tiered(args, torch, P, synth, dev)
    else:
        out = run_passage(args, torch, P, synth, dev)
    out["pool_allocation"] = dict(SETTLE)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
