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
in HBM. ``roofline`` = the gather kernel's algorithmic bytes (pool read +
cache write of every matched block) over its average duration, measured with
HIP events the library records on the launch stream. ``cpu_baseline`` = the
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
METRIC = "prefix lookup+KV gather: requests/s and achieved HBM GB/s (% of peak), 1 GPU"

# bytes the lookup must touch per examined block with one probe: 64 B of the
# request's tokens, a 16 B index slot, 64 B of stored tokens, 4 B parent, 4 B id out
LOOKUP_BYTES_PER_BLOCK = 152


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="llama8b", choices=["llama8b", "tiny"])
    ap.add_argument("--cpu-sample", type=int, default=256,
                    help="requests of the workload the CPU oracle is timed on (0: skip)")
    ap.add_argument("--copy-shape", default="", help="chunks_per_group,threads of the copy kernels")
    ap.add_argument("--seed", type=int, default=1234)
    return ap.parse_args()


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def recorded_traffic(config: str):
    """HBM bytes per gather launch from the committed rocprofv3 counter record,
    or None if there is none for this workload or the copy kernel changed since."""
    from paper_2607_22648_amd.profile_summary import copy_source_sha
    path = os.path.join(ROOT, "profiles", f"gather_{config}_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("copy_hip_sha256") != copy_source_sha():
        return None
    return rec["traffic_bytes_per_launch"]


def prefill(store, w, dev, torch, batch_passages: int):
    """Insert the stored passages and scatter random KV for their blocks."""
    from paper_2607_22648_amd import ptstore as P
    sh = w.shape
    st_toks, st_offs = w.store_batch()
    nb = w.passage_blocks
    Rs = len(st_offs) - 1
    g = torch.Generator(device=dev)
    t_ins = t_sc = 0.0
    n_ins = n_sc = 0
    bytes_sc = 0
    ids_all = []
    cache = None
    for lo in range(0, Rs, batch_passages):
        hi = min(Rs, lo + batch_passages)
        R = hi - lo
        toks = torch.from_numpy(st_toks[st_offs[lo]:st_offs[hi]]).to(dev)
        offs = torch.from_numpy((st_offs[lo:hi + 1] - st_offs[lo]).astype(np.int64)).to(dev)
        n_cache = sh.layers * 2 * R * nb * sh.chunk_bytes
        if cache is None or cache.numel() != n_cache:
            cache = torch.empty(n_cache, dtype=torch.uint8, device=dev)
        g.manual_seed(1000 + lo)
        cache.random_(0, 256, generator=g)
        bt = torch.arange(R * nb, dtype=torch.int32, device=dev).view(R, nb)
        m, ids, created = store.insert(toks, offs, nb)
        store.scatter(ids, created, bt, cache)
        ids_all.append(ids)
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
    cache = np.empty(sh.layers * 2 * cache_blocks * sh.chunk_bytes, dtype=np.uint8)
    cache[:] = 0xA5
    moved = 0
    dt = 0.0
    for lo, hi in subs:
        toks, offs = w.request_slice(lo, hi)
        R = hi - lo
        bt = np.arange(R * maxb, dtype=np.int32).reshape(R, maxb)
        t0 = time.perf_counter()
        m, ids = o.lookup(toks, offs, maxb)
        o.gather(ids, m, bt, cache, cache_blocks)
        dt += time.perf_counter() - t0
        moved += int(m.sum()) * 2 * sh.block_bytes
    o.close()
    what = "all" if sample == w.n_requests else f"the first {sample} of"
    return {"value": round(sample / dt, 3), "unit": "requests/s", "cores": 1, "kind": "oracle",
            "sample": f"{what} {w.n_requests} requests in sub-batches of {w.sub_batch} "
                      f"({moved / 1e9:.1f} GB moved); the oracle store holds the {len(need)} "
                      f"stored passages they reference",
            "seconds": round(dt, 3), "GBps": round(moved / dt / 1e9, 2),
            "host_cpus": os.cpu_count()}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(json.dumps({"error": "this build runs on one GPU only; the multi-GPU sharding of "
                                   "the store is a design, not code (--gpus 1)"}))
        sys.exit(2)
    import torch
    from paper_2607_22648_amd import ptstore as P
    from workloads import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t0 = time.time()
    w = synth.build(args.config, seed=args.seed)
    log(f"workload {args.config}: {w.n_requests} requests, max_blocks {w.max_blocks}, "
        f"{len(w.stored)} stored passages, generated in {time.time() - t0:.1f}s")
    sh = w.shape
    shape = P.StoreShape(sh.layers, sh.kv_heads, sh.head_dim, sh.block_tokens, sh.elem_bytes)
    pool_blocks = len(w.stored) * w.passage_blocks
    store = P.PrefixStore(shape, pool_blocks, flags=P.PTSTORE_FLAG_TIMING)
    if args.copy_shape:
        cpg, thr = (int(x) for x in args.copy_shape.split(","))
        store.set_copy_shape(cpg, thr)
    t0 = time.time()
    pre = prefill(store, w, dev, torch, batch_passages=32 if sh.layers > 2 else 64)
    log(f"prefill: {pre} ({time.time() - t0:.1f}s)")

    # requests resident in HBM, one paged cache shared by the sub-batches
    subs = w.sub_batches()
    maxb = w.max_blocks
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
    max_R = max(s["R"] for s in sub_inputs)
    cache = torch.full((sh.layers * 2 * max_R * maxb * sh.chunk_bytes,), 0xA5, dtype=torch.uint8,
                       device=dev)
    log(f"cache {cache.numel() / 1e9:.1f} GB, {len(subs)} sub-batches")

    def step():
        for s in sub_inputs:
            store.lookup_gather(s["toks"], s["offs"], maxb, s["bt"], cache, m=s["m"], ids=s["ids"])

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    store.kernel_times(P.KIND_GATHER)
    store.kernel_times(P.KIND_LOOKUP)
    matched = sum(int(s["m"].sum().item()) for s in sub_inputs)
    blocks_examined = sum(int(np.minimum(np.diff(w.request_slice(lo, hi)[1]) // sh.block_tokens,
                                         maxb).sum()) for lo, hi in subs)

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    g_ms, g_n = store.kernel_times(P.KIND_GATHER)
    l_ms, l_n = store.kernel_times(P.KIND_LOOKUP)

    ms_per_step = elapsed * 1e3 / args.steps
    req_per_s = w.n_requests * args.steps / elapsed
    gather_bytes_step = matched * 2 * sh.block_bytes
    lookup_bytes_step = blocks_examined * LOOKUP_BYTES_PER_BLOCK
    step_GBps = (gather_bytes_step + lookup_bytes_step) / (ms_per_step * 1e6)
    gather_avg_ms = g_ms / max(g_n, 1)
    gather_bytes_launch = gather_bytes_step / len(subs)
    achieved = gather_bytes_launch / (gather_avg_ms * 1e6)

    # copy ceiling: a plain device-to-device copy of 8 GiB through torch
    a = torch.empty(8 << 30, dtype=torch.uint8, device=dev)
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    d2d = 2 * a.numel() * 5 / (e0.elapsed_time(e1) * 1e6)
    del a, b

    st = store.stats()
    cpu = None
    if args.cpu_sample:
        log("timing the CPU oracle ...")
        cpu = cpu_baseline(w, args.cpu_sample)
        log(f"cpu baseline: {cpu}")

    out = {
        "metric": METRIC,
        "value": round(req_per_s, 2),
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "config": {"workload": "llama8b-shaped KV, 256 req x 4096 tok (3584-tok Zipf-1.1 passage "
                               "of 512 + 512 fresh), store = top-256 passages"
                   if args.config == "llama8b" else args.config,
                   "layers": sh.layers, "kv_heads": sh.kv_heads, "head_dim": sh.head_dim,
                   "block_tokens": sh.block_tokens, "kv_dtype": sh.dtype,
                   "requests": w.n_requests, "sub_batches": len(subs), "sub_batch": w.sub_batch,
                   "stored_blocks": st["blocks_stored"], "block_bytes": sh.block_bytes},
        "hbm_GBps": round(step_GBps, 1),
        "hbm_frac": round(step_GBps / HBM_PEAK_GBPS, 4),
        "matched_blocks_per_step": matched,
        "roofline": {"bound": "hbm", "kernel": "k_copy<gather>",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": recorded_traffic(args.config),
                     "avg_launch_ms": round(gather_avg_ms, 4), "launches": g_n,
                     "bytes_per_launch": int(gather_bytes_launch)},
        "lookup_kernel_avg_ms": round(l_ms / max(l_n, 1), 4),
        "d2d_copy_GBps": round(d2d, 1),
        "prefill": pre,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    store.close()


if __name__ == "__main__":
    main()
