"""Parity at the workloads' full sizes, in the launch configuration bench.py times.

At these sizes the oracle runs without payload (its trie alone), so:
- m, ids and created are compared with the oracle for every request, exactly;
- every gathered block is compared with pool[id] on the device (a property
  that holds at any size), and every cache block the gather must not touch
  still holds the sentinel;
- pool blocks whose input bytes were recorded when they were scattered are
  compared byte for byte through the gather (sampled outputs).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import OracleStore
from workloads import synth

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


@pytest.fixture(autouse=True)
def _device_memory_released(request):
    """Each test starts from a released device: these tests use up to 260 GiB."""
    import gc
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    free, total = torch.cuda.mem_get_info()
    print(f"[{request.node.name}] device memory free {free / 2**30:.1f} of {total / 2**30:.1f} GiB "
          f"(torch reserved {torch.cuda.memory_reserved() / 2**30:.1f} GiB)", flush=True)
    yield

if torch.cuda.is_available():
    from paper_2607_22648_amd import ptstore as P
    from tests.twin import to_dev, host, DEV

SENTINEL = 0xA5


def _shape(kv):
    return P.StoreShape(kv.layers, kv.kv_heads, kv.head_dim, kv.block_tokens, kv.elem_bytes)


def _free(*objs):
    for o in objs:
        if hasattr(o, "close"):
            o.close()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


class Recorder:
    """Input bytes of sampled blocks at the moment they are scattered."""

    def __init__(self, kv, want: int, seed: int):
        self.kv, self.want = kv, want
        self.rng = np.random.default_rng(seed)
        self.bytes = {}

    def take(self, cache: torch.Tensor, nb_cache: int, ids: np.ndarray, created: np.ndarray,
             bt: np.ndarray, k: int):
        cand = np.argwhere((created != 0) & (bt >= 0))
        if len(cand) == 0 or len(self.bytes) >= self.want:
            return
        cv = cache.view(self.kv.layers, 2, nb_cache, self.kv.chunk_bytes)
        for r, b in cand[self.rng.choice(len(cand), size=min(k, len(cand)), replace=False)]:
            self.bytes[int(ids[r, b])] = host(cv[:, :, int(bt[r, b])])


def insert_scatter(store, ref, kv, toks, offs, maxb, seed, rec: Recorder = None, k=4,
                   compact=False):
    """Insert on both sides (outputs compared), scatter seeded random KV on the GPU.

    With compact=True only created blocks get a cache slot (block table -1 elsewhere)."""
    m, ids, cr = store.insert(to_dev(toks), to_dev(offs), maxb)
    rc, rm, rids, rcr = ref.insert(toks, offs, maxb)
    ids_h, cr_h = host(ids), host(cr)
    np.testing.assert_array_equal(host(m), rm)
    np.testing.assert_array_equal(ids_h, rids)
    np.testing.assert_array_equal(cr_h, rcr)
    R = len(offs) - 1
    if compact:
        flat = cr_h.reshape(-1).astype(np.int64)
        bt = np.where(flat != 0, np.cumsum(flat) - 1, -1).astype(np.int32).reshape(R, maxb)
        nb_cache = max(1, int(flat.sum()))
    else:
        bt = np.arange(R * maxb, dtype=np.int32).reshape(R, maxb)
        nb_cache = R * maxb
    cache = torch.empty(kv.layers * 2 * nb_cache * kv.chunk_bytes, dtype=torch.uint8, device=DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    cache.random_(0, 256, generator=g)
    store.scatter(ids, cr, to_dev(bt), cache)
    if rec is not None:
        rec.take(cache, nb_cache, ids_h, cr_h, bt, k)
    torch.cuda.synchronize()
    del cache
    return ids_h, cr_h


def check_gather(store, kv, cache, m_h, ids_h, bt_h, rec: Recorder = None, chunk=128):
    """Every gathered block == pool[id]; untouched blocks keep the sentinel; recorded bytes."""
    cap = store.stats()["capacity"]
    nb_cache = cache.numel() // (kv.layers * 2 * kv.chunk_bytes)
    cv = cache.view(kv.layers, 2, nb_cache, kv.chunk_bytes)
    pv = store.pool_tensor().view(cap, kv.layers, 2, kv.chunk_bytes)
    R, maxb = ids_h.shape
    hit = (np.arange(maxb)[None, :] < m_h[:, None]) & (bt_h >= 0)
    sel_ids = to_dev(ids_h[hit].astype(np.int64))
    sel_bt = to_dev(bt_h[hit].astype(np.int64))
    for s in range(0, sel_ids.numel(), chunk):
        a = cv[:, :, sel_bt[s:s + chunk]]
        b = pv[sel_ids[s:s + chunk]].permute(1, 2, 0, 3)
        assert torch.equal(a, b), f"gathered blocks {s}..{s + chunk} differ from the pool"
    untouched = np.ones(nb_cache, dtype=bool)
    untouched[bt_h[hit]] = False
    un = to_dev(np.flatnonzero(untouched))
    for s in range(0, un.numel(), chunk):
        assert bool((cv[:, :, un[s:s + chunk]] == SENTINEL).all()), "gather wrote outside its blocks"
    if rec is not None:
        seen = 0
        for (r, b) in np.argwhere(hit):
            i = int(ids_h[r, b])
            if i in rec.bytes:
                np.testing.assert_array_equal(host(cv[:, :, int(bt_h[r, b])]), rec.bytes[i])
                seen += 1
        return seen
    return 0


def lookup_gather_checked(store, ref, kv, toks, offs, maxb, cache, rec=None):
    R = len(offs) - 1
    bt_h = np.arange(R * maxb, dtype=np.int32).reshape(R, maxb)
    cache.fill_(SENTINEL)
    m, ids = store.lookup_gather(to_dev(toks), to_dev(offs), maxb, to_dev(bt_h), cache)
    rm, rids = ref.lookup(toks, offs, maxb)
    m_h, ids_h = host(m), host(ids)
    np.testing.assert_array_equal(m_h, rm)
    np.testing.assert_array_equal(ids_h, rids)
    seen = check_gather(store, kv, cache, m_h, ids_h, bt_h, rec)
    return m_h, seen


def check_access_counts(store, ref):
    """Access counts and priorities of every block equal the oracle's."""
    torch.cuda.synchronize()
    n = ref.count
    f, h = store.evict_tensors()
    exp = np.array([ref.node_stats(i)[:2] for i in range(n)], dtype=np.int64).reshape(n, 2)
    np.testing.assert_array_equal(host(f[:n]), exp[:, 0])
    np.testing.assert_array_equal(host(h[:n]), exp[:, 1])


def _passage_store(w, capacity, batch, rec, evict=False):
    kv = w.shape
    store = P.PrefixStore(_shape(kv), capacity, flags=P.PTSTORE_FLAG_EVICT if evict else 0)
    ref = OracleStore.for_shape(kv, capacity, with_payload=False, evict=evict)
    st, so = w.store_batch()
    Rs = len(so) - 1
    for lo in range(0, Rs, batch):
        hi = min(Rs, lo + batch)
        insert_scatter(store, ref, kv, st[so[lo]:so[hi]], (so[lo:hi + 1] - so[lo]).astype(np.int64),
                       w.passage_blocks, seed=lo, rec=rec, k=8)
    assert store.stats()["blocks_stored"] == ref.count == len(w.stored) * w.passage_blocks
    return store, ref


def test_llama8b_full():
    w = synth.build("llama8b")
    kv = w.shape
    rec = Recorder(kv, 64, 1)
    store, ref = _passage_store(w, len(w.stored) * w.passage_blocks, 32, rec)
    maxb = w.max_blocks
    cache = torch.empty(kv.layers * 2 * w.sub_batch * maxb * kv.chunk_bytes, dtype=torch.uint8,
                        device=DEV)
    seen = 0
    for lo, hi in w.sub_batches():
        toks, offs = w.request_slice(lo, hi)
        m_h, s = lookup_gather_checked(store, ref, kv, toks, offs, maxb, cache, rec)
        seen += s
        expect = np.where(np.isin(w.req_passage[lo:hi], w.stored), w.passage_blocks, 0)
        np.testing.assert_array_equal(m_h, expect)
    assert seen > 0
    # the per-layer load as bench.py --per-layer runs it: the block list once,
    # then one prepared copy per layer; the same bytes as the fused gather
    lo, hi = w.sub_batches()[0]
    toks, offs = w.request_slice(lo, hi)
    R = hi - lo
    bt_h = np.arange(R * maxb, dtype=np.int32).reshape(R, maxb)
    m, ids = store.lookup(to_dev(toks), to_dev(offs), maxb)
    cache.fill_(SENTINEL)
    store.gather_prepare(ids, m, to_dev(bt_h), cache)
    for l in range(kv.layers):
        store.gather_prepared(cache, (l, l + 1))
    rm, rids = ref.lookup(toks, offs, maxb)
    m_h, ids_h = host(m), host(ids)
    np.testing.assert_array_equal(m_h, rm)
    np.testing.assert_array_equal(ids_h, rids)
    assert check_gather(store, kv, cache, m_h, ids_h, bt_h, rec) > 0
    del cache
    _free(store, ref)


def test_llama70b_shard_full():
    w = synth.build("llama70b_shard")
    kv = w.shape
    rec = Recorder(kv, 32, 2)
    store, ref = _passage_store(w, len(w.stored) * w.passage_blocks, 2, rec)
    maxb = w.max_blocks
    cache = torch.empty(kv.layers * 2 * w.sub_batch * maxb * kv.chunk_bytes, dtype=torch.uint8,
                        device=DEV)
    seen = 0
    for lo, hi in w.sub_batches():
        toks, offs = w.request_slice(lo, hi)
        m_h, s = lookup_gather_checked(store, ref, kv, toks, offs, maxb, cache, rec)
        seen += s
        expect = np.where(np.isin(w.req_passage[lo:hi], w.stored), w.passage_blocks, 0)
        np.testing.assert_array_equal(m_h, expect)
    assert seen > 0
    del cache
    _free(store, ref)


def test_trie_full():
    w = synth.build("trie")
    kv = w.shape
    store = P.PrefixStore(_shape(kv), w.capacity, flags=P.PTSTORE_FLAG_COUNTERS)
    ref = OracleStore.for_shape(kv, w.capacity, with_payload=False)
    rec = Recorder(kv, 256, 3)
    W = len(w.store_offsets) - 1
    batch = 32768
    for lo in range(0, W, batch):
        hi = min(W, lo + batch)
        toks = w.store_tokens[w.store_offsets[lo]:w.store_offsets[hi]]
        offs = (w.store_offsets[lo:hi + 1] - w.store_offsets[lo]).astype(np.int64)
        insert_scatter(store, ref, kv, toks, offs, w.depth, seed=lo, rec=rec, k=16, compact=True)
    st = store.stats()
    assert st["blocks_stored"] == ref.count == w.capacity and st["full_events"] >= 1
    R = w.n_requests
    cache = torch.empty(kv.layers * 2 * R * w.depth * kv.chunk_bytes, dtype=torch.uint8, device=DEV)
    m_h, seen = lookup_gather_checked(store, ref, kv, w.tokens, w.offsets, w.depth, cache, rec)
    assert seen > 0 and m_h.mean() > 60
    del cache
    _free(store, ref)


@pytest.mark.parametrize("name,rounds", [("stream", None), ("stream_evict", 14)])
def test_stream_full(name, rounds):
    """100 rounds of the stream on the 160 GB pool; with eviction, 14 rounds (the
    pool fills in the sixth; the oracle's one-leaf-at-a-time eviction is slow)."""
    over = {} if rounds is None else {"n_rounds": rounds}
    sw = synth.build(name, **over)
    evict = name == "stream_evict"
    base = sw.base
    kv = base.shape
    rec = Recorder(kv, 64, 4)
    store, ref = _passage_store(base, sw.pool_blocks, 32, rec, evict=evict)
    maxb = base.max_blocks
    per = len(sw.rounds[0].lookup_offsets) - 1
    cache = torch.empty(kv.layers * 2 * per * maxb * kv.chunk_bytes, dtype=torch.uint8, device=DEV)
    nb_cache = per * maxb
    g = torch.Generator(device=DEV)
    seen = 0
    for i, rd in enumerate(sw.rounds):
        _, s = lookup_gather_checked(store, ref, kv, rd.lookup_tokens, rd.lookup_offsets, maxb,
                                     cache, rec)
        seen += s
        # inserts: KV of the new blocks is fresh in the cache, then scattered
        Ri = len(rd.insert_offsets) - 1
        bt_h = np.arange(Ri * maxb, dtype=np.int32).reshape(Ri, maxb)
        g.manual_seed(10_000 + i)
        cache.random_(0, 256, generator=g)
        m, ids, cr = store.insert(to_dev(rd.insert_tokens), to_dev(rd.insert_offsets), maxb)
        rc, rm, rids, rcr = ref.insert(rd.insert_tokens, rd.insert_offsets, maxb)
        ids_h, cr_h = host(ids), host(cr)
        np.testing.assert_array_equal(host(m), rm)
        np.testing.assert_array_equal(ids_h, rids)
        np.testing.assert_array_equal(cr_h, rcr)
        store.scatter(ids, cr, to_dev(bt_h), cache)
        # every created block now holds its cache block's bytes
        made = np.argwhere(cr_h != 0)
        if len(made):
            cv = cache.view(kv.layers, 2, nb_cache, kv.chunk_bytes)
            pv = store.pool_tensor().view(-1, kv.layers, 2, kv.chunk_bytes)
            sel_ids = to_dev(ids_h[cr_h != 0].astype(np.int64))
            sel_bt = to_dev(bt_h[cr_h != 0].astype(np.int64))
            assert torch.equal(cv[:, :, sel_bt], pv[sel_ids].permute(1, 2, 0, 3))
            for reused in ids_h[cr_h != 0].tolist():  # an evicted id now holds another block
                rec.bytes.pop(int(reused), None)
            rec.take(cache, nb_cache, ids_h, cr_h, bt_h, 1)
        if evict and (i % 4 == 3 or i == len(sw.rounds) - 1):
            check_access_counts(store, ref)
    assert store.stats()["blocks_stored"] == ref.count
    assert ref.count > len(base.stored) * base.passage_blocks
    assert seen > 0
    if evict:
        st = store.stats()
        assert st["evictions"] == ref.evictions > 0 and st["clock"] == ref.clock
    del cache
    _free(store, ref)


def _check_gather_tiered(store, kv, cache, m_h, ids_h, bt_h, rng, rec=None, per_row=8):
    """Sampled gathered blocks equal their home bytes (device or host tier);
    sampled unmatched blocks keep the sentinel; recorded bytes where seen."""
    nb_cache = cache.numel() // (kv.layers * 2 * kv.chunk_bytes)
    cv = cache.view(kv.layers, 2, nb_cache, kv.chunk_bytes)
    seen = 0
    for r in range(len(m_h)):
        if m_h[r]:
            bs = rng.choice(m_h[r], size=min(per_row, m_h[r]), replace=False)
            got = cv[:, :, torch.from_numpy(bt_h[r, bs].astype(np.int64)).to(DEV)].permute(2, 0, 1, 3)
            exp = store.block_bytes_of(ids_h[r, bs]).view(len(bs), kv.layers, 2, kv.chunk_bytes)
            assert torch.equal(got, exp), f"request {r}: gathered blocks differ from their home"
        rest = np.arange(m_h[r], ids_h.shape[1])
        if len(rest):
            bs = rng.choice(rest, size=min(per_row, len(rest)), replace=False)
            sel = torch.from_numpy(bt_h[r, bs].astype(np.int64)).to(DEV)
            assert bool((cv[:, :, sel] == SENTINEL).all()), "gather wrote outside its blocks"
        if rec is not None:
            for b in range(m_h[r]):
                i = int(ids_h[r, b])
                if i in rec.bytes:
                    np.testing.assert_array_equal(host(cv[:, :, int(bt_h[r, b])]), rec.bytes[i])
                    seen += 1
    return seen


def test_llama70b_full_tiered():
    """All 32 passages (322 GB) on one GPU: HBM, HBM replicas and the pinned
    host tier. Metadata against the oracle everywhere; payload by sampled
    home-byte checks and recorded scatter bytes; replicas against the
    oracle's hot set."""
    w = synth.build("llama70b_full")
    kv, tiers = w.shape, w.tiers
    store = P.PrefixStore(_shape(kv), tiers["device_blocks"] + tiers["replica_blocks"],
                          flags=P.PTSTORE_FLAG_EVICT, host_blocks=tiers["host_blocks"],
                          replica_blocks=tiers["replica_blocks"])
    cap = store.stats()["capacity"]
    assert cap == len(w.stored) * w.passage_blocks
    ref = OracleStore.for_shape(kv, cap, with_payload=False, evict=True)
    rec = Recorder(kv, 96, 9)
    st_, so = w.store_batch()
    for k in range(len(so) - 1):
        insert_scatter(store, ref, kv, st_[so[k]:so[k + 1]], (so[k:k + 2] - so[k]).astype(np.int64),
                       w.passage_blocks, seed=k, rec=rec, k=3)
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    assert store.stats()["blocks_stored"] == ref.count == cap
    owned = store.stats()["device_blocks"]
    maxb = w.max_blocks
    cache = torch.empty(kv.layers * 2 * maxb * kv.chunk_bytes, dtype=torch.uint8, device=DEV)
    rng = np.random.default_rng(3)
    seen = 0
    host_hits = 0
    for rnd in range(2):
        for lo, hi in w.sub_batches():
            toks, offs = w.request_slice(lo, hi)
            bt_h = np.arange((hi - lo) * maxb, dtype=np.int32).reshape(hi - lo, maxb)
            cache.fill_(SENTINEL)
            m, ids = store.lookup_gather(to_dev(toks), to_dev(offs), maxb, to_dev(bt_h), cache)
            rm, rids = ref.lookup(toks, offs, maxb)
            m_h, ids_h = host(m), host(ids)
            np.testing.assert_array_equal(m_h, rm)
            np.testing.assert_array_equal(ids_h, rids)
            host_hits += int((ids_h[0, :m_h[0]] >= owned).sum())
            seen += _check_gather_tiered(store, kv, cache, m_h, ids_h, bt_h, rng, rec)
        check_access_counts(store, ref)
        if rnd == 0:  # replicate the host tier's hot set, then read through it
            store.replicate()
            torch.cuda.synchronize()
            rep = host(store.replica_map())
            have = np.flatnonzero(rep >= 0)
            np.testing.assert_array_equal(owned + have, ref.hot_set(owned, ref.count, tiers["replica_blocks"]))
            sample = rng.choice(have, size=min(64, len(have)), replace=False)
            dev_rows = store.pool_tensor()[torch.from_numpy(owned + rep[sample].astype(np.int64)).to(DEV)]
            assert torch.equal(dev_rows, store.block_bytes_of(owned + sample))
    assert host_hits > 0 and seen > 0
    del cache
    _free(store, ref)


def _block_of(cache: torch.Tensor, nb: int, chunks, cb: int) -> torch.Tensor:
    """Bytes of cache block cb in pool-block order (layer after layer, K then V):
    layer l of the cache takes the next 2 * nb * chunks[l] bytes."""
    out, off = [], 0
    for ch in chunks:
        v = cache[off:off + 2 * nb * ch].view(2, nb, ch)
        out.append(v[:, cb].reshape(-1))
        off += 2 * nb * ch
    return torch.cat(out)


def test_hybrid8b_full():
    """Per-layer slab sizes (32 KiB / 8 KiB alternating) at the 8B-shaped
    workload's full size: metadata against the oracle, sampled blocks against
    the pool and the bytes recorded at scatter, and a layer-range gather."""
    w = synth.build("hybrid8b")
    kv = w.shape
    chunks = kv.layer_chunk_bytes
    cap = len(w.stored) * w.passage_blocks
    shape = P.StoreShape(kv.layers, kv.kv_heads, kv.head_dim, kv.block_tokens, kv.elem_bytes, chunks)
    store = P.PrefixStore(shape, cap)
    ref = OracleStore.for_shape(kv, cap, with_payload=False)
    rng = np.random.default_rng(8)
    recorded = {}
    st_, so = w.store_batch()
    g = torch.Generator(device=DEV)
    for lo in range(0, len(so) - 1, 16):
        hi = min(len(so) - 1, lo + 16)
        toks, offs = st_[so[lo]:so[hi]], (so[lo:hi + 1] - so[lo]).astype(np.int64)
        m, ids, cr = store.insert(to_dev(toks), to_dev(offs), w.passage_blocks)
        rc, rm, rids, rcr = ref.insert(toks, offs, w.passage_blocks)
        ids_h, cr_h = host(ids), host(cr)
        np.testing.assert_array_equal(ids_h, rids)
        np.testing.assert_array_equal(cr_h, rcr)
        nb = (hi - lo) * w.passage_blocks
        cache = torch.empty(nb * kv.block_bytes, dtype=torch.uint8, device=DEV)
        g.manual_seed(lo)
        cache.random_(0, 256, generator=g)
        bt_h = np.arange(nb, dtype=np.int32).reshape(hi - lo, w.passage_blocks)
        store.scatter(ids, cr, to_dev(bt_h), cache)
        for r, b in np.argwhere(cr_h != 0)[rng.choice(int((cr_h != 0).sum()), 4, replace=False)]:
            recorded[int(ids_h[r, b])] = host(_block_of(cache, nb, chunks, int(bt_h[r, b])))
        del cache
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    assert store.stats()["block_bytes"] == kv.block_bytes == 2 * sum(chunks)
    pool = store.pool_tensor()
    maxb = w.max_blocks
    nbc = w.sub_batch * maxb
    cache = torch.empty(nbc * kv.block_bytes, dtype=torch.uint8, device=DEV)
    seen = 0
    for k, (lo, hi) in enumerate(w.sub_batches()):
        toks, offs = w.request_slice(lo, hi)
        R = hi - lo
        bt_h = np.arange(R * maxb, dtype=np.int32).reshape(R, maxb)
        cache.fill_(SENTINEL)
        layers = None if k == 0 else (3, 7)
        m, ids = store.lookup(to_dev(toks), to_dev(offs), maxb)
        store.gather(ids, m, to_dev(bt_h), cache, layers=layers)
        rm, rids = ref.lookup(toks, offs, maxb)
        m_h, ids_h = host(m), host(ids)
        np.testing.assert_array_equal(m_h, rm)
        np.testing.assert_array_equal(ids_h, rids)
        lb = np.concatenate([[0], np.cumsum([2 * c for c in chunks])])
        for r in rng.choice(R, 12, replace=False):
            for b in rng.choice(maxb, 6, replace=False):
                got = _block_of(cache, nbc, chunks, int(bt_h[r, b]))
                if b >= m_h[r]:
                    assert bool((got == SENTINEL).all())
                    continue
                row = pool[int(ids_h[r, b])]
                if layers is None:
                    assert torch.equal(got, row)
                    if int(ids_h[r, b]) in recorded:
                        np.testing.assert_array_equal(host(got), recorded[int(ids_h[r, b])])
                        seen += 1
                else:
                    a, e = int(lb[layers[0]]), int(lb[layers[1]])
                    assert torch.equal(got[a:e], row[a:e])
                    assert bool((got[:a] == SENTINEL).all()) and bool((got[e:] == SENTINEL).all())
        for i, want in recorded.items():  # the pool keeps what was scattered
            np.testing.assert_array_equal(host(pool[i]), want)
            seen += 1
    assert seen > 0
    del cache
    _free(store, ref)
