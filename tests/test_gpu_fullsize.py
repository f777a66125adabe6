"""Parity at the workloads' full sizes, in the launch configuration bench.py times.

At these sizes the oracle runs without payload (its trie alone). Every
copied byte is still checked, through this chain:
1. m, ids and created of every insert and lookup equal the oracle's, exactly;
2. right after each scatter, every block it created holds, in its home row
   (device pool or host tier), exactly the bytes of its cache block;
3. after the prefill, the whole pool is checked once more against its
   inputs: each scatter's seeded cache is drawn again and every block holds
   the bytes of the scatter that last wrote it (a later scatter writing
   outside its own blocks fails here);
4. every gathered block equals its home row, and every cache block or
   layer the gather must not touch still holds the sentinel.
Bytes recorded from sampled blocks at scatter time are compared with what
the gathers return as an end-to-end check of the same chain.
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
CMP_BYTES = 512 << 20  # bytes of blocks compared per step


def _shape(kv):
    return P.StoreShape(kv.layers, kv.kv_heads, kv.head_dim, kv.block_tokens, kv.elem_bytes,
                        kv.layer_chunk_bytes)


def _free(*objs):
    for o in objs:
        if hasattr(o, "close"):
            o.close()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def seeded_cache(kv, nb_cache: int, seed: int) -> torch.Tensor:
    """A flat paged cache of nb_cache blocks filled with seeded random bytes
    (the same bytes every time for the same seed and size)."""
    cache = torch.empty(nb_cache * kv.block_bytes, dtype=torch.uint8, device=DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    cache.random_(0, 256, generator=g)
    return cache


def cache_block_bytes(kv, cache: torch.Tensor, nb_cache: int, cbs: torch.Tensor) -> torch.Tensor:
    """[n, block_bytes]: cache blocks cbs in pool-block order (layer after layer,
    K then V). Layer l of the cache takes the next 2 * nb_cache * slab_l bytes."""
    n = cbs.numel()
    if kv.layer_chunk_bytes is None:
        cv = cache.view(kv.layers, 2, nb_cache, kv.chunk_bytes)
        return cv[:, :, cbs].permute(2, 0, 1, 3).reshape(n, kv.block_bytes)
    pieces, off = [], 0
    for ch in kv.layer_chunk_bytes:
        v = cache[off:off + 2 * nb_cache * ch].view(2, nb_cache, ch)
        pieces.append(v[:, cbs].permute(1, 0, 2).reshape(n, 2 * ch))
        off += 2 * nb_cache * ch
    return torch.cat(pieces, dim=1)


def compare_blocks(store, kv, cache, nb_cache, ids: np.ndarray, cbs: np.ndarray, what: str,
                   cols=None):
    """Home bytes of block ids[k] == bytes of cache block cbs[k], for every k
    (only byte columns cols[0]:cols[1] of the block when given)."""
    per = max(1, CMP_BYTES // kv.block_bytes)
    a, e = cols if cols is not None else (0, kv.block_bytes)
    for s in range(0, len(ids), per):
        got = store.block_bytes_of(ids[s:s + per])[:, a:e]
        exp = cache_block_bytes(kv, cache, nb_cache, to_dev(cbs[s:s + per].astype(np.int64)))[:, a:e]
        if not torch.equal(got, exp):
            k = int(torch.nonzero((got != exp).any(dim=1))[0])
            raise AssertionError(f"{what}: block id {ids[s + k]} differs from cache block "
                                 f"{cbs[s + k]} ({len(ids)} blocks compared in all)")


class Ledger:
    """Which scatter last wrote each block id, from which cache block; a
    scatter's cache is kept as (seed, size) and drawn again to re-check."""

    def __init__(self, kv, capacity: int):
        self.kv = kv
        self.calls = []  # (seed, nb_cache)
        self.writer = np.full(capacity, -1, dtype=np.int64)
        self.block = np.full(capacity, -1, dtype=np.int64)

    def record(self, seed: int, nb_cache: int, ids: np.ndarray, cbs: np.ndarray):
        self.calls.append((seed, nb_cache))
        self.writer[ids] = len(self.calls) - 1
        self.block[ids] = cbs

    def verify(self, store, count: int):
        """Every block id < count holds the bytes of the scatter that last wrote it."""
        assert (self.writer[:count] >= 0).all(), "a stored block was never scattered"
        checked = 0
        for k, (seed, nb) in enumerate(self.calls):
            ids = np.flatnonzero(self.writer[:count] == k)
            if len(ids) == 0:
                continue
            cache = seeded_cache(self.kv, nb, seed)
            compare_blocks(store, self.kv, cache, nb, ids, self.block[ids],
                           f"pool re-check, scatter {k}")
            checked += len(ids)
            del cache
        assert checked == count
        return checked


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
        for r, b in cand[self.rng.choice(len(cand), size=min(k, len(cand)), replace=False)]:
            sel = torch.tensor([int(bt[r, b])], dtype=torch.int64, device=DEV)
            self.bytes[int(ids[r, b])] = host(cache_block_bytes(self.kv, cache, nb_cache, sel)[0])


def insert_scatter(store, ref, kv, toks, offs, maxb, seed, ledger: Ledger, rec: Recorder = None,
                   k=4, compact=False):
    """Insert on both sides (outputs compared), scatter seeded random KV on the
    GPU, then compare every created block with its cache block.

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
    cache = seeded_cache(kv, nb_cache, seed)
    store.scatter(ids, cr, to_dev(bt), cache)
    made = (cr_h != 0) & (bt >= 0)
    compare_blocks(store, kv, cache, nb_cache, ids_h[made], bt[made], f"scatter seed {seed}")
    ledger.record(seed, nb_cache, ids_h[made], bt[made])
    if rec is not None:
        rec.take(cache, nb_cache, ids_h, cr_h, bt, k)
    torch.cuda.synchronize()
    del cache
    return ids_h, cr_h


def check_gather(store, kv, cache, m_h, ids_h, bt_h, rec: Recorder = None, layers=None):
    """Every gathered block equals its home row (within the layer range when
    given: the rest of every block keeps the sentinel); every cache block the
    gather must not touch keeps the sentinel; recorded bytes where seen."""
    nb_cache = cache.numel() // kv.block_bytes
    hit = (np.arange(ids_h.shape[1])[None, :] < m_h[:, None]) & (bt_h >= 0)
    cols = None
    if layers is not None:
        lb = np.concatenate([[0], np.cumsum([2 * c for c in (kv.layer_chunk_bytes or
                                                             [kv.chunk_bytes] * kv.layers)])])
        cols = (int(lb[layers[0]]), int(lb[layers[1]]))
    compare_blocks(store, kv, cache, nb_cache, ids_h[hit].astype(np.int64),
                   bt_h[hit].astype(np.int64), "gather", cols=cols)
    per = max(1, CMP_BYTES // kv.block_bytes)
    if cols is not None:  # the other layers of the gathered blocks are untouched
        sel = bt_h[hit].astype(np.int64)
        for s in range(0, len(sel), per):
            got = cache_block_bytes(kv, cache, nb_cache, to_dev(sel[s:s + per]))
            assert bool((got[:, :cols[0]] == SENTINEL).all()) and \
                bool((got[:, cols[1]:] == SENTINEL).all()), "gather wrote outside its layers"
    untouched = np.ones(nb_cache, dtype=bool)
    untouched[bt_h[hit]] = False
    un = np.flatnonzero(untouched)
    for s in range(0, len(un), per):
        got = cache_block_bytes(kv, cache, nb_cache, to_dev(un[s:s + per]))
        assert bool((got == SENTINEL).all()), "gather wrote outside its blocks"
    seen = 0
    if rec is not None:
        for (r, b) in np.argwhere(hit):
            i = int(ids_h[r, b])
            if i in rec.bytes:
                sel = torch.tensor([int(bt_h[r, b])], dtype=torch.int64, device=DEV)
                got = host(cache_block_bytes(kv, cache, nb_cache, sel)[0])
                a, e = cols if cols is not None else (0, kv.block_bytes)
                np.testing.assert_array_equal(got[a:e], rec.bytes[i][a:e])
                seen += 1
    return seen


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
    return m_h, ids_h, seen


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
    cap = store.stats()["capacity"]
    ref = OracleStore.for_shape(kv, cap, with_payload=False, evict=evict)
    ledger = Ledger(kv, cap)
    st, so = w.store_batch()
    Rs = len(so) - 1
    for lo in range(0, Rs, batch):
        hi = min(Rs, lo + batch)
        insert_scatter(store, ref, kv, st[so[lo]:so[hi]], (so[lo:hi + 1] - so[lo]).astype(np.int64),
                       w.passage_blocks, seed=lo, ledger=ledger, rec=rec, k=8)
    assert store.stats()["blocks_stored"] == ref.count == len(w.stored) * w.passage_blocks
    assert ledger.verify(store, ref.count) == ref.count
    return store, ref, ledger


def test_llama8b_full():
    w = synth.build("llama8b")
    kv = w.shape
    rec = Recorder(kv, 64, 1)
    store, ref, _ = _passage_store(w, len(w.stored) * w.passage_blocks, 32, rec)
    maxb = w.max_blocks
    cache = torch.empty(w.sub_batch * maxb * kv.block_bytes, dtype=torch.uint8, device=DEV)
    seen = 0
    for lo, hi in w.sub_batches():
        toks, offs = w.request_slice(lo, hi)
        m_h, _, s = lookup_gather_checked(store, ref, kv, toks, offs, maxb, cache, rec)
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
    store, ref, _ = _passage_store(w, len(w.stored) * w.passage_blocks, 2, rec)
    maxb = w.max_blocks
    cache = torch.empty(w.sub_batch * maxb * kv.block_bytes, dtype=torch.uint8, device=DEV)
    seen = 0
    for lo, hi in w.sub_batches():
        toks, offs = w.request_slice(lo, hi)
        m_h, _, s = lookup_gather_checked(store, ref, kv, toks, offs, maxb, cache, rec)
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
    ledger = Ledger(kv, w.capacity)
    rec = Recorder(kv, 256, 3)
    W = len(w.store_offsets) - 1
    batch = 32768
    for lo in range(0, W, batch):
        hi = min(W, lo + batch)
        toks = w.store_tokens[w.store_offsets[lo]:w.store_offsets[hi]]
        offs = (w.store_offsets[lo:hi + 1] - w.store_offsets[lo]).astype(np.int64)
        insert_scatter(store, ref, kv, toks, offs, w.depth, seed=lo, ledger=ledger, rec=rec, k=16,
                       compact=True)
    st = store.stats()
    assert st["blocks_stored"] == ref.count == w.capacity and st["full_events"] >= 1
    assert ledger.verify(store, ref.count) == w.capacity
    R = w.n_requests
    cache = torch.empty(R * w.depth * kv.block_bytes, dtype=torch.uint8, device=DEV)
    m_h, _, seen = lookup_gather_checked(store, ref, kv, w.tokens, w.offsets, w.depth, cache, rec)
    assert seen > 0 and m_h.mean() > 60
    del cache
    _free(store, ref)


@pytest.mark.parametrize("name,rounds", [("stream", None), ("stream_evict", 14)])
def test_stream_full(name, rounds):
    """100 rounds of the stream on the 160 GB pool; with eviction, 14 rounds (the
    pool fills in the sixth; the oracle's one-leaf-at-a-time eviction is slow).
    Each round's lookup cache is re-filled with seeded bytes for its inserts'
    scatter; at the end the whole pool is re-checked against those draws."""
    over = {} if rounds is None else {"n_rounds": rounds}
    sw = synth.build(name, **over)
    evict = name == "stream_evict"
    base = sw.base
    kv = base.shape
    rec = Recorder(kv, 64, 4)
    store, ref, ledger = _passage_store(base, sw.pool_blocks, 32, rec, evict=evict)
    maxb = base.max_blocks
    per = len(sw.rounds[0].lookup_offsets) - 1
    nb_cache = per * maxb
    cache = torch.empty(nb_cache * kv.block_bytes, dtype=torch.uint8, device=DEV)
    g = torch.Generator(device=DEV)
    seen = 0
    for i, rd in enumerate(sw.rounds):
        _, _, s = lookup_gather_checked(store, ref, kv, rd.lookup_tokens, rd.lookup_offsets, maxb,
                                        cache, rec)
        seen += s
        # inserts: KV of the new blocks is fresh in the cache, then scattered
        Ri = len(rd.insert_offsets) - 1
        bt_h = np.arange(Ri * maxb, dtype=np.int32).reshape(Ri, maxb)
        seed = 10_000 + i
        g.manual_seed(seed)
        cache.random_(0, 256, generator=g)  # the bytes seeded_cache(kv, nb_cache, seed) draws
        m, ids, cr = store.insert(to_dev(rd.insert_tokens), to_dev(rd.insert_offsets), maxb)
        rc, rm, rids, rcr = ref.insert(rd.insert_tokens, rd.insert_offsets, maxb)
        ids_h, cr_h = host(ids), host(cr)
        np.testing.assert_array_equal(host(m), rm)
        np.testing.assert_array_equal(ids_h, rids)
        np.testing.assert_array_equal(cr_h, rcr)
        store.scatter(ids, cr, to_dev(bt_h), cache)
        made = cr_h != 0
        if made.any():
            compare_blocks(store, kv, cache, nb_cache, ids_h[made], bt_h[made], f"round {i} scatter")
            ledger.record(seed, nb_cache, ids_h[made], bt_h[made])
            for reused in ids_h[made].tolist():  # an evicted id now holds another block
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
    torch.cuda.empty_cache()
    assert ledger.verify(store, ref.count) == ref.count
    _free(store, ref)


def test_llama70b_full_tiered():
    """All 32 passages (322 GB) on one GPU: HBM, HBM replicas and the pinned
    host tier. Metadata against the oracle everywhere; every scattered and
    every gathered block against its home bytes (host-tier rows read back
    from pinned memory); replicas against the oracle's hot set and their
    home bytes."""
    w = synth.build("llama70b_full")
    kv, tiers = w.shape, w.tiers
    store = P.PrefixStore(_shape(kv), tiers["device_blocks"] + tiers["replica_blocks"],
                          flags=P.PTSTORE_FLAG_EVICT, host_blocks=tiers["host_blocks"],
                          replica_blocks=tiers["replica_blocks"])
    cap = store.stats()["capacity"]
    assert cap == len(w.stored) * w.passage_blocks
    ref = OracleStore.for_shape(kv, cap, with_payload=False, evict=True)
    ledger = Ledger(kv, cap)
    rec = Recorder(kv, 96, 9)
    st_, so = w.store_batch()
    for k in range(len(so) - 1):
        insert_scatter(store, ref, kv, st_[so[k]:so[k + 1]], (so[k:k + 2] - so[k]).astype(np.int64),
                       w.passage_blocks, seed=k, ledger=ledger, rec=rec, k=3)
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    assert store.stats()["blocks_stored"] == ref.count == cap
    assert ledger.verify(store, cap) == cap
    owned = store.stats()["device_blocks"]
    maxb = w.max_blocks
    cache = torch.empty(maxb * kv.block_bytes, dtype=torch.uint8, device=DEV)
    seen = 0
    host_hits = 0
    for rnd in range(2):
        for lo, hi in w.sub_batches():
            toks, offs = w.request_slice(lo, hi)
            m_h, ids_h, s = lookup_gather_checked(store, ref, kv, toks, offs, maxb, cache, rec)
            host_hits += int((ids_h[0, :m_h[0]] >= owned).sum())
            seen += s
        check_access_counts(store, ref)
        if rnd == 1:
            # all requests looked up at once, then loads of requests that read
            # the host tier on one stream and of the others on a second, two
            # caches, pairs in flight together; every byte checked per pair
            toks, offs = w.request_slice(0, w.n_requests)
            m, ids = store.lookup(to_dev(toks), to_dev(offs), maxb)
            rm, rids = ref.lookup(toks, offs, maxb)
            m_h, ids_h = host(m), host(ids)
            np.testing.assert_array_equal(m_h, rm)
            np.testing.assert_array_equal(ids_h, rids)
            rep = host(store.replica_map())
            on_host = [bool(((ids_h[r, :m_h[r]] >= owned) &
                             (rep[np.maximum(ids_h[r, :m_h[r]] - owned, 0)] < 0)).any())
                       for r in range(len(m_h))]
            hr = [r for r in range(len(m_h)) if on_host[r]]
            dr = [r for r in range(len(m_h)) if not on_host[r]]
            assert hr and dr
            cache2 = torch.empty_like(cache)
            s_h, s_d = torch.cuda.Stream(), torch.cuda.Stream()
            bt1 = np.arange(maxb, dtype=np.int32).reshape(1, maxb)
            for k in range(max(len(hr), len(dr))):
                pair = [(s_h, hr[k], cache2)] if k < len(hr) else []
                pair += [(s_d, dr[k], cache)] if k < len(dr) else []
                torch.cuda.synchronize()
                for st_, r, c in pair:
                    c.fill_(SENTINEL)
                torch.cuda.synchronize()
                for st_, r, c in pair:
                    store.gather(ids[r:r + 1], m[r:r + 1], to_dev(bt1), c, stream=st_)
                torch.cuda.synchronize()
                for st_, r, c in pair:
                    seen += check_gather(store, kv, c, m_h[r:r + 1], ids_h[r:r + 1], bt1, rec)
            del cache2
            check_access_counts(store, ref)  # the one lookup of this phase, on both sides
        if rnd == 0:  # replicate the host tier's hot set, then read through it
            store.replicate()
            torch.cuda.synchronize()
            rep = host(store.replica_map())
            have = np.flatnonzero(rep >= 0)
            np.testing.assert_array_equal(owned + have, ref.hot_set(owned, ref.count, tiers["replica_blocks"]))
            per = max(1, CMP_BYTES // kv.block_bytes)
            for s in range(0, len(have), per):  # every replica row holds its home bytes
                h = have[s:s + per]
                dev_rows = store.pool_tensor()[torch.from_numpy(owned + rep[h].astype(np.int64)).to(DEV)]
                assert torch.equal(dev_rows, store.block_bytes_of(owned + h)), "replica bytes"
    assert host_hits > 0 and seen > 0
    del cache
    _free(store, ref)


def test_hybrid8b_full():
    """Per-layer slab sizes (32 KiB / 8 KiB alternating) at the 8B-shaped
    workload's full size: metadata against the oracle, every scattered and
    gathered block against its home row, and a layer-range gather."""
    w = synth.build("hybrid8b")
    kv = w.shape
    cap = len(w.stored) * w.passage_blocks
    store = P.PrefixStore(_shape(kv), cap)
    ref = OracleStore.for_shape(kv, cap, with_payload=False)
    ledger = Ledger(kv, cap)
    rec = Recorder(kv, 64, 8)
    st_, so = w.store_batch()
    for lo in range(0, len(so) - 1, 16):
        hi = min(len(so) - 1, lo + 16)
        insert_scatter(store, ref, kv, st_[so[lo]:so[hi]], (so[lo:hi + 1] - so[lo]).astype(np.int64),
                       w.passage_blocks, seed=lo, ledger=ledger, rec=rec, k=4)
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    assert store.stats()["block_bytes"] == kv.block_bytes == 2 * sum(kv.layer_chunk_bytes)
    assert store.stats()["blocks_stored"] == ref.count == cap
    assert ledger.verify(store, cap) == cap
    maxb = w.max_blocks
    cache = torch.empty(w.sub_batch * maxb * kv.block_bytes, dtype=torch.uint8, device=DEV)
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
        seen += check_gather(store, kv, cache, m_h, ids_h, bt_h, rec, layers=layers)
    assert seen > 0
    del cache
    _free(store, ref)
