"""Gathers in which many cache blocks need the same stored block, vs the oracle.

Section 4.1 (one batched transfer moves the matched KV blocks of a whole
batch of requests into the paged cache): when requests share a prefix,
several entries of one gather read the same stored block. The library
groups a call's entries by stored row and reads each row once, writing it
to every cache block that needs it, at most 64 cache blocks per copy
descriptor. These cases make rows with up to several hundred destinations:
requests that share one long passage, on both sides of the one-workgroup
limit of the list build (8,192 (request, block) slots), with host-tier and
replica rows, with per-layer slab sizes and with a list built once and
copied layer by layer. Every byte of the cache is compared with the
oracle's gather, which copies entry by entry.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from workloads.synth import concat_requests

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2607_22648_amd import ptstore as P
    from tests.twin import Twin, host, to_dev


def _store_passages(t, rng, lengths, seed):
    """Insert one passage per length (in blocks) and scatter seeded bytes into
    them; returns the passages' tokens."""
    bt = t.shape.block_tokens
    seqs = [rng.integers(0, 1 << 20, size=n * bt, dtype=np.int32) for n in lengths]
    toks, offs = concat_requests(seqs)
    maxb = max(lengths)
    R = len(seqs)
    (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, maxb)
    bt_tab = np.arange(R * maxb, dtype=np.int32).reshape(R, maxb)
    t.scatter_random(ids, cr, rids, rcr, bt_tab, seed=seed)
    return seqs


def _requests(rng, passages, R, maxb, bt, p_full=0.5):
    """R requests, each a prefix of one passage (the first passage for about
    two thirds of them), at most maxb blocks long (the whole passage up to
    maxb with probability p_full), then a few fresh tokens."""
    seqs = []
    for _ in range(R):
        p = passages[0] if rng.random() < 0.67 else passages[int(rng.integers(0, len(passages)))]
        nb = min(len(p) // bt, maxb)
        k = nb if rng.random() < p_full else int(rng.integers(0, nb + 1))
        tail = rng.integers(1 << 21, 1 << 22, size=int(rng.integers(0, 2 * bt)), dtype=np.int32)
        seqs.append(np.concatenate([p[:k * bt], tail]).astype(np.int32))
    return concat_requests(seqs)


def _table(rng, R, maxb, holes=0.05):
    """A block table of distinct cache blocks in random order (so that every
    cache block has one writer), with some holes (-1)."""
    nb = R * maxb + 7
    tab = rng.permutation(nb)[:R * maxb].astype(np.int32).reshape(R, maxb)
    tab[rng.random(tab.shape) < holes] = -1
    return tab, nb


def _max_sharing(ids, m):
    """The largest number of entries of the call that read one block."""
    ids, m = host(ids), host(m)
    rows = np.concatenate([ids[r, :m[r]] for r in range(len(m))] + [np.zeros(0, np.int32)])
    return int(np.bincount(rows).max()) if rows.size else 0


@pytest.mark.parametrize("R,maxb", [(2, 64), (40, 16), (300, 16), (600, 16), (17, 600), (130, 70)])
def test_shared_passage(R, maxb):
    """Many requests read the same passage: rows with up to R destinations,
    split over several descriptors, in a one-workgroup list (R * maxb <=
    8192) or the multi-kernel one."""
    rng = np.random.default_rng(R * 1000 + maxb)
    t = Twin(2, 1, 8, 4, 3 * maxb + 64)
    passages = _store_passages(t, rng, [maxb, maxb // 2 + 1, maxb // 3 + 1], seed=R)
    toks, offs = _requests(rng, passages, R, maxb, 4)
    tab, nb = _table(rng, R, maxb)
    bad0 = t.gpu.stats()["bad_entries"]
    (m, ids, _), _ = t.lookup_gather(toks, offs, maxb, tab, nb)
    assert t.gpu.stats()["bad_entries"] == bad0
    if R >= 130:
        assert _max_sharing(ids, m) > 64  # some row needs more than one descriptor
    t.close()


@pytest.mark.parametrize("R", [5, 64, 65, 257])
def test_every_request_reads_every_block(R):
    """All R requests are the same passage: every row has exactly R
    destinations (R // 64 full descriptors and a partial one)."""
    rng = np.random.default_rng(R)
    maxb = 24
    t = Twin(2, 1, 8, 4, 64)
    (p,) = _store_passages(t, rng, [maxb], seed=3)
    toks, offs = concat_requests([p] * R)
    tab, nb = _table(rng, R, maxb, holes=0.0)
    (m, ids, _), _ = t.lookup_gather(toks, offs, maxb, tab, nb)
    assert (host(m) == maxb).all() and _max_sharing(ids, m) == R
    t.close()


@pytest.mark.parametrize("replicate", [False, True])
def test_shared_rows_in_the_host_tier(replicate):
    """The passage's blocks lie partly in device rows, partly in host-tier
    rows (and, after a replicate, in replica rows): rows of both parts of
    the list are shared."""
    rng = np.random.default_rng(11 + replicate)
    maxb = 48
    # replica slots come with the access counts that choose them (eviction on)
    t = Twin(2, 1, 8, 4, 40, host_blocks=200, replica_blocks=8 if replicate else 0,
             flags=P.PTSTORE_FLAG_EVICT if replicate else 0)
    passages = _store_passages(t, rng, [maxb, 20], seed=5)
    assert t.gpu.stats()["device_blocks"] < maxb  # the passage spills into the host tier
    for k in range(3):
        toks, offs = _requests(rng, passages, 90, maxb, 4)
        tab, nb = _table(rng, 90, maxb)
        t.lookup_gather(toks, offs, maxb, tab, nb)
        if replicate:
            t.gpu.replicate()
            t.check_replicas(hot_set=False)
    t.close()


@pytest.mark.parametrize("chunks", [[32, 96, 16, 64, 48], None])
@pytest.mark.parametrize("R", [40, 400])
def test_shared_rows_prepared_per_layer(chunks, R):
    """A list with shared rows built once (ptstore_gather_prepare) and copied
    one layer at a time, with uniform and with per-layer slab sizes: the
    same bytes as the oracle's whole gather."""
    rng = np.random.default_rng(R + (0 if chunks else 1))
    maxb = 12
    if chunks is None:
        t = Twin(5, 2, 8, 2, 64)
    else:
        t = Twin(len(chunks), 1, 1, 2, 64, layer_chunk_bytes=chunks)
    passages = _store_passages(t, rng, [maxb, 7, 5], seed=9)
    toks, offs = _requests(rng, passages, R, maxb, 2)
    (m, ids), (rm, rids) = t.lookup(toks, offs, maxb)
    tab, nb = _table(rng, R, maxb)
    n = nb * t.shape.block_bytes
    dst = torch.full((n,), 0xA5, dtype=torch.uint8, device="cuda")
    t.gpu.gather_prepare(ids, m, to_dev(tab), dst)
    for layer in range(t.shape.layers):
        t.gpu.gather_prepared(dst, (layer, layer + 1))
    rdst = np.full(n, 0xA5, dtype=np.uint8)
    t.ref.gather(rids, rm, tab, rdst, nb)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(dst), rdst)
    # and a layer-range gather of the same list, which builds it again
    dst2, _ = t.gather_layers(m, ids, rm, rids, tab, nb, (1, 4))
    t.close()


@pytest.mark.parametrize("seed", range(12))
def test_random_sharing(seed):
    """Random batch sizes (2-700 requests, 1-40 blocks) over a few passages,
    so that sharing ranges from none to hundreds of destinations per row."""
    rng = np.random.default_rng(500 + seed)
    maxb = int(rng.choice([1, 4, 16, 40]))
    R = int(rng.integers(2, 701))
    t = Twin(2, 1, 8, 4, 4 * maxb + 64)
    lengths = [maxb] + [int(rng.integers(1, maxb + 1)) for _ in range(3)]
    passages = _store_passages(t, rng, lengths, seed=seed)
    toks, offs = _requests(rng, passages, R, maxb, 4, p_full=float(rng.random()))
    tab, nb = _table(rng, R, maxb, holes=float(rng.choice([0.0, 0.1])))
    t.lookup_gather(toks, offs, maxb, tab, nb)
    t.close()
