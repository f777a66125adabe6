"""Lookups and loads of one store on several streams at once, against the oracle.

Each stream has its own descriptor scratch, so lookup + gather calls enqueued
on two streams without any ordering between them both return the oracle's
results: m, ids and every byte of their caches. With eviction on, the access
counts of all those lookups add up to the oracle's (they commute). A store
with a host tier moves host-tier rows with a small grid of its own; the
bytes are still exact.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from tests.helpers import random_block_batch, block_table_identity

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2607_22648_amd import ptstore as P
    from tests.twin import Twin, to_dev, host, DEV


def _atoms(rng, n, bt, vocab):
    while True:
        a = rng.integers(0, vocab, size=(n, bt), dtype=np.int32)
        if len({r.tobytes() for r in a}) == n:
            return a


def _filled(rng, atoms, t, n_batches, R, maxb):
    for k in range(n_batches):
        toks, offs = random_block_batch(rng, R, atoms, maxb, tail_p=0.2)
        (_, ids, cr), (_, _, rids, rcr) = t.insert(toks, offs, maxb)
        Ri = len(offs) - 1
        t.scatter_random(ids, cr, rids, rcr, block_table_identity(Ri, maxb), seed=1000 + k)


@pytest.mark.parametrize("sizes", [(37, 11), (100, 11)])
@pytest.mark.parametrize("host_blocks,evict", [(0, False), (300, False), (300, True)])
def test_loads_on_two_streams(host_blocks, evict, sizes):
    """Two streams' lookups + gathers with no order between them; with
    (100, 11) requests one stream lists its blocks in three kernels and the
    other in one workgroup."""
    rng = np.random.default_rng(11 + host_blocks + evict + sizes[0])
    atoms = _atoms(rng, 6, 4, 500)
    maxb = 10
    flags = P.PTSTORE_FLAG_EVICT if evict else 0
    t = Twin(3, 2, 8, 4, 120, flags=flags, host_blocks=host_blocks,
             replica_blocks=20 if evict and host_blocks else 0)
    _filled(rng, atoms, t, 8, 24, maxb)
    if evict and host_blocks:
        t.gpu.replicate()
        t.check_replicas()
    batches = []
    for R in sizes:  # different sizes: each stream's scratch has its own size
        toks, offs = random_block_batch(rng, R, atoms, maxb + 2, tail_p=0.3)
        batches.append((toks, offs, R))
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    reps = 4
    outs = []
    for (toks, offs, R), st in zip(batches, (s1, s2)):
        tt, oo, bt = to_dev(toks), to_dev(offs), to_dev(block_table_identity(R, maxb))
        cache = torch.full((R * maxb * t.shape.block_bytes,), 0xA5, dtype=torch.uint8, device=DEV)
        m = torch.empty(R, dtype=torch.int32, device=DEV)
        ids = torch.empty((R, maxb), dtype=torch.int32, device=DEV)
        outs.append((tt, oo, bt, cache, m, ids, R))
    torch.cuda.synchronize()
    for _ in range(reps):  # the two streams' calls interleaved, nothing orders them
        for (tt, oo, bt, cache, m, ids, R), st in zip(outs, (s1, s2)):
            t.gpu.lookup_gather(tt, oo, maxb, bt, cache, m=m, ids=ids, stream=st)
    torch.cuda.synchronize()
    for (toks, offs, R), (tt, oo, bt, cache, m, ids, _) in zip(batches, outs):
        for _ in range(reps):  # the oracle counts the same accesses
            rm, rids = t.ref.lookup(toks, offs, maxb)
        rdst = np.full(cache.numel(), 0xA5, dtype=np.uint8)
        t.ref.gather(rids, rm, block_table_identity(R, maxb), rdst, R * maxb)
        np.testing.assert_array_equal(host(m), rm)
        np.testing.assert_array_equal(host(ids), rids)
        np.testing.assert_array_equal(host(cache), rdst)
        assert rm.sum() > 0
    if evict:
        t.check_evict()
    t.close()


def test_streams_per_store_are_bounded():
    """Sixteen streams each get a descriptor scratch (the current stream, used
    by the filling inserts and scatters, and fifteen more); a seventeenth is
    refused before any work is enqueued."""
    rng = np.random.default_rng(5)
    atoms = _atoms(rng, 4, 4, 100)
    t = Twin(1, 1, 8, 4, 200)
    _filled(rng, atoms, t, 2, 8, 6)
    toks, offs = random_block_batch(rng, 5, atoms, 6)
    (m, ids), (rm, rids) = t.lookup(toks, offs, 6)
    bt = to_dev(block_table_identity(5, 6))
    streams = [torch.cuda.Stream() for _ in range(16)]
    caches = []
    for st in streams[:15]:
        cache = torch.zeros(5 * 6 * t.shape.block_bytes, dtype=torch.uint8, device=DEV)
        t.gpu.gather(ids, m, bt, cache, stream=st)
        caches.append(cache)
    with pytest.raises(P.PTStoreError) as ei:
        t.gpu.gather(ids, m, bt, caches[0], stream=streams[15])
    assert ei.value.code == P.PTSTORE_ERR_INVALID
    torch.cuda.synchronize()
    rdst = np.zeros(caches[0].numel(), dtype=np.uint8)
    t.ref.gather(rids, rm, block_table_identity(5, 6), rdst, 30)
    for c in caches:
        np.testing.assert_array_equal(host(c), rdst)
    t.close()
