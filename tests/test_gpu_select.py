"""Both ways of building the copies' descriptor list, at their boundary, against the oracle.

A gather or scatter first lists the blocks it moves (the bulk list of
segments of a load or store, Section 4.1). Small batches, at most 64
requests and 8,192 (request, block) entries, build the list in one
workgroup; larger ones in three kernels (count, scan, fill). On both sides
of that boundary, with a host tier (rows read and written over the host link,
listed after the device rows), holes (-1) and out-of-range cache blocks in
the block table, every gathered and scattered byte, m, ids and the number of
skipped entries must equal the oracle's.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from tests.helpers import random_block_batch, block_table_identity

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from tests.twin import Twin


def _atoms(rng, n, bt, vocab):
    while True:
        a = rng.integers(0, vocab, size=(n, bt), dtype=np.int32)
        if len({r.tobytes() for r in a}) == n:
            return a


# (R, max_blocks): one workgroup up to 64 requests and 8,192 entries, three
# kernels past either limit
SIZES = [(1, 1), (1, 64), (40, 8), (64, 128), (64, 129), (65, 64), (16, 512), (17, 512), (130, 40)]


@pytest.mark.parametrize("R,maxb", SIZES)
def test_list_build_both_ways(R, maxb):
    rng = np.random.default_rng(R * 1000 + maxb)
    atoms = _atoms(rng, 6, 4, 700)
    # ids 0..99 live in device memory, the next 5,000 in the host tier
    t = Twin(2, 1, 8, 4, 100, host_blocks=5000)
    batches = [random_block_batch(rng, R, atoms, maxb, tail_p=0.3) for _ in range(3)]
    for k, (toks, offs) in enumerate(batches):  # inserts and scatters at this size
        (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, maxb)
        t.scatter_random(ids, cr, rids, rcr, block_table_identity(R, maxb), seed=50 + k)
    t.check_pool()
    stored = t.ref.count
    # a gather of the first batch again (stored whole while the store was
    # empty: long matches in both tiers) through a permuted table with holes
    # and out-of-range entries
    toks, offs = batches[0]
    NB = R * maxb + 5
    bt = rng.permutation(NB)[:R * maxb].astype(np.int32).reshape(R, maxb)
    bt[rng.random(bt.shape) < 0.15] = -1
    oob = rng.random(bt.shape) < 0.05
    bt[oob] = NB + rng.integers(0, 50, size=int(oob.sum()), dtype=np.int32)
    b0, r0 = t.gpu.stats()["bad_entries"], t.ref.bad_entries
    (m, ids, dst), (rm, rids, rdst) = t.lookup_gather(toks, offs, maxb, bt, NB)
    assert t.gpu.stats()["bad_entries"] - b0 == t.ref.bad_entries - r0
    moved = (np.arange(maxb)[None, :] < rm[:, None]) & (bt >= 0) & (bt < NB)
    if R >= 16:  # these cases move blocks of both tiers
        assert stored > 100 and (rids[moved] >= 100).any() and (rids[moved] < 100).any()
    t.close()


@pytest.mark.parametrize("seed", range(40))
def test_random_sizes_against_the_oracle(seed):
    """Random batch shapes on both sides of the small-batch limit (1-130
    requests, 1-600 blocks each), block sizes 4 and 16, eviction and a host
    tier with replicas on or off, some scatters split by layers: inserts,
    scatters, the pool, a gather through a table with holes and out-of-range
    entries, and with eviction every access count, against the oracle."""
    from paper_2607_22648_amd import ptstore as P
    rng = np.random.default_rng(7000 + seed)
    bt = int(rng.choice([4, 16]))
    atoms = _atoms(rng, int(rng.integers(3, 8)), bt, 900)
    R = int(rng.integers(1, 131))
    maxb = int(rng.choice([1, 8, 40, 64, 65, 128, 129, 300, 600]))
    evict = bool(rng.random() < 0.4)
    host = int(rng.choice([0, 0, 400]))
    pool = int(rng.choice([60, 300, 2000]))
    reps = min(20, pool // 2) if (evict and host) else 0
    t = Twin(3, 1, 8, bt, pool, flags=P.PTSTORE_FLAG_EVICT if evict else 0, host_blocks=host,
             replica_blocks=reps)
    batches = []
    for k in range(3):
        toks, offs = random_block_batch(rng, R, atoms, maxb, tail_p=0.3)
        batches.append((toks, offs))
        (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, maxb)
        if rng.random() < 0.7:
            t.scatter_random(ids, cr, rids, rcr, block_table_identity(R, maxb), seed=seed * 10 + k)
        else:  # in two calls by layer range; every layer is written (unwritten bytes are undefined)
            for j, lay in enumerate(((0, 2), (2, 3))):
                t.scatter_random(ids, cr, rids, rcr, block_table_identity(R, maxb),
                                 seed=seed * 10 + k + 100 * j, layers=lay)
        if reps and rng.random() < 0.5:
            t.gpu.replicate()
            t.check_replicas(hot_set=True)
    t.check_pool()
    toks, offs = batches[int(rng.integers(0, 3))]
    NB = R * maxb + 3
    tab = rng.permutation(NB)[:R * maxb].astype(np.int32).reshape(R, maxb)
    tab[rng.random(tab.shape) < 0.1] = -1
    oob = rng.random(tab.shape) < 0.03
    tab[oob] = NB + rng.integers(0, 9, size=int(oob.sum()), dtype=np.int32)
    b0, r0 = t.gpu.stats()["bad_entries"], t.ref.bad_entries
    t.lookup_gather(toks, offs, maxb, tab, NB)
    assert t.gpu.stats()["bad_entries"] - b0 == t.ref.bad_entries - r0
    if evict:
        t.check_evict()
    t.close()
