"""Every option together, at random: GPU library vs the CPU oracle.

Each seed draws a store (block size, uniform or per-layer slabs, capacity,
index size, eviction, host tier and replicas, 8-bit keys, copy shape) and a
sequence of operations (insert + whole or per-layer scatter, lookup + whole
gather, lookup + layer-range gather, replicate) and compares every output,
every gathered byte, the pool, the block metadata and, with eviction, every
block's access count and priority, after every step.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from tests.helpers import random_block_batch, block_table_identity

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2607_22648_amd import ptstore as P
    from tests.twin import Twin


def _atoms(rng, n, bt, vocab):
    while True:
        a = rng.integers(0, vocab, size=(n, bt), dtype=np.int32)
        if len({r.tobytes() for r in a}) == n:
            return a


def _draw_store(rng):
    bt = int(rng.choice([1, 2, 3, 16]))
    layers = int(rng.integers(1, 5))
    chunks = None
    if rng.random() < 0.5:
        chunks = [int(16 * rng.integers(1, 7)) for _ in range(layers)]
    evict = rng.random() < 0.6
    flags = (P.PTSTORE_FLAG_EVICT if evict else 0) | (P.PTSTORE_FLAG_WEAK_HASH if rng.random() < 0.3 else 0)
    pool = int(rng.integers(2, 14))
    host_blocks = int(rng.integers(0, 20)) if rng.random() < 0.5 else 0
    replicas = 0
    if evict and host_blocks and rng.random() < 0.7:
        replicas = int(rng.integers(1, pool // 2 + 1))
    index_slots = int(rng.choice([0, 0, 64, 128]))
    kw = dict(flags=flags, host_blocks=host_blocks, replica_blocks=replicas, index_slots=index_slots)
    if chunks:
        t = Twin(layers, 1, 1, bt, pool, layer_chunk_bytes=chunks, **kw)
    else:
        t = Twin(layers, 1, 8, bt, pool, **kw)  # uniform slabs of bt * 8 * 2 bytes
    if rng.random() < 0.4:
        t.gpu.set_copy_shape(int(rng.choice([1, 2, 3, 5])), int(rng.choice([64, 256, 1024])), 0)
    return t, bt, evict, replicas


@pytest.mark.parametrize("seed", range(24))
def test_random_combination(seed):
    rng = np.random.default_rng(9000 + seed)
    t, bt, evict, replicas = _draw_store(rng)
    L = t.shape.layers
    atoms = _atoms(rng, int(rng.integers(2, 6)), bt, 500)
    maxb = int(rng.integers(2, 8))
    for i in range(25):
        toks, offs = random_block_batch(rng, int(rng.integers(1, 9)), atoms, maxb + 1)
        R = len(offs) - 1
        bt_tab = block_table_identity(R, maxb)
        u = rng.random()
        if replicas and u < 0.15:
            t.gpu.replicate()
            t.check_replicas()
        elif u < 0.45:
            (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, maxb)
            if L > 1 and rng.random() < 0.5:
                cut = int(rng.integers(1, L))
                t.scatter_random(ids, cr, rids, rcr, bt_tab, seed=seed * 1000 + i, layers=(0, cut))
                t.scatter_random(ids, cr, rids, rcr, bt_tab, seed=seed * 1000 + i + 500,
                                 layers=(cut, L))
            else:
                t.scatter_random(ids, cr, rids, rcr, bt_tab, seed=seed * 1000 + i)
        elif u < 0.75:
            t.lookup_gather(toks, offs, maxb, bt_tab, R * maxb)
        else:
            (m, ids), (rm, rids) = t.lookup(toks, offs, maxb)
            l0 = int(rng.integers(0, L))
            l1 = int(rng.integers(l0 + 1, L + 1))
            t.gather_layers(m, ids, rm, rids, bt_tab, R * maxb, (l0, l1))
        if evict:
            t.check_evict()
    t.check_pool()
    t.check_meta()
    if replicas:
        t.check_replicas(hot_set=False)
    t.close()
