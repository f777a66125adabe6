"""Pins of the oracle's layer ranges and per-layer slab sizes (no GPU).

Section 5: clients read and write subsets of tensors, and prefixes are
combinations of tensors of variable sizes. Here a load or store may name a
range of layers, and each layer's (K|V) slab may have its own size. The
layouts are restated by slicing flat buffers layer after layer:
- paged cache: layer l takes the next 2 * cache_blocks * chunk[l] bytes,
  as [K|V][cache block][chunk[l]];
- pool block: layer l takes the next 2 * chunk[l] bytes, as [K|V][chunk[l]].
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import OracleStore, ORC_OK
from tests.helpers import random_block_batch, block_table_identity

CHUNKS = [32, 96, 16, 64, 48]  # bytes per (layer, K|V) slab, layer by layer


def cache_layers(cache: np.ndarray, nb: int, chunks):
    out, off = [], 0
    for c in chunks:
        out.append(cache[off:off + 2 * nb * c].reshape(2, nb, c))
        off += 2 * nb * c
    assert off == cache.size
    return out


def block_layers(row: np.ndarray, chunks):
    out, off = [], 0
    for c in chunks:
        out.append(row[off:off + 2 * c].reshape(2, c))
        off += 2 * c
    assert off == row.size
    return out


def _atoms(rng, n, bt, vocab):
    while True:
        a = rng.integers(0, vocab, size=(n, bt), dtype=np.int32)
        if len({r.tobytes() for r in a}) == n:
            return a


def _store(chunks, cap=64, bt=2):
    return OracleStore(len(chunks), 1, 1, bt, 1, cap, True, layer_chunk_bytes=chunks)


def _filled(rng, chunks):
    o = _store(chunks)
    atoms = _atoms(rng, 3, 2, 9)
    toks, offs = random_block_batch(rng, 16, atoms, 5, tail_p=0.0)
    R, maxb = len(offs) - 1, 5
    nb = R * maxb
    cache = rng.integers(0, 256, size=nb * o.block_bytes, dtype=np.uint8)
    rc, m, ids, created = o.insert(toks, offs, maxb)
    assert rc == ORC_OK
    o.scatter(ids, created, block_table_identity(R, maxb), cache, nb)
    return o, toks, offs, maxb, m, ids, created, cache


@pytest.mark.parametrize("chunks", [CHUNKS, [48] * 4, [16]])
def test_variable_slabs_scatter_then_gather(chunks):
    rng = np.random.default_rng(11)
    o, toks, offs, maxb, m, ids, created, cache = _filled(rng, chunks)
    assert o.block_bytes == 2 * sum(chunks)
    nb = (len(offs) - 1) * maxb
    cl = cache_layers(cache, nb, chunks)
    pool = o.pool()
    for r, b in np.argwhere(created != 0):
        row = block_layers(pool[ids[r, b]], chunks)
        for l in range(len(chunks)):
            np.testing.assert_array_equal(row[l], cl[l][:, r * maxb + b])
    # gather everything into a sentinel cache: matched blocks equal the pool, the rest untouched
    m2, ids2 = o.lookup(toks, offs, maxb)
    dst = np.full(cache.size, 0xA5, dtype=np.uint8)
    o.gather(ids2, m2, block_table_identity(len(m2), maxb), dst, nb)
    dl = cache_layers(dst, nb, chunks)
    for r in range(len(m2)):
        for b in range(maxb):
            for l in range(len(chunks)):
                got = dl[l][:, r * maxb + b]
                if b < m2[r]:
                    np.testing.assert_array_equal(got, block_layers(pool[ids2[r, b]], chunks)[l])
                else:
                    assert (got == 0xA5).all()


@pytest.mark.parametrize("l0,l1", [(0, 1), (1, 3), (4, 5), (0, 5), (2, 4)])
def test_layer_range_gather_writes_only_its_layers(l0, l1):
    rng = np.random.default_rng(20 + l0 * 7 + l1)
    o, toks, offs, maxb, m, ids, created, cache = _filled(rng, CHUNKS)
    nb = (len(offs) - 1) * maxb
    m2, ids2 = o.lookup(toks, offs, maxb)
    dst = np.full(cache.size, 0xA5, dtype=np.uint8)
    o.gather(ids2, m2, block_table_identity(len(m2), maxb), dst, nb, layers=(l0, l1))
    dl = cache_layers(dst, nb, CHUNKS)
    pool = o.pool()
    for r in range(len(m2)):
        for b in range(m2[r]):
            row = block_layers(pool[ids2[r, b]], CHUNKS)
            for l in range(len(CHUNKS)):
                got = dl[l][:, r * maxb + b]
                if l0 <= l < l1:
                    np.testing.assert_array_equal(got, row[l])
                else:
                    assert (got == 0xA5).all(), (l, l0, l1)


@pytest.mark.parametrize("l0,l1", [(0, 2), (3, 5), (2, 3)])
def test_layer_range_scatter_writes_only_its_layers(l0, l1):
    rng = np.random.default_rng(40 + l0)
    o = _store(CHUNKS)
    atoms = _atoms(rng, 3, 2, 9)
    toks, offs = random_block_batch(rng, 12, atoms, 4, tail_p=0.0)
    R, maxb = len(offs) - 1, 4
    nb = R * maxb
    cache = rng.integers(1, 256, size=nb * o.block_bytes, dtype=np.uint8)  # never 0
    rc, m, ids, created = o.insert(toks, offs, maxb)
    o.scatter(ids, created, block_table_identity(R, maxb), cache, nb, layers=(l0, l1))
    cl = cache_layers(cache, nb, CHUNKS)
    pool = o.pool()
    for r, b in np.argwhere(created != 0):
        row = block_layers(pool[ids[r, b]], CHUNKS)
        for l in range(len(CHUNKS)):
            if l0 <= l < l1:
                np.testing.assert_array_equal(row[l], cl[l][:, r * maxb + b])
            else:
                assert (row[l] == 0).all()  # the pool starts zeroed


def test_bad_layer_ranges_are_rejected():
    rng = np.random.default_rng(5)
    o, toks, offs, maxb, m, ids, created, cache = _filled(rng, CHUNKS)
    nb = (len(offs) - 1) * maxb
    for rng_ in ((2, 2), (3, 1), (-1, 2), (0, 6)):
        with pytest.raises(ValueError):
            o.gather(ids, m, block_table_identity(len(m), maxb), cache.copy(), nb, layers=rng_)
