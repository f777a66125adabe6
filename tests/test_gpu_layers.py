"""Layer ranges and per-layer slab sizes: GPU library vs the CPU oracle.

Section 4.1 (transfers overlap computation) and Section 5 (clients read and
write subsets of tensors; prefixes combine tensors of variable sizes): a
gather or scatter may move a range of layers, and each layer may have its
own slab size. Every byte of the caches and of the pool is compared with the
oracle, which restates the layouts layer after layer.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from tests.helpers import random_block_batch, block_table_identity

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2607_22648_amd import ptstore as P
    from tests.twin import Twin, host, to_dev

CHUNKS = [32, 96, 16, 64, 48]  # per-layer slab bytes (multiples of 16)


def _atoms(rng, n, bt, vocab):
    while True:
        a = rng.integers(0, vocab, size=(n, bt), dtype=np.int32)
        if len({r.tobytes() for r in a}) == n:
            return a


def _twin(chunks, cap=64, bt=2, **kw):
    if chunks is None:
        return Twin(5, 2, 8, bt, cap, **kw)  # uniform: 5 layers of 2 x 2 x 8 x 2 bytes
    return Twin(len(chunks), 1, 1, bt, cap, layer_chunk_bytes=chunks, **kw)


def _fill(t, rng, rounds=4, maxb=6, seed=0):
    atoms = _atoms(rng, 4, t.shape.block_tokens, 50)
    for i in range(rounds):
        toks, offs = random_block_batch(rng, 10, atoms, maxb, tail_p=0.2)
        R = len(offs) - 1
        (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, maxb)
        t.scatter_random(ids, cr, rids, rcr, block_table_identity(R, maxb), seed=seed + i)
    return atoms


@pytest.mark.parametrize("chunks", [CHUNKS, None])
def test_full_gather_with_variable_slabs(chunks):
    rng = np.random.default_rng(1)
    t = _twin(chunks)
    atoms = _fill(t, rng)
    t.check_pool()
    toks, offs = random_block_batch(rng, 12, atoms, 6, tail_p=0.3)
    R = len(offs) - 1
    t.lookup_gather(toks, offs, 6, block_table_identity(R, 6), R * 6)
    t.close()


@pytest.mark.parametrize("chunks", [CHUNKS, None])
@pytest.mark.parametrize("rng_", [(0, 1), (1, 3), (4, 5), (0, 5), (2, 4)])
def test_layer_range_gather(chunks, rng_):
    rng = np.random.default_rng(2)
    t = _twin(chunks)
    atoms = _fill(t, rng)
    toks, offs = random_block_batch(rng, 12, atoms, 6, tail_p=0.3)
    R = len(offs) - 1
    (m, ids), (rm, rids) = t.lookup(toks, offs, 6)
    t.gather_layers(m, ids, rm, rids, block_table_identity(R, 6), R * 6, rng_)
    t.close()


@pytest.mark.parametrize("chunks", [CHUNKS, None])
def test_per_layer_gathers_equal_one_full_gather(chunks):
    """Layer after layer into one cache (what a pipelined prefill does) gives
    the full gather's bytes."""
    rng = np.random.default_rng(3)
    t = _twin(chunks)
    atoms = _fill(t, rng)
    toks, offs = random_block_batch(rng, 12, atoms, 6, tail_p=0.3)
    R = len(offs) - 1
    (m, ids), (rm, rids) = t.lookup(toks, offs, 6)
    bt = block_table_identity(R, 6)
    dst, rdst = None, None
    for l in range(t.shape.layers):
        dst, rdst = t.gather_layers(m, ids, rm, rids, bt, R * 6, (l, l + 1), dst, rdst)
    full = torch.full_like(dst, 0xA5)
    t.gpu.gather(ids, m, to_dev(bt), full)
    torch.cuda.synchronize()
    assert torch.equal(full, dst)
    t.close()


@pytest.mark.parametrize("chunks", [CHUNKS, None])
def test_layer_range_scatters(chunks):
    """New blocks written in two layer ranges from two different caches."""
    rng = np.random.default_rng(4)
    t = _twin(chunks)
    atoms = _atoms(rng, 4, 2, 50)
    for i in range(3):
        toks, offs = random_block_batch(rng, 10, atoms, 6, tail_p=0.2)
        R = len(offs) - 1
        (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, 6)
        bt = block_table_identity(R, 6)
        t.scatter_random(ids, cr, rids, rcr, bt, seed=10 + i, layers=(0, 2))
        t.scatter_random(ids, cr, rids, rcr, bt, seed=20 + i, layers=(2, t.shape.layers))
    t.check_pool()
    t.close()


@pytest.mark.parametrize("cpg,threads", [(3, 256), (1, 64), (64, 1024)])
def test_layer_ranges_with_other_copy_shapes(cpg, threads):
    rng = np.random.default_rng(5)
    t = _twin(CHUNKS)
    t.gpu.set_copy_shape(cpg, threads, 0)
    atoms = _fill(t, rng)
    toks, offs = random_block_batch(rng, 12, atoms, 6, tail_p=0.3)
    R = len(offs) - 1
    (m, ids), (rm, rids) = t.lookup(toks, offs, 6)
    for rng_ in ((1, 4), (0, 5)):
        t.gather_layers(m, ids, rm, rids, block_table_identity(R, 6), R * 6, rng_)
    t.close()


def test_variable_slabs_with_host_tier_and_replicas():
    rng = np.random.default_rng(6)
    t = _twin(CHUNKS, cap=8, flags=P.PTSTORE_FLAG_EVICT, host_blocks=24, replica_blocks=4)
    atoms = _atoms(rng, 5, 2, 50)
    for i in range(20):
        toks, offs = random_block_batch(rng, 8, atoms, 6, tail_p=0.2)
        R = len(offs) - 1
        if i % 4 == 3:
            t.gpu.replicate()
            t.check_replicas()
        elif i % 2:
            t.lookup_gather(toks, offs, 6, block_table_identity(R, 6), R * 6)
        else:
            (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, 6)
            t.scatter_random(ids, cr, rids, rcr, block_table_identity(R, 6), seed=30 + i)
    t.check_pool()
    t.check_evict()
    assert t.gpu.stats()["replica_copies"] > 0
    t.close()


def test_bad_layer_ranges_and_sizes_are_rejected():
    t = _twin(CHUNKS)
    ids = torch.zeros((1, 2), dtype=torch.int32, device="cuda")
    m = torch.zeros(1, dtype=torch.int32, device="cuda")
    bt = torch.zeros((1, 2), dtype=torch.int32, device="cuda")
    cache = torch.zeros(2 * t.shape.block_bytes, dtype=torch.uint8, device="cuda")
    for rng_ in ((2, 2), (3, 1), (-1, 2), (0, 6)):
        with pytest.raises(P.PTStoreError):
            t.gpu.gather(ids, m, bt, cache, layers=rng_)
    t.close()
    for bad in ([32, 8], [32, 0], [32, -16]):
        with pytest.raises(P.PTStoreError):
            P.PrefixStore(P.StoreShape(2, 1, 1, 2, 1, tuple(bad)), 8)


@pytest.mark.parametrize("chunks", [CHUNKS, None])
def test_prepared_per_layer_gather(chunks):
    """The block list built once, then one copy per layer: the same bytes as
    layer-range gathers; any other call discards the list."""
    rng = np.random.default_rng(7)
    t = _twin(chunks)
    atoms = _fill(t, rng)
    toks, offs = random_block_batch(rng, 12, atoms, 6, tail_p=0.3)
    R = len(offs) - 1
    (m, ids), (rm, rids) = t.lookup(toks, offs, 6)
    bt = block_table_identity(R, 6)
    n = R * 6 * t.shape.block_bytes
    dst = torch.full((n,), 0xA5, dtype=torch.uint8, device="cuda")
    t.gpu.gather_prepare(ids, m, to_dev(bt), dst)
    for l in range(t.shape.layers):
        t.gpu.gather_prepared(dst, (l, l + 1))
    rdst = np.full(n, 0xA5, dtype=np.uint8)
    t.ref.gather(rids, rm, bt, rdst, R * 6)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(dst), rdst)
    # still valid for another range, then discarded by a gather
    t.gpu.gather_prepared(dst, (0, t.shape.layers))
    t.gpu.gather(ids, m, to_dev(bt), dst)
    with pytest.raises(P.PTStoreError):
        t.gpu.gather_prepared(dst, (0, 1))
    # discarded by an insert; a cache of another size is refused
    t.gpu.gather_prepare(ids, m, to_dev(bt), dst)
    with pytest.raises(P.PTStoreError):
        t.gpu.gather_prepared(dst[: n - t.shape.block_bytes], (0, 1))
    t.insert(toks, offs, 6)
    with pytest.raises(P.PTStoreError):
        t.gpu.gather_prepared(dst, (0, 1))
    t.close()


def test_large_variable_slabs_span_several_units():
    """Blocks of per-layer slabs larger than one span-copy unit (256 KiB), with
    layer boundaries inside units, gathered whole and by layer ranges, and
    scattered by layer ranges."""
    chunks = [32 << 10, 8 << 10, 96 << 10, 16, 48 << 10, 112]  # blocks of 368.3 KiB
    rng = np.random.default_rng(31)
    t = Twin(len(chunks), 1, 1, 2, 40, layer_chunk_bytes=chunks)
    atoms = _atoms(rng, 4, 2, 50)
    for i in range(3):
        toks, offs = random_block_batch(rng, 6, atoms, 5, tail_p=0.2)
        R = len(offs) - 1
        (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, 5)
        t.scatter_random(ids, cr, rids, rcr, block_table_identity(R, 5), seed=70 + i,
                         layers=(0, 3) if i == 1 else None)
        if i == 1:
            t.scatter_random(ids, cr, rids, rcr, block_table_identity(R, 5), seed=80, layers=(3, 6))
    t.check_pool()
    toks, offs = random_block_batch(rng, 8, atoms, 5, tail_p=0.3)
    R = len(offs) - 1
    (m, ids, _), (rm, rids, _) = t.lookup_gather(toks, offs, 5, block_table_identity(R, 5), R * 5)
    for layers in ((0, 6), (2, 3), (1, 5), (5, 6)):
        t.gather_layers(m, ids, rm, rids, block_table_identity(R, 5), R * 5, layers)
    t.close()


def test_variable_slabs_beyond_the_gather_grid_cap():
    """More span units than the gather launches workgroups (20,000 requests x
    64 blocks, one unit each): workgroups take a second unit one grid on."""
    rng = np.random.default_rng(14)
    R, maxb = 20_000, 64
    toks = rng.integers(0, 32000, size=R * maxb * 2, dtype=np.int32)
    offs = np.arange(R + 1, dtype=np.int64) * (maxb * 2)
    t = Twin(2, 1, 1, 2, R * maxb, layer_chunk_bytes=[16, 32])
    (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, maxb)
    t.scatter_random(ids, cr, rids, rcr, block_table_identity(R, maxb), seed=19)
    t.check_pool()
    t.lookup_gather(toks, offs, maxb, block_table_identity(R, maxb), R * maxb)
    t.close()


@pytest.mark.parametrize("prepared", [False, True])
def test_narrow_layer_ranges_with_shared_rows(prepared):
    """A layer range of at most 4 chunks per block (one or two layers) moves
    as one copy unit per descriptor, a wider one as the store's own units:
    ranges of 1, 2 and 3 layers at every start, through a gather per range
    or one prepared list, with many requests sharing rows (slices of several
    cache blocks), against the oracle's range gathers into one cache."""
    rng = np.random.default_rng(31 + prepared)
    t = Twin(7, 2, 8, 2, 96)  # uniform: 14 chunks per block, one chunk per unit
    atoms = _fill(t, rng)
    # 40 requests drawn from a few atoms share most of their blocks
    toks, offs = random_block_batch(rng, 40, atoms, 6, tail_p=0.3)
    R = len(offs) - 1
    (m, ids), (rm, rids) = t.lookup(toks, offs, 6)
    bt = block_table_identity(R, 6)
    n = R * 6 * t.shape.block_bytes
    dst = torch.full((n,), 0xA5, dtype=torch.uint8, device="cuda")
    rdst = np.full(n, 0xA5, dtype=np.uint8)
    if prepared:
        t.gpu.gather_prepare(ids, m, to_dev(bt), dst)
    L = t.shape.layers
    for width in (1, 2, 3):
        for l0 in range(0, L - width + 1):
            rng_ = (l0, l0 + width)
            if prepared:
                t.gpu.gather_prepared(dst, rng_)
            else:
                t.gpu.gather(ids, m, to_dev(bt), dst, layers=rng_)
            t.ref.gather(rids, rm, bt, rdst, R * 6, layers=rng_)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(host(dst), rdst, err_msg=f"layers {rng_}")
    rows = host(ids)[np.arange(6)[None, :] < host(m)[:, None]]
    assert np.bincount(rows).max() > 1  # some rows have several cache blocks
    t.close()
