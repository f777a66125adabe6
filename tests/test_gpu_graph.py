"""The hot path under HIP graph capture.

A lookup + gather captured once replays bit-exact against the oracle, three
times, with eager work of the program between the replays: inserts and
scatters that grow the store (so each replay must see the store as it is
then, not as it was at capture), sentinel fills of the outputs and
synchronisations. An insert + scatter captured once stores, replay after
replay, the new batch written into its captured buffers. The calls allocate nothing and wait for nothing once the
store's scratch has grown to the batch size, which a first eager call does;
later calls on the store must not need a larger copy scratch than the
captured one (a larger batch regrows it).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from tests.helpers import random_block_batch, block_table_identity

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2607_22648_amd import ptstore as P
    from tests.twin import Twin, host, to_dev, random_bytes


def _atoms(rng, n, bt, vocab):
    while True:
        a = rng.integers(0, vocab, size=(n, bt), dtype=np.int32)
        if len({r.tobytes() for r in a}) == n:
            return a


def _grow(t, rng, atoms, R, maxb, seed):
    toks, offs = random_block_batch(rng, R, atoms, maxb, tail_p=0.2)
    Ri = len(offs) - 1
    (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, maxb)
    t.scatter_random(ids, cr, rids, rcr, block_table_identity(Ri, maxb), seed=seed)


@pytest.mark.parametrize("chunks,R,maxb", [(None, 16, 8), ([32, 96, 16], 16, 8), (None, 160, 64)])
def test_captured_lookup_gather_replays(chunks, R, maxb):
    """16 x 8 entries take the one-workgroup list build; 160 x 64 (past its
    8,192 entries) the multi-kernel one, whose device-wide row table every
    replay must find empty and leave empty. Requests drawn from 5 atoms share
    their first blocks, so rows have several cache blocks."""
    rng = np.random.default_rng(41)
    bt_ = 4
    if chunks is None:
        t = Twin(3, 2, 8, bt_, 2000)
    else:
        t = Twin(len(chunks), 1, 1, bt_, 2000, layer_chunk_bytes=chunks)
    atoms = _atoms(rng, 5, bt_, 200)
    _grow(t, rng, atoms, 8, maxb, seed=1)
    toks, offs = random_block_batch(rng, R, atoms, maxb + 2, tail_p=0.3)
    tt, oo = to_dev(toks), to_dev(offs)
    bt_np = block_table_identity(R, maxb)
    bt = to_dev(bt_np)
    m = torch.empty(R, dtype=torch.int32, device="cuda")
    ids = torch.empty((R, maxb), dtype=torch.int32, device="cuda")
    n = R * maxb * t.shape.block_bytes
    cache = torch.full((n,), 0xA5, dtype=torch.uint8, device="cuda")
    t.gpu.lookup_gather(tt, oo, maxb, bt, cache, m=m, ids=ids)  # grows the scratch
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        t.gpu.lookup_gather(tt, oo, maxb, bt, cache, m=m, ids=ids)
    torch.cuda.synchronize()
    seen = set()
    for rep in range(3):
        cache.fill_(0xA5)
        m.fill_(-7)
        ids.fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        rm, rids = t.ref.lookup(toks, offs, maxb)
        rdst = np.full(n, 0xA5, dtype=np.uint8)
        t.ref.gather(rids, rm, bt_np, rdst, R * maxb)
        np.testing.assert_array_equal(host(m), rm, err_msg=f"replay {rep}: m")
        np.testing.assert_array_equal(host(ids), rids, err_msg=f"replay {rep}: ids")
        np.testing.assert_array_equal(host(cache), rdst, err_msg=f"replay {rep}: gathered bytes")
        seen.add(int(rm.sum()))
        # eager work between replays: the store grows (batches no larger
        # than the captured one, so the copy scratch stays where it was)
        _grow(t, rng, atoms, 8, maxb, seed=10 + rep)
    assert len(seen) > 1, "the replays should have seen the store grow"
    t.close()


def test_captured_insert_and_scatter_replays():
    """An insert and a scatter captured once, replayed with new token contents
    and new KV bytes written into the captured buffers between replays: each
    replay stores exactly what the oracle stores for that batch (ids,
    created flags, block metadata, pool bytes)."""
    rng = np.random.default_rng(43)
    bt_, R, maxb = 4, 8, 6
    t = Twin(2, 1, 8, bt_, 5000)
    atoms = _atoms(rng, 4, bt_, 300)

    def batch():  # every request exactly maxb blocks: the offsets stay the same
        return atoms[rng.integers(0, 4, size=(R, maxb))].reshape(-1).astype(np.int32)

    offs = (np.arange(R + 1, dtype=np.int64) * maxb * bt_)
    oo = to_dev(offs)
    tt = to_dev(batch())
    bt_np = block_table_identity(R, maxb)
    bt = to_dev(bt_np)
    n = R * maxb * t.shape.block_bytes
    cache = torch.empty(n, dtype=torch.uint8, device="cuda")
    m = torch.empty(R, dtype=torch.int32, device="cuda")
    ids = torch.empty((R, maxb), dtype=torch.int32, device="cuda")
    cr = torch.empty((R, maxb), dtype=torch.uint8, device="cuda")

    def eager_twin_step(toks, seed):
        cache.copy_(random_bytes(n, seed))
        rc, rm, rids, rcr = t.ref.insert(toks, offs, maxb)
        t.ref.scatter(rids, rcr, bt_np, host(cache), R * maxb)
        return rm, rids, rcr

    # warm-up: an eager insert + scatter of this size grows the scratch
    toks0 = host(tt)
    rm, rids, rcr = eager_twin_step(toks0, 100)
    P.ptstore_insert(t.gpu.h, tt, oo, maxb, m, ids, cr)
    P.ptstore_scatter(t.gpu.h, ids, cr, bt, cache, R * maxb)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(ids), rids)

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        P.ptstore_insert(t.gpu.h, tt, oo, maxb, m, ids, cr)
        P.ptstore_scatter(t.gpu.h, ids, cr, bt, cache, R * maxb)
    torch.cuda.synchronize()  # capture only records; nothing has run
    created_total = 0
    for rep in range(3):
        toks = batch()
        tt.copy_(to_dev(toks))
        rm, rids, rcr = eager_twin_step(toks, 200 + rep)
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(m), rm, err_msg=f"replay {rep}: m")
        np.testing.assert_array_equal(host(ids), rids, err_msg=f"replay {rep}: ids")
        np.testing.assert_array_equal(host(cr), rcr, err_msg=f"replay {rep}: created")
        created_total += int(rcr.sum())
    assert created_total > 0
    t.check_meta()
    t.check_pool()
    t.close()


def test_captured_evicting_insert_replays():
    """With PTSTORE_FLAG_EVICT: an insert and a scatter captured once, replayed
    on new batches with eager lookups (accesses) between the replays. Each
    replay protects its own batch's matches (the epoch advances on the
    device), so victims, ids, access counts, the clock and the pool follow
    the oracle replay after replay."""
    rng = np.random.default_rng(47)
    bt_, R, maxb = 4, 8, 6
    t = Twin(2, 1, 8, bt_, 60, flags=P.PTSTORE_FLAG_EVICT)
    atoms = _atoms(rng, 6, bt_, 300)

    def batch():
        return atoms[rng.integers(0, 6, size=(R, maxb))].reshape(-1).astype(np.int32)

    offs = (np.arange(R + 1, dtype=np.int64) * maxb * bt_)
    oo = to_dev(offs)
    tt = to_dev(batch())
    bt_np = block_table_identity(R, maxb)
    bt = to_dev(bt_np)
    n = R * maxb * t.shape.block_bytes
    cache = torch.empty(n, dtype=torch.uint8, device="cuda")
    m = torch.empty(R, dtype=torch.int32, device="cuda")
    ids = torch.empty((R, maxb), dtype=torch.int32, device="cuda")
    cr = torch.empty((R, maxb), dtype=torch.uint8, device="cuda")

    def eager_twin_step(toks, seed):
        cache.copy_(random_bytes(n, seed))
        rc, rm, rids, rcr = t.ref.insert(toks, offs, maxb)
        t.ref.scatter(rids, rcr, bt_np, host(cache), R * maxb)
        return rm, rids, rcr

    toks0 = host(tt)
    rm, rids, rcr = eager_twin_step(toks0, 300)
    P.ptstore_insert(t.gpu.h, tt, oo, maxb, m, ids, cr)
    P.ptstore_scatter(t.gpu.h, ids, cr, bt, cache, R * maxb)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(ids), rids)

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        P.ptstore_insert(t.gpu.h, tt, oo, maxb, m, ids, cr)
        P.ptstore_scatter(t.gpu.h, ids, cr, bt, cache, R * maxb)
    torch.cuda.synchronize()
    for rep in range(6):
        # eager lookups between replays count accesses on both sides
        lt, lo = random_block_batch(rng, 6, atoms, maxb, tail_p=0.2)
        t.lookup(lt, lo, maxb)
        toks = batch()
        tt.copy_(to_dev(toks))
        rm, rids, rcr = eager_twin_step(toks, 400 + rep)
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(m), rm, err_msg=f"replay {rep}: m")
        np.testing.assert_array_equal(host(ids), rids, err_msg=f"replay {rep}: ids")
        np.testing.assert_array_equal(host(cr), rcr, err_msg=f"replay {rep}: created")
        t.check_evict()
    assert t.gpu.stats()["evictions"] > 0
    t.check_meta()
    t.check_pool()
    t.close()


def test_capture_that_needs_more_scratch_is_refused():
    """A captured load or insert larger than any earlier call on the store
    would have to grow a scratch: the call returns INVALID and allocates
    nothing (the capture is not broken by an allocation or a wait), and the
    store works as before afterwards."""
    rng = np.random.default_rng(53)
    t = Twin(1, 1, 8, 4, 3000)
    atoms = _atoms(rng, 4, 4, 300)
    _grow(t, rng, atoms, 4, 6, seed=1)  # scratch for 4 requests x 6 blocks
    R, maxb = 64, 12
    toks, offs = random_block_batch(rng, R, atoms, maxb)
    tt, oo = to_dev(toks), to_dev(offs)
    bt = to_dev(block_table_identity(R, maxb))
    cache = torch.zeros(R * maxb * t.shape.block_bytes, dtype=torch.uint8, device="cuda")
    m = torch.empty(R, dtype=torch.int32, device="cuda")
    ids = torch.empty((R, maxb), dtype=torch.int32, device="cuda")
    cr = torch.empty((R, maxb), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    for call in ("gather", "insert"):
        g = torch.cuda.CUDAGraph()
        with pytest.raises(P.PTStoreError) as ei:
            with torch.cuda.graph(g):
                m.fill_(0)  # the graph is not empty when the refused call ends it
                if call == "gather":
                    P.ptstore_gather(t.gpu.h, ids, m, bt, cache, R * maxb)
                else:
                    P.ptstore_insert(t.gpu.h, tt, oo, maxb, m, ids, cr)
        assert ei.value.code == P.PTSTORE_ERR_INVALID
        assert "captur" in P.ptstore_last_error()
        torch.cuda.synchronize()
    # the waiting insert is refused under capture whatever its size
    one = torch.tensor([0, 16], dtype=torch.int64, device="cuda")  # a request of 4 blocks
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with pytest.raises(P.PTStoreError) as ei:
        with torch.cuda.graph(g):
            m.fill_(0)
            P.ptstore_insert_sync(t.gpu.h, tt[:16], one, 4, m, ids, cr)
    assert ei.value.code == P.PTSTORE_ERR_INVALID and "captured" in P.ptstore_last_error()
    torch.cuda.synchronize()
    # eagerly the same calls grow the scratch and match the oracle
    t.lookup_gather(toks, offs, maxb, block_table_identity(R, maxb), R * maxb)
    (_, ids2, cr2), (_, _, rids, rcr) = t.insert(toks, offs, maxb)
    t.check_meta()
    t.close()
