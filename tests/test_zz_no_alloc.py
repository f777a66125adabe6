"""The allocation-free lookup + gather against ptstore_lookup_gather, through the C ABI.

ptstore_lookup_gather_noalloc keeps its descriptor list in the library's one
static device array instead of store-owned scratch. Each case calls it twice
in a row, the second time with a smaller batch (the array then still holds
the first call's list), and compares m, ids and every cache byte with what
ptstore_lookup_gather gives on the same inputs; that call is itself checked
against the oracle by the twin. The bar is bit-exact.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from workloads import synth

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2607_22648_amd import ptstore as P
    from tests.twin import Twin, to_dev, host, DEV

SENTINEL = 0xA5


def _stored_tiny(n_requests=64):
    w = synth.build("tiny", n_requests=n_requests)
    t = Twin.for_shape(w.shape, 4096)
    st, so = w.store_batch()
    R, maxb = len(so) - 1, w.passage_blocks
    (_, ids, cr), (_, _, rids, rcr) = t.insert(st, so, maxb)
    bt = np.arange(R * maxb, dtype=np.int32).reshape(R, maxb)
    t.scatter_random(ids, cr, rids, rcr, bt, seed=11)
    return w, t


def _compare(t, toks, offs, maxb, bt, nb):
    """Both entry points on the same inputs; returns matched blocks."""
    (m1, ids1, dst1), (rm, _, _) = t.lookup_gather(toks, offs, maxb, bt, nb)
    R = len(offs) - 1
    m2 = torch.full((R,), -7, dtype=torch.int32, device=DEV)
    ids2 = torch.full((R, maxb), -7, dtype=torch.int32, device=DEV)
    dst2 = torch.full((nb * t.shape.block_bytes,), SENTINEL, dtype=torch.uint8, device=DEV)
    t.gpu.lookup_gather_noalloc(to_dev(toks), to_dev(offs), maxb, to_dev(bt), dst2, m2, ids2)
    torch.cuda.synchronize()
    assert torch.equal(m1, m2), "m differs from ptstore_lookup_gather"
    assert torch.equal(ids1, ids2), "ids differ from ptstore_lookup_gather"
    if not torch.equal(dst1, dst2):
        bad = torch.nonzero(dst1 != dst2).flatten()[:8].tolist()
        raise AssertionError(f"cache bytes differ from ptstore_lookup_gather, first at {bad}")
    return int(rm.sum())


def test_noalloc_matches_lookup_gather_twice_smaller_second():
    w, t = _stored_tiny()
    R, maxb = w.n_requests, w.max_blocks
    bt = np.arange(R * maxb, dtype=np.int32).reshape(R, maxb)
    got = _compare(t, w.tokens, w.offsets, maxb, bt, R * maxb)
    assert got > 0
    # second call: fewer requests, fewer blocks each, a shuffled block table
    # with holes and spare cache blocks
    rng = np.random.default_rng(3)
    lo, hi, maxb2 = 5, 14, 40
    toks = w.tokens[w.offsets[lo]:w.offsets[hi]]
    offs = (w.offsets[lo:hi + 1] - w.offsets[lo]).astype(np.int64)
    R2 = hi - lo
    nb2 = R2 * maxb2 + 7
    bt2 = rng.permutation(nb2)[:R2 * maxb2].astype(np.int32).reshape(R2, maxb2)
    bt2[rng.random(bt2.shape) < 0.2] = -1
    got2 = _compare(t, toks, offs, maxb2, bt2, nb2)
    assert 0 < got2 < got
    t.close()


def test_noalloc_long_requests_twice_smaller_second():
    """Matches of several 64-block windows (the workgroup-per-request lookup):
    lookups re-read stored sequences cut at a random depth, then diverge."""
    rng = np.random.default_rng(21)
    t = Twin(2, 2, 16, 16, 20_000)
    stored = []
    for k in range(3):
        seqs = [rng.integers(0, 32000, size=16 * int(rng.integers(150, 300)), dtype=np.int32)
                for _ in range(24)]
        toks, offs = synth.concat_requests(seqs)
        R = len(seqs)
        (_, ids, cr), (_, _, rids, rcr) = t.insert(toks, offs, 300)
        t.scatter_random(ids, cr, rids, rcr, np.arange(R * 300, dtype=np.int32).reshape(R, 300),
                         seed=100 + k)
        stored += seqs
    for R, maxb in ((48, 300), (17, 130)):
        reqs = []
        for _ in range(R):
            s = stored[int(rng.integers(len(stored)))]
            cut = 16 * int(rng.integers(0, len(s) // 16 + 1))
            tail = rng.integers(0, 32000, size=int(rng.integers(0, 40 * 16)), dtype=np.int32)
            reqs.append(np.concatenate([s[:cut], tail]))
        toks, offs = synth.concat_requests(reqs)
        bt = np.arange(R * maxb, dtype=np.int32).reshape(R, maxb)
        assert _compare(t, toks, offs, maxb, bt, R * maxb) > 64 * R // 4
    t.close()


def test_noalloc_allocates_nothing():
    """Device memory free before and after a no-alloc call larger than any
    earlier batch of the store is the same."""
    w, t = _stored_tiny()
    small = 4
    bt_s = np.arange(small * w.max_blocks, dtype=np.int32).reshape(small, w.max_blocks)
    t.lookup_gather(w.tokens[:w.offsets[small]], w.offsets[:small + 1], w.max_blocks, bt_s,
                    small * w.max_blocks)  # loads the kernels; the store's own list stays small
    R, maxb = w.n_requests, w.max_blocks
    toks, offs = to_dev(w.tokens), to_dev(w.offsets)
    bt = to_dev(np.arange(R * maxb, dtype=np.int32).reshape(R, maxb))
    cache = torch.full((R * maxb * t.shape.block_bytes,), SENTINEL, dtype=torch.uint8, device=DEV)
    m = torch.empty(R, dtype=torch.int32, device=DEV)
    ids = torch.empty((R, maxb), dtype=torch.int32, device=DEV)
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    for _ in range(3):
        t.gpu.lookup_gather_noalloc(toks, offs, maxb, bt, cache, m, ids)
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    assert free1 == free0, f"device memory free changed by {free0 - free1} bytes"
    rm, rids = t.ref.lookup(w.tokens, w.offsets, maxb)
    np.testing.assert_array_equal(host(m), rm)
    np.testing.assert_array_equal(host(ids), rids)
    t.close()


def test_noalloc_refuses_a_batch_over_its_limit():
    w, t = _stored_tiny(n_requests=4)
    R, maxb = 2048, 1024  # 2^21 entries > PTSTORE_NOALLOC_MAX_ENTRIES
    assert R * maxb > P.PTSTORE_NOALLOC_MAX_ENTRIES
    offs = to_dev(np.zeros(R + 1, dtype=np.int64))
    toks = to_dev(np.zeros(16, dtype=np.int32))
    m = torch.empty(R, dtype=torch.int32, device=DEV)
    ids = torch.empty((R, maxb), dtype=torch.int32, device=DEV)
    bt = torch.zeros((R, maxb), dtype=torch.int32, device=DEV)
    cache = torch.empty(t.shape.block_bytes, dtype=torch.uint8, device=DEV)
    with pytest.raises(P.PTStoreError) as ei:
        t.gpu.lookup_gather_noalloc(toks, offs, maxb, bt, cache, m, ids)
    assert ei.value.code == P.PTSTORE_ERR_INVALID
    assert "PTSTORE_NOALLOC_MAX_ENTRIES" in P.ptstore_last_error()
    t.close()
