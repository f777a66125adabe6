"""GPU library vs the CPU oracle, element by element, through the C ABI.

Sizes here are small enough for the oracle to finish in seconds but span
several 64-block windows, several copy groups and ragged tails. The bar is
bit-exact: all outputs are integers, indices and copied bytes.
"""
from __future__ import annotations

import ctypes as C

import numpy as np
import pytest
import torch

from workloads import synth
from tests.helpers import load_golden, spell_batch, random_block_batch, block_table_identity

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2607_22648_amd import ptstore as P
    from tests.twin import Twin, to_dev, host, DEV


def _atoms(rng, n, bt, vocab, shared_head=False):
    while True:
        a = rng.integers(0, vocab, size=(n, bt), dtype=np.int32)
        if shared_head:
            a[:, :-1] = a[0, :-1]
        if len({r.tobytes() for r in a}) == n:
            return a


# ---------------------------------------------------------------------------
# golden example and random tries
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("case", load_golden("incremental_ids.json")["cases"], ids=lambda c: c["name"])
def test_golden_example(case):
    g = load_golden("incremental_ids.json")
    t = Twin(1, 1, 8, g["block_tokens"], case["capacity"])
    toks, offs = spell_batch(case["insert"], g["blocks"])
    (m, ids, cr), _ = t.insert(toks, offs, case["insert_max_blocks"])
    e = case["expect_insert"]
    assert host(m).tolist() == e["m"] and host(ids).tolist() == e["ids"]
    assert host(cr).tolist() == e["created"]
    assert t.gpu.stats()["blocks_stored"] == e["count"]
    assert (t.gpu.stats()["full_events"] > 0) == e["rc_full"]
    toks, offs = spell_batch(case["lookup"], g["blocks"])
    (m, ids), _ = t.lookup(toks, offs, case["lookup_max_blocks"])
    assert host(m).tolist() == case["expect_lookup"]["m"]
    assert host(ids).tolist() == case["expect_lookup"]["ids"]
    t.close()


@pytest.mark.parametrize("bt", [16, 2, 5, 1, 63, 64])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_random_tries(seed, bt):
    rng = np.random.default_rng(100 + seed)
    atoms = _atoms(rng, 3, bt, 4, shared_head=(seed == 2))
    maxb = 70  # crosses a 64-block window
    cap = [10_000, 150, 40][seed]
    t = Twin(1, 1, 8, bt, cap)
    for rnd in range(4):
        toks, offs = random_block_batch(rng, 48, atoms, 80)
        t.insert(toks, offs, maxb)
        toks, offs = random_block_batch(rng, 48, atoms, 90)
        t.lookup(toks, offs, maxb)
    t.check_meta()
    assert t.gpu.stats()["insert_fallbacks"] == 0  # 61-bit keys: the parallel claim held
    t.close()


def test_weak_hash_gives_same_results():
    """Index keys masked to 8 bits: collisions everywhere, same outputs."""
    rng = np.random.default_rng(5)
    atoms = _atoms(rng, 4, 16, 6)
    t = Twin(1, 1, 8, 16, 3000, flags=P.PTSTORE_FLAG_WEAK_HASH | P.PTSTORE_FLAG_COUNTERS)
    for _ in range(3):
        toks, offs = random_block_batch(rng, 64, atoms, 40)
        t.insert(toks, offs, 40)
        toks, offs = random_block_batch(rng, 64, atoms, 45)
        t.lookup(toks, offs, 40)
    st = t.gpu.stats()
    assert st["token_compares"] > st["probes"] // 4  # collisions really happened
    assert st["insert_fallbacks"] >= 1  # and the inserts took the exact path
    t.close()


@pytest.mark.parametrize("weak_hash", [False, True])
def test_one_request_blocks_sharing_a_batch_entry(weak_hash):
    """An insert names each new block in its batch table by chained key and
    depth. The weak test tags keep only the depth's parity; with 8-bit index
    keys on top, blocks of a single request at different depths then share
    entries. The claim records each entry's depth, verification finds the
    sharing and the insert takes its exact path, with the sequential
    results. One request per call, so no other request can be what raises
    the flag. With full keys the weak tags alone share nothing: the parallel
    claim holds."""
    rng = np.random.default_rng(23)
    flags = P.PTSTORE_FLAG_WEAK_TAGS | (P.PTSTORE_FLAG_WEAK_HASH if weak_hash else 0)
    t = Twin(1, 1, 8, 16, 5000, flags=flags)
    seqs = []
    for i in range(8):
        if i % 2 == 0 or not seqs:  # fresh tokens: 48 new blocks
            s = rng.integers(0, 32000, size=48 * 16, dtype=np.int32)
        else:  # an earlier sequence cut at a block boundary, then new blocks
            base = seqs[int(rng.integers(0, len(seqs)))]
            cut = int(rng.integers(1, 40)) * 16
            s = np.concatenate([base[:cut], rng.integers(0, 32000, size=24 * 16, dtype=np.int32)])
        seqs.append(s)
        offs = np.array([0, s.size], dtype=np.int64)
        t.insert(s, offs, 64)
        t.lookup(s, offs, 64)
    toks = np.concatenate(seqs)
    offs = np.concatenate([[0], np.cumsum([x.size for x in seqs])]).astype(np.int64)
    (m, _), (rm, _) = t.lookup(toks, offs, 64)
    assert (rm == offs[1:] // 16 - offs[:-1] // 16).all()  # every sequence stored whole
    t.check_meta()
    fb = t.gpu.stats()["insert_fallbacks"]
    if weak_hash:
        assert fb >= 1  # single-request inserts shared entries across depths
    else:
        assert fb == 0
    t.close()


@pytest.mark.parametrize("bt", [4, 16])
@pytest.mark.parametrize("maxb", [130, 300, 700])
def test_weak_hash_long_requests(maxb, bt):
    """Key collisions in requests of several windows, looked up a workgroup
    per request with windows in parallel (4, 8 and 16 waves). Three distinct
    blocks make up every request, so equal blocks under different parents
    abound, and 8-bit index keys make them collide often: a key hit may hold
    other tokens, or the right tokens under another parent; either way the
    lane probes on, at any lane of a window, and the result is the
    sequential one. 16-token blocks take the kernels' LDS-staged path, with
    stored rows compared four lanes to a row; 4-token blocks the generic
    one."""
    rng = np.random.default_rng(maxb + bt)
    atoms = _atoms(rng, 3, bt, 3)
    t = Twin(1, 1, 8, bt, 100_000, flags=P.PTSTORE_FLAG_WEAK_HASH | P.PTSTORE_FLAG_COUNTERS)
    for _ in range(3):
        toks, offs = random_block_batch(rng, 24, atoms, maxb + 20)
        t.insert(toks, offs, maxb)
        toks, offs = random_block_batch(rng, 24, atoms, maxb + 20)
        t.lookup(toks, offs, maxb)
    # lookups of stored sequences themselves: full matches through every window
    toks, offs = random_block_batch(rng, 12, atoms, maxb, tail_p=0.0)
    t.insert(toks, offs, maxb)
    (m, ids), (rm, rids) = t.lookup(toks, offs, maxb)
    assert (rm == np.diff(offs) // bt).all()
    t.check_meta()
    t.close()


def test_counters_switch_at_run_time():
    """ptstore_set_counters turns counting on and off between calls; the
    outputs do not change, and a lookup counts one probe or more per examined
    block only while counting is on."""
    rng = np.random.default_rng(8)
    atoms = _atoms(rng, 3, 16, 5)
    s = P.PrefixStore(P.StoreShape(1, 1, 8, 16), 5000)
    toks, offs = random_block_batch(rng, 40, atoms, 90)
    s.insert(to_dev(toks), to_dev(offs), 90)
    lk = [to_dev(a) for a in random_block_batch(rng, 60, atoms, 100)]
    outs, probes = [], []
    for on in (False, True, False):
        s.set_counters(on)
        s.reset_counters()
        m, ids = s.lookup(lk[0], lk[1], 100)
        outs.append((host(m), host(ids)))
        st = s.stats()
        probes.append((st["probes"], st["token_compares"]))
    s.close()
    examined = int(np.minimum(np.diff(host(lk[1])) // 16, 100).sum())
    assert probes[0] == (0, 0) and probes[2] == (0, 0)
    assert probes[1][0] >= examined and probes[1][1] >= int(outs[1][0].sum())
    for m, ids in outs[1:]:
        np.testing.assert_array_equal(m, outs[0][0])
        np.testing.assert_array_equal(ids, outs[0][1])


def test_timing_switch_at_run_time():
    """ptstore_set_timing turns the per-kernel events on and off between
    calls: only the calls made while it is on are reported, pairs recorded
    before a switch-off stay until read, and the outputs do not change."""
    rng = np.random.default_rng(9)
    atoms = _atoms(rng, 3, 16, 5)
    s = P.PrefixStore(P.StoreShape(1, 1, 8, 16), 5000)  # starts with timing off
    toks, offs = random_block_batch(rng, 40, atoms, 90)
    s.insert(to_dev(toks), to_dev(offs), 90)
    lk = [to_dev(a) for a in random_block_batch(rng, 60, atoms, 100)]
    ref = [host(a) for a in s.lookup(lk[0], lk[1], 100)]
    assert s.kernel_times(P.KIND_LOOKUP)[1] == 0
    s.set_timing(True)
    for _ in range(3):
        s.lookup(lk[0], lk[1], 100)
    s.set_timing(False)
    for _ in range(2):
        m, ids = s.lookup(lk[0], lk[1], 100)
    ms, n = s.kernel_times(P.KIND_LOOKUP)
    assert n == 3 and ms > 0
    assert s.kernel_times(P.KIND_LOOKUP)[1] == 0  # read once
    np.testing.assert_array_equal(host(m), ref[0])
    np.testing.assert_array_equal(host(ids), ref[1])
    s.close()


def test_timing_of_some_kinds_only():
    """ptstore_set_timing_kinds records the kinds whose bit is set and no
    other: with kinds = 1 a fused lookup + gather reports its copy kernel
    alone. A bit above the last kind is refused."""
    rng = np.random.default_rng(19)
    atoms = _atoms(rng, 3, 16, 5)
    sh = P.StoreShape(2, 1, 8, 16)
    s = P.PrefixStore(sh, 3000)
    toks, offs = random_block_batch(rng, 30, atoms, 40)
    m0, ids0, cr = s.insert(to_dev(toks), to_dev(offs), 40)
    R = len(offs) - 1
    bt = to_dev(block_table_identity(R, 40))
    src = torch.randint(0, 256, (R * 40 * sh.block_bytes,), dtype=torch.uint8, device=DEV)
    s.scatter(ids0, cr, bt, src)
    cache = torch.zeros_like(src)
    s.set_timing_kinds(1 << P.KIND_GATHER)
    for _ in range(2):
        m, ids = s.lookup_gather(to_dev(toks), to_dev(offs), 40, bt, cache)
    torch.cuda.synchronize()
    g_ms, g_n = s.kernel_times(P.KIND_GATHER)
    assert g_n == 2 and g_ms > 0
    for k in (P.KIND_LOOKUP, P.KIND_SELECT, P.KIND_INSERT, P.KIND_SCATTER):
        assert s.kernel_times(k)[1] == 0
    s.set_timing_kinds(1 << P.KIND_LOOKUP | 1 << P.KIND_SELECT)
    s.lookup_gather(to_dev(toks), to_dev(offs), 40, bt, cache, m=m, ids=ids)
    assert s.kernel_times(P.KIND_GATHER)[1] == 0
    assert s.kernel_times(P.KIND_LOOKUP)[1] == 1 and s.kernel_times(P.KIND_SELECT)[1] == 1
    with pytest.raises(P.PTStoreError) as ei:
        s.set_timing_kinds(1 << 7)
    assert ei.value.code == P.PTSTORE_ERR_INVALID
    # the outputs: the ids the insert returned, and the same bytes as a load
    # with every event off
    s.set_timing_kinds(0)
    cache2 = torch.zeros_like(src)
    m2, ids2 = s.lookup_gather(to_dev(toks), to_dev(offs), 40, bt, cache2)
    assert s.kernel_times(P.KIND_GATHER)[1] == 0
    np.testing.assert_array_equal(host(m), host(m0))
    np.testing.assert_array_equal(host(ids), host(ids0))
    np.testing.assert_array_equal(host(m2), host(m0))
    np.testing.assert_array_equal(host(ids2), host(ids0))
    np.testing.assert_array_equal(host(cache), host(cache2))
    assert int(host(m).sum()) > 0
    s.close()


def test_hash_seed_does_not_change_results():
    rng = np.random.default_rng(6)
    atoms = _atoms(rng, 3, 16, 5)
    ins = [random_block_batch(rng, 40, atoms, 30) for _ in range(3)]
    lk = random_block_batch(rng, 80, atoms, 35)
    outs = []
    for seed in (1, 2, 0xDEADBEEF):
        s = P.PrefixStore(P.StoreShape(1, 1, 8, 16), 5000, hash_seed=seed)
        for toks, offs in ins:
            s.insert(to_dev(toks), to_dev(offs), 30)
        m, ids = s.lookup(to_dev(lk[0]), to_dev(lk[1]), 30)
        outs.append((host(m), host(ids)))
        s.close()
    for m, ids in outs[1:]:
        np.testing.assert_array_equal(m, outs[0][0])
        np.testing.assert_array_equal(ids, outs[0][1])


def test_insert_is_deterministic_across_copy_shapes():
    rng = np.random.default_rng(8)
    atoms = _atoms(rng, 2, 16, 3)
    toks, offs = random_block_batch(rng, 300, atoms, 20)
    res = []
    for shape in ((8, 256), (1, 64), (3, 1024)):
        s = P.PrefixStore(P.StoreShape(2, 1, 8, 16), 8000, hash_seed=shape[0])
        s.set_copy_shape(*shape)
        m, ids, cr = s.insert(to_dev(toks), to_dev(offs), 20)
        res.append((host(m), host(ids), host(cr)))
        s.close()
    for r in res[1:]:
        for a, b in zip(r, res[0]):
            np.testing.assert_array_equal(a, b)


# ---------------------------------------------------------------------------
# payload movement
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("cpg,threads,grid", [(8, 256, 0), (1, 64, 0), (5, 512, 7), (64, 1024, 0),
                                             (1, 1024, 1), (2, 128, 3000)])
def test_scatter_then_gather_bytes(cpg, threads, grid):
    rng = np.random.default_rng(9)
    L, H, D, bt = 3, 2, 4, 16  # chunk = 2*16*4*2 = 256 B, 6 chunks per block
    atoms = _atoms(rng, 3, bt, 5)
    t = Twin(L, H, D, bt, 500)
    t.gpu.set_copy_shape(cpg, threads, grid)
    toks, offs = random_block_batch(rng, 40, atoms, 8, tail_p=0.3)
    R, maxb = len(offs) - 1, 8
    (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, maxb)
    t.scatter_random(ids, cr, rids, rcr, block_table_identity(R, maxb), seed=11)
    t.check_pool()
    # gather through a permuted block table with holes into a sentinel cache
    lt, lo = random_block_batch(rng, 30, atoms, 10, tail_p=0.5)
    R2, maxb2 = len(lo) - 1, 10
    NB2 = R2 * maxb2 + 13
    perm = rng.permutation(NB2)[:R2 * maxb2].astype(np.int32).reshape(R2, maxb2)
    perm[rng.random(perm.shape) < 0.2] = -1
    t.lookup_gather(lt, lo, maxb2, perm, NB2)
    assert t.gpu.stats()["bad_entries"] == 0
    t.close()


def test_gather_skips_out_of_range_entries():
    t = Twin(2, 1, 8, 16, 64)
    toks, offs = synth.concat_requests([np.arange(48, dtype=np.int32)])
    (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, 3)
    t.scatter_random(ids, cr, rids, rcr, np.array([[0, 1, 2]], np.int32), seed=3)
    bt_tab = np.array([[0, 99, 1]], dtype=np.int32)  # 99 >= cache_blocks
    t.lookup_gather(toks, offs, 3, bt_tab, 4)
    assert t.gpu.stats()["bad_entries"] == 1 and t.ref.bad_entries == 1
    # ids beyond the stored count through the plain gather entry point
    cache = torch.zeros(2 * 2 * 4 * t.shape.chunk_bytes, dtype=torch.uint8, device=DEV)
    bad_ids = to_dev(np.array([[0, 7, -3]], np.int32))
    t.gpu.gather(bad_ids, to_dev(np.array([3], np.int32)), to_dev(np.array([[0, 1, 2]], np.int32)),
                 cache)
    assert t.gpu.stats()["bad_entries"] == 3
    t.close()


# ---------------------------------------------------------------------------
# capacity and edge cases
# ---------------------------------------------------------------------------

def test_capacity_cut_matches_oracle():
    rng = np.random.default_rng(12)
    atoms = _atoms(rng, 3, 16, 4)
    t = Twin(1, 1, 8, 16, 37)
    for _ in range(3):
        toks, offs = random_block_batch(rng, 30, atoms, 12)
        t.insert(toks, offs, 12)
    assert t.gpu.stats()["blocks_stored"] == 37 and t.gpu.stats()["full_events"] >= 1
    toks, offs = random_block_batch(rng, 30, atoms, 12)
    t.lookup(toks, offs, 12)
    t.close()


def test_tiny_index_limits_capacity():
    t = Twin(1, 1, 8, 16, 1000, index_slots=16)  # at most 8 blocks
    assert t.capacity == 8
    toks, offs = synth.concat_requests([np.arange(16 * 12, dtype=np.int32)])
    t.insert(toks, offs, 12)
    assert t.gpu.stats()["blocks_stored"] == 8
    t.lookup(toks, offs, 12)
    t.close()


def test_edge_cases():
    t = Twin(1, 1, 8, 16, 100)
    # empty batch
    (m, ids), _ = t.lookup(np.zeros(0, np.int32), np.zeros(1, np.int64), 4)
    assert m.numel() == 0
    t.insert(np.zeros(0, np.int32), np.zeros(1, np.int64), 4)
    # empty requests, shorter than one block, ragged tails, exactly one block
    seqs = [np.zeros(0, np.int32), np.arange(5, dtype=np.int32), np.arange(16, dtype=np.int32),
            np.arange(37, dtype=np.int32), np.arange(16 * 70 + 3, dtype=np.int32)]
    toks, offs = synth.concat_requests(seqs)
    t.insert(toks, offs, 1)     # max_blocks = 1
    t.insert(toks, offs, 64)    # exactly one window
    t.insert(toks, offs, 65)    # one block into the second window
    t.lookup(toks, offs, 200)   # more room than any request needs
    # full match: every block of the request is stored
    (m, ids), _ = t.lookup(toks[offs[3]:offs[4]], np.array([0, 37]), 10)
    assert host(m).tolist() == [2]
    t.close()


def test_invalid_arguments_are_rejected():
    lib = P.lib()
    s = P.PrefixStore(P.StoreShape(1, 1, 8, 16), 10)
    d = torch.zeros(64, dtype=torch.int32, device=DEV)
    o = torch.zeros(2, dtype=torch.int64, device=DEV)
    bad = [
        lib.ptstore_lookup(s.h, d.data_ptr(), o.data_ptr(), 64, 1, 0, d.data_ptr(), d.data_ptr(), None),
        lib.ptstore_lookup(s.h, d.data_ptr(), o.data_ptr(), 64, -1, 4, d.data_ptr(), d.data_ptr(), None),
        lib.ptstore_lookup(s.h, d.data_ptr(), None, 64, 1, 4, d.data_ptr(), d.data_ptr(), None),
        lib.ptstore_lookup(None, d.data_ptr(), o.data_ptr(), 64, 1, 4, d.data_ptr(), d.data_ptr(), None),
        lib.ptstore_gather(s.h, d.data_ptr(), d.data_ptr(), d.data_ptr(), 1, 4, d.data_ptr() + 4, 1, None),
        lib.ptstore_insert(s.h, d.data_ptr(), o.data_ptr(), 1 << 33, 1, 4, d.data_ptr(), d.data_ptr(),
                           d.data_ptr(), None),
    ]
    assert all(rc == P.PTSTORE_ERR_INVALID for rc in bad), bad
    cfg = P.ptstore_config_t(1, 1, 8, 16, 2, 10, 6, 0, 0)  # index_slots not a power of two
    h = C.c_void_p()
    assert lib.ptstore_create(C.byref(cfg), C.byref(h)) == P.PTSTORE_ERR_INVALID
    cfg = P.ptstore_config_t(1, 1, 3, 1, 2, 10, 0, 0, 0)  # chunk of 6 bytes
    assert lib.ptstore_create(C.byref(cfg), C.byref(h)) == P.PTSTORE_ERR_INVALID
    s.close()


def test_malformed_offsets_are_empty_and_counted():
    s = P.PrefixStore(P.StoreShape(1, 1, 8, 16), 100)
    toks = to_dev(np.arange(64, dtype=np.int32))
    offs = to_dev(np.array([0, 32, 16, 200], np.int64))  # decreasing, then beyond n_tokens
    m, ids, cr = s.insert(toks, offs, 4)
    torch.cuda.synchronize()
    assert host(m).tolist() == [2, 0, 0]
    assert s.stats()["bad_entries"] == 2
    s.close()


# ---------------------------------------------------------------------------
# workload-shaped cases, scaled down
# ---------------------------------------------------------------------------

def _prefill(t: Twin, toks, offs, maxb, seed, batch=64):
    """Insert + scatter in batches, checking every output."""
    R = len(offs) - 1
    for lo in range(0, R, batch):
        hi = min(R, lo + batch)
        bt_, bo = toks[offs[lo]:offs[hi]], (offs[lo:hi + 1] - offs[lo]).astype(np.int64)
        (m, ids, cr), (rc, rm, rids, rcr) = t.insert(bt_, bo, maxb)
        t.scatter_random(ids, cr, rids, rcr, block_table_identity(hi - lo, maxb), seed=seed + lo)


def test_tiny_config_full():
    w = synth.build("tiny")
    t = Twin.for_shape(w.shape, 4096)
    st_, so = w.store_batch()
    _prefill(t, st_, so, w.passage_blocks, seed=21)
    t.check_pool()
    R, maxb = w.n_requests, w.max_blocks
    (m, ids, _), _ = t.lookup_gather(w.tokens, w.offsets, maxb, block_table_identity(R, maxb), R * maxb)
    expect = np.where(np.isin(w.req_passage, w.stored), w.passage_blocks, 0)
    np.testing.assert_array_equal(host(m), expect)
    t.close()


def test_llama8b_shape_small():
    """32 layers x 8 heads x 128 bf16 (2 MiB blocks), few passages."""
    w = synth.build("llama8b", n_passages=8, n_requests=8, stored_ranks=[1, 2, 3, 4])
    t = Twin.for_shape(w.shape, 4 * 224 + 64)
    st_, so = w.store_batch()
    _prefill(t, st_, so, w.passage_blocks, seed=31, batch=2)
    R, maxb = w.n_requests, w.max_blocks
    t.lookup_gather(w.tokens, w.offsets, maxb, block_table_identity(R, maxb), R * maxb)
    t.close()


def test_llama70b_shape_short_passages():
    """80 layers (5 MiB blocks, 160 chunks per block) with short passages."""
    w = synth.build("llama70b_shard", n_passages=4, passage_tokens=1024, suffix_tokens=256,
                    n_requests=4, stored_ranks=[1, 3])
    t = Twin.for_shape(w.shape, 256)
    st_, so = w.store_batch()
    _prefill(t, st_, so, w.passage_blocks, seed=41, batch=2)
    R, maxb = w.n_requests, w.max_blocks
    t.lookup_gather(w.tokens, w.offsets, maxb, block_table_identity(R, maxb), R * maxb)
    t.close()


def test_long_requests_many_windows():
    """32768-token requests (2048 blocks = 32 windows) with a small KV shape."""
    kv = synth.KVShape(1, 1, 8, 16, "fp16")
    w = synth.make_passage_workload("long", kv, 6, 30720, 2048, 8, 1.2, [1, 3, 5], 4, seed=5)
    t = Twin.for_shape(kv, 3 * 1920 + 16)
    st_, so = w.store_batch()
    _prefill(t, st_, so, w.passage_blocks, seed=51, batch=3)
    R, maxb = w.n_requests, w.max_blocks
    (m, _, _), _ = t.lookup_gather(w.tokens, w.offsets, maxb, block_table_identity(R, maxb), R * maxb)
    expect = np.where(np.isin(w.req_passage, w.stored), 1920, 0)
    np.testing.assert_array_equal(host(m), expect)
    # branch inside a window and exactly on window boundaries
    base = w.passages[0]
    seqs = []
    for cut in (63, 64, 65, 127, 128, 1000, 1919):
        s = base.copy()
        s[cut * 16 + 3] += 1
        seqs.append(s)
    toks, offs = synth.concat_requests(seqs)
    (m, _), _ = t.lookup(toks, offs, 2048)
    assert host(m).tolist() == [63, 64, 65, 127, 128, 1000, 1919]
    t.close()


def test_trie_config_small():
    cap = 20_000
    w = synth.build("trie", capacity=cap, n_requests=1024, chunk_walks=4096)
    t = Twin.for_shape(w.shape, cap)
    R = len(w.store_offsets) - 1
    for lo in range(0, R, 512):
        hi = min(R, lo + 512)
        toks = w.store_tokens[w.store_offsets[lo]:w.store_offsets[hi]]
        offs = (w.store_offsets[lo:hi + 1] - w.store_offsets[lo]).astype(np.int64)
        (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, w.depth)
        t.scatter_random(ids, cr, rids, rcr, block_table_identity(hi - lo, w.depth), seed=lo)
    assert t.gpu.stats()["blocks_stored"] == cap
    t.check_pool()
    Rq = w.n_requests
    t.lookup_gather(w.tokens, w.offsets, w.depth, block_table_identity(Rq, w.depth), Rq * w.depth)
    t.close()


def test_stream_config_small():
    kv = synth.KVShape(2, 8, 128, 16, "bf16")
    sw = synth.build("stream", n_rounds=6, per_round=24, pool_blocks=4000,
                     base_override=dict(shape=kv, n_passages=24, passage_tokens=512,
                                        suffix_tokens=128, n_requests=24,
                                        stored_ranks=list(range(1, 13))))
    base = sw.base
    t = Twin.for_shape(kv, sw.pool_blocks)
    st_, so = base.store_batch()
    _prefill(t, st_, so, base.passage_blocks, seed=61)
    maxb = int(np.diff(base.offsets).max()) // 16
    for i, rd in enumerate(sw.rounds):
        R = len(rd.lookup_offsets) - 1
        t.lookup_gather(rd.lookup_tokens, rd.lookup_offsets, maxb, block_table_identity(R, maxb),
                        R * maxb)
        Ri = len(rd.insert_offsets) - 1
        (m, ids, cr), (rc, rm, rids, rcr) = t.insert(rd.insert_tokens, rd.insert_offsets, maxb)
        t.scatter_random(ids, cr, rids, rcr, block_table_identity(Ri, maxb), seed=1000 + i)
    t.check_pool()
    t.check_meta()
    t.close()


def test_copy_grid_beyond_launch_limit():
    """More (request, block, chunk) units than one launch may hold: the copy
    kernels walk them grid-stride (20,000 requests x 64 blocks x 2 chunks)."""
    rng = np.random.default_rng(13)
    R, maxb = 20_000, 64
    toks = rng.integers(0, 32000, size=R * maxb * 16, dtype=np.int32)
    offs = np.arange(R + 1, dtype=np.int64) * (maxb * 16)
    t = Twin(1, 1, 8, 16, R * maxb)
    (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, maxb)
    t.scatter_random(ids, cr, rids, rcr, block_table_identity(R, maxb), seed=17)
    t.check_pool()
    t.lookup_gather(toks, offs, maxb, block_table_identity(R, maxb), R * maxb)
    t.close()


def test_batch_at_the_size_limit():
    """R x max_blocks at its limit, 2^29 (8192 requests x 65,536 blocks of
    room): lookup, insert and gather agree with the oracle on every request,
    all room past a request's blocks reads -1, and one entry more is refused
    before any work."""
    R, maxb = 1 << 13, 1 << 16
    rng = np.random.default_rng(23)
    bt_ = 16
    stored = [rng.integers(0, 32000, size=bt_ * k, dtype=np.int32) for k in (1, 2, 3, 4)]
    t = Twin(1, 1, 8, bt_, 64)
    st_toks, st_offs = synth.concat_requests(stored[1:3])
    (m, ids, cr), (rc, rm, rids, rcr) = t.insert(st_toks, st_offs, 4)
    t.scatter_random(ids, cr, rids, rcr, block_table_identity(2, 4), seed=5)
    # every request is one of the four sequences, some of them extended
    pick = rng.integers(0, 4, size=R)
    seqs = [stored[p] if i % 3 else np.concatenate([stored[p], stored[0]]) for i, p in enumerate(pick)]
    toks, offs = synth.concat_requests(seqs)
    tt, oo = to_dev(toks), to_dev(offs)
    s = t.gpu
    m = torch.empty(R, dtype=torch.int32, device=DEV)
    ids = torch.empty((R, maxb), dtype=torch.int32, device=DEV)
    s.lookup(tt, oo, maxb, m=m, ids=ids)
    om, oids = t.ref.lookup(toks, offs, 8)  # no request has more than 5 blocks
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(m), om)
    np.testing.assert_array_equal(host(ids[:, :8]), oids)
    assert bool((ids[:, 8:] == -1).all())
    # gather: destinations for the first 8 columns only, the rest -1
    bt = torch.full((R, maxb), -1, dtype=torch.int32, device=DEV)
    bt[:, :8] = torch.arange(R * 8, dtype=torch.int32, device=DEV).view(R, 8)
    n = R * 8 * t.shape.block_bytes
    cache = torch.full((n,), 0xA5, dtype=torch.uint8, device=DEV)
    s.gather(ids, m, bt, cache)
    rdst = np.full(n, 0xA5, dtype=np.uint8)
    t.ref.gather(oids, om, block_table_identity(R, 8), rdst, R * 8)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(cache), rdst)
    # insert of the same batch: the new blocks, each created once
    im, iids, icr = s.insert(tt, oo, maxb)
    orc = t.ref.insert(toks, offs, 8)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(im), orc[1])
    np.testing.assert_array_equal(host(iids[:, :8]), orc[2])
    np.testing.assert_array_equal(host(icr[:, :8]).astype(bool), orc[3].astype(bool))
    assert bool((iids[:, 8:] == -1).all()) and int(icr[:, 8:].sum()) == 0
    # one more request over the limit is refused on the host, by every call
    lib = P.lib()
    over = [
        lib.ptstore_lookup(s.h, tt.data_ptr(), oo.data_ptr(), tt.numel(), R + 1, maxb,
                           m.data_ptr(), ids.data_ptr(), None),
        lib.ptstore_gather(s.h, ids.data_ptr(), m.data_ptr(), bt.data_ptr(), R + 1, maxb,
                           cache.data_ptr(), R * 8, None),
        lib.ptstore_gather_prepare(s.h, ids.data_ptr(), m.data_ptr(), bt.data_ptr(), R + 1, maxb,
                                   R * 8, None),
        lib.ptstore_scatter(s.h, iids.data_ptr(), icr.data_ptr(), bt.data_ptr(), R + 1, maxb,
                            cache.data_ptr(), R * 8, None),
        lib.ptstore_insert(s.h, tt.data_ptr(), oo.data_ptr(), tt.numel(), R + 1, maxb,
                           im.data_ptr(), iids.data_ptr(), icr.data_ptr(), None),
    ]
    assert all(rc == P.PTSTORE_ERR_INVALID for rc in over), over
    t.close()


@pytest.mark.parametrize("evict", [False, True])
def test_insert_sync_reports_refused_blocks(evict):
    """ptstore_insert_sync returns PTSTORE_ERR_FULL exactly when the oracle's
    insert refused blocks, with the same outputs either way."""
    from oracle import ORC_ERR_FULL
    rng = np.random.default_rng(71 + evict)
    atoms = _atoms(rng, 5, 4, 50)
    t = Twin(1, 1, 8, 4, 30, flags=P.PTSTORE_FLAG_EVICT if evict else 0)
    codes = set()
    for i in range(10):  # small and large batches taking turns
        toks, offs = random_block_batch(rng, 10 if i % 2 else 2, atoms, 9)
        rc, m, ids, cr = t.gpu.insert_sync(to_dev(toks), to_dev(offs), 9)
        orc, rm, rids, rcr = t.ref.insert(toks, offs, 9)
        assert (rc == P.PTSTORE_ERR_FULL) == (orc == ORC_ERR_FULL), (rc, orc)
        np.testing.assert_array_equal(host(m), rm)
        np.testing.assert_array_equal(host(ids), rids)
        np.testing.assert_array_equal(host(cr), rcr)
        codes.add(rc)
    assert codes == {P.PTSTORE_OK, P.PTSTORE_ERR_FULL}
    assert t.gpu.stats()["blocks_stored"] == t.ref.count
    t.close()


@pytest.mark.parametrize("fill", [0.25, 0.4, 0.5])
def test_index_load_factors(fill):
    """A 4096-slot index filled to 25, 40 and 50 % of its slots (50 % is the
    most a store holds): lookups of stored, extended and fresh sequences
    match the oracle at every fill, and probing stays short."""
    rng = np.random.default_rng(int(fill * 100))
    slots = 4096
    t = Twin(1, 1, 8, 4, 10_000, index_slots=slots, flags=P.PTSTORE_FLAG_COUNTERS)
    assert t.gpu.stats()["capacity"] == slots // 2
    want = int(fill * slots)
    seqs = []
    while t.ref.count < want:
        n = int(rng.integers(1, 9))
        need = min(8, want - t.ref.count)  # fill to the exact count
        s = rng.integers(0, 50, size=4 * min(n, need), dtype=np.int32)
        toks, offs = synth.concat_requests([s])
        t.insert(toks, offs, 8)
        seqs.append(s)
    assert t.gpu.stats()["blocks_stored"] == t.ref.count == want
    looks = []
    for _ in range(300):
        u = rng.random()
        s = seqs[int(rng.integers(len(seqs)))]
        if u < 0.4:
            looks.append(s)  # stored
        elif u < 0.7:
            looks.append(np.concatenate([s, rng.integers(0, 50, size=8, dtype=np.int32)]))  # extended
        else:
            looks.append(rng.integers(0, 50, size=4 * int(rng.integers(1, 9)), dtype=np.int32))  # fresh
    toks, offs = synth.concat_requests(looks)
    t.gpu.reset_counters()
    (m, ids), (rm, rids) = t.lookup(toks, offs, 12)
    st = t.gpu.stats()
    examined = int(np.minimum(np.diff(offs) // 4, 12).sum())
    assert st["probes"] <= 3 * examined  # linear probing at load <= 0.5 stays short
    assert rm.sum() > 0
    t.check_meta()
    t.close()
