"""Pins of the CPU oracle against things other than itself (no GPU).

- hand-derived golden example (tests/golden/incremental_ids.json);
- a brute force that takes the LCP as a maximum over all stored objects and
  ids as first-occurrence ranks of whole prefixes (oracle/brute.py);
- invariants stated by the paper (Section 1: redundancy-free trie growth;
  Section 4.1: inherited id lists, tensors guaranteed to exist);
- generator ground truth: which passage / tree node a request came from fixes
  its match length without any store;
- the pool / paged-cache layouts restated with numpy reshapes.
"""
from __future__ import annotations

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st, HealthCheck

from oracle import OracleStore, ORC_OK, ORC_ERR_FULL, brute
from workloads import synth
from tests.helpers import (load_golden, spell_batch, random_block_batch, block_table_identity,
                           cache_view, pool_view)


def small_store(block_tokens, capacity, layers=1, heads=1, dim=8, payload=True):
    return OracleStore(layers, heads, dim, block_tokens, 2, capacity, payload)


# --------------------------------------------------------------------------
# golden worked example
# --------------------------------------------------------------------------

@pytest.mark.parametrize("case", load_golden("incremental_ids.json")["cases"], ids=lambda c: c["name"])
def test_golden_oracle(case):
    g = load_golden("incremental_ids.json")
    blocks, bt = g["blocks"], g["block_tokens"]
    o = small_store(bt, case["capacity"])
    toks, offs = spell_batch(case["insert"], blocks)
    rc, m, ids, created = o.insert(toks, offs, case["insert_max_blocks"])
    e = case["expect_insert"]
    assert (rc == ORC_ERR_FULL) == e["rc_full"]
    assert m.tolist() == e["m"]
    assert ids.tolist() == e["ids"]
    assert created.tolist() == e["created"]
    assert o.count == e["count"]
    toks, offs = spell_batch(case["lookup"], blocks)
    m, ids = o.lookup(toks, offs, case["lookup_max_blocks"])
    assert m.tolist() == case["expect_lookup"]["m"]
    assert ids.tolist() == case["expect_lookup"]["ids"]


@pytest.mark.parametrize("case", load_golden("incremental_ids.json")["cases"], ids=lambda c: c["name"])
def test_golden_brute(case):
    g = load_golden("incremental_ids.json")
    blocks, bt = g["blocks"], g["block_tokens"]
    b = brute.BruteStore(bt, case["capacity"])
    toks, offs = spell_batch(case["insert"], blocks)
    full, m, ids, created = b.insert(toks, offs, case["insert_max_blocks"])
    e = case["expect_insert"]
    assert full == e["rc_full"]
    assert m.tolist() == e["m"] and ids.tolist() == e["ids"] and created.tolist() == e["created"]
    toks, offs = spell_batch(case["lookup"], blocks)
    m, ids = b.lookup(toks, offs, case["lookup_max_blocks"])
    assert m.tolist() == case["expect_lookup"]["m"]
    assert ids.tolist() == case["expect_lookup"]["ids"]


# --------------------------------------------------------------------------
# brute force on random tiny tries
# --------------------------------------------------------------------------

def _atoms(rng, n_atoms, bt, vocab, shared_head=False):
    """``n_atoms`` distinct blocks; with ``shared_head`` they differ only in the last token."""
    while True:
        a = rng.integers(0, vocab, size=(n_atoms, bt), dtype=np.int32)
        if shared_head:
            a[:, :-1] = a[0, :-1]
        if len({r.tobytes() for r in a}) == n_atoms:
            return a


def _check_against_brute(seed, bt, n_atoms, vocab, max_len, max_blocks, capacity, rounds, n_req,
                         shared_head=False):
    rng = np.random.default_rng(seed)
    atoms = _atoms(rng, n_atoms, bt, vocab, shared_head)
    o = small_store(bt, capacity, payload=False)
    b = brute.BruteStore(bt, capacity)
    for _ in range(rounds):
        toks, offs = random_block_batch(rng, n_req, atoms, max_len)
        rc, m, ids, created = o.insert(toks, offs, max_blocks)
        full, bm, bids, bcreated = b.insert(toks, offs, max_blocks)
        assert (rc == ORC_ERR_FULL) == full
        np.testing.assert_array_equal(m, bm)
        np.testing.assert_array_equal(ids, bids)
        np.testing.assert_array_equal(created, bcreated)
        assert o.count == b.count
        toks, offs = random_block_batch(rng, n_req, atoms, max_len + 2)
        m, ids = o.lookup(toks, offs, max_blocks)
        bm, bids = b.lookup(toks, offs, max_blocks)
        np.testing.assert_array_equal(m, bm)
        np.testing.assert_array_equal(ids, bids)


@settings(max_examples=60, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(seed=st.integers(0, 2**31 - 1), bt=st.sampled_from([1, 2, 3, 4, 16]),
       n_atoms=st.integers(1, 4), max_len=st.integers(0, 7), max_blocks=st.integers(1, 8),
       capacity=st.integers(0, 40), shared_head=st.booleans())
def test_oracle_matches_brute_force(seed, bt, n_atoms, max_len, max_blocks, capacity, shared_head):
    if shared_head and n_atoms > 4:
        n_atoms = 4
    _check_against_brute(seed, bt, n_atoms, 4, max_len, max_blocks, capacity, rounds=3, n_req=12,
                         shared_head=shared_head)


def test_oracle_matches_brute_force_larger():
    # more requests per batch, deeper sequences, no capacity pressure
    _check_against_brute(7, 4, 3, 3, 12, 10, 10_000, rounds=4, n_req=60)
    # blocks that differ only in their last token
    _check_against_brute(8, 16, 3, 4, 8, 8, 10_000, rounds=3, n_req=40, shared_head=True)


# --------------------------------------------------------------------------
# invariants
# --------------------------------------------------------------------------

def test_invariants_after_inserts():
    rng = np.random.default_rng(11)
    bt, maxb = 3, 9
    atoms = _atoms(rng, 3, bt, 5)
    o = small_store(bt, 10_000, payload=False)
    inserted = []
    for _ in range(5):
        toks, offs = random_block_batch(rng, 40, atoms, 9)
        rc, m, ids, created = o.insert(toks, offs, maxb)
        assert rc == ORC_OK
        for r in range(len(offs) - 1):
            seq = toks[offs[r]:offs[r + 1]]
            n = min(len(seq) // bt, maxb)
            assert m[r] == n  # nothing refused without capacity pressure
            for k in range(n):
                parent, btoks = o.node(int(ids[r, k]))
                # (ii) parent link and tokens of every id on the path
                assert parent == (ids[r, k - 1] if k else -1)
                np.testing.assert_array_equal(btoks, seq[k * bt:(k + 1) * bt])
            inserted.append((seq, ids[r, :n].copy()))
    # (i) no two nodes share (parent, tokens): the store is redundancy-free
    keys = set()
    for i in range(o.count):
        p, t = o.node(i)
        keys.add((p, t.tobytes()))
    assert len(keys) == o.count
    # count == number of distinct whole-block prefixes inserted
    prefixes = set()
    for seq, _ in inserted:
        n = min(len(seq) // bt, maxb)
        for k in range(1, n + 1):
            prefixes.add(seq[:k * bt].tobytes())
    assert len(prefixes) == o.count
    # (iii) looking up an inserted sequence returns the ids its insert returned
    toks, offs = synth.concat_requests([s for s, _ in inserted])
    m, ids = o.lookup(toks, offs, maxb)
    for r, (seq, got) in enumerate(inserted):
        assert m[r] == len(got)
        np.testing.assert_array_equal(ids[r, :len(got)], got)


def test_gather_scatter_layout_and_sentinel():
    """(iv) gathered bytes == pool bytes, nothing else written; (v) scatter copies
    the first occurrence of a shared new block."""
    rng = np.random.default_rng(3)
    L, H, D, bt = 3, 2, 4, 2
    o = OracleStore(L, H, D, bt, 2, 64, True)
    chunk = H * bt * D * 2
    atoms = _atoms(rng, 3, bt, 6)
    toks, offs = random_block_batch(rng, 20, atoms, 5, tail_p=0.0)
    R, maxb = len(offs) - 1, 5
    NB = R * maxb
    cache = rng.integers(0, 256, size=L * 2 * NB * chunk, dtype=np.uint8)
    bt_tab = block_table_identity(R, maxb)
    rc, m, ids, created = o.insert(toks, offs, maxb)
    assert rc == ORC_OK
    o.scatter(ids, created, bt_tab, cache, NB)
    cv = cache_view(cache, L, NB, chunk)
    pv = pool_view(o.pool(), L, chunk)
    seen = set()
    for r in range(R):
        for b in range(m[r]):
            i = ids[r, b]
            if created[r, b]:
                assert i not in seen
                seen.add(i)
                for l in range(L):
                    for kv in range(2):
                        np.testing.assert_array_equal(pv[i, l, kv], cv[l, kv, bt_tab[r, b]])
    assert seen == set(range(o.count))
    # gather into a sentinel-filled cache through a permuted block table with holes
    lt, lo = random_block_batch(rng, 15, atoms, 6, tail_p=0.5)
    R2, maxb2 = len(lo) - 1, 6
    NB2 = R2 * maxb2 + 7
    m2, ids2 = o.lookup(lt, lo, maxb2)
    perm = rng.permutation(NB2)[:R2 * maxb2].astype(np.int32).reshape(R2, maxb2)
    perm[rng.random(perm.shape) < 0.2] = -1
    dst = np.full(L * 2 * NB2 * chunk, 0xA5, dtype=np.uint8)
    o.gather(ids2, m2, perm, dst, NB2)
    dv = cache_view(dst, L, NB2, chunk)
    touched = np.zeros(NB2, dtype=bool)
    for r in range(R2):
        for b in range(m2[r]):
            if perm[r, b] < 0:
                continue
            touched[perm[r, b]] = True
            for l in range(L):
                for kv in range(2):
                    np.testing.assert_array_equal(dv[l, kv, perm[r, b]], pv[ids2[r, b], l, kv])
    assert (dv[:, :, ~touched] == 0xA5).all()
    assert o.bad_entries == 0


def test_gather_skips_out_of_range_entries():
    o = OracleStore(1, 1, 8, 2, 2, 8, True)
    toks, offs = spell_batch(["AB"], {"A": [1, 2], "B": [3, 4]})
    rc, m, ids, created = o.insert(toks, offs, 2)
    chunk = 1 * 2 * 8 * 2
    cache = np.zeros(2 * 4 * chunk, dtype=np.uint8)
    bt_tab = np.array([[0, 9]], dtype=np.int32)  # 9 >= cache_blocks (4)
    o.gather(ids, m, bt_tab, cache, 4)
    assert o.bad_entries == 1
    bad_ids = np.array([[0, 5]], dtype=np.int32)  # id 5 was never created
    o.gather(bad_ids, m, np.array([[0, 1]], dtype=np.int32), cache, 4)
    assert o.bad_entries == 2


# --------------------------------------------------------------------------
# generator ground truth
# --------------------------------------------------------------------------

def test_ground_truth_tiny():
    w = synth.build("tiny")
    o = OracleStore.for_shape(w.shape, capacity=4096, with_payload=False)
    st_toks, st_offs = w.store_batch()
    rc, m, ids, created = o.insert(st_toks, st_offs, w.passage_blocks)
    assert rc == ORC_OK and o.count == 16 * 48
    # ids are handed out passage after passage, block after block
    np.testing.assert_array_equal(ids, np.arange(16 * 48).reshape(16, 48))
    m, ids = o.lookup(w.tokens, w.offsets, w.max_blocks)
    expect = np.where(np.isin(w.req_passage, w.stored), w.passage_blocks, 0)
    np.testing.assert_array_equal(m, expect)
    rank_of = {int(p): i for i, p in enumerate(w.stored)}
    for r in range(w.n_requests):
        if m[r]:
            base = rank_of[int(w.req_passage[r])] * 48
            np.testing.assert_array_equal(ids[r, :48], np.arange(base, base + 48))


@pytest.mark.slow
def test_ground_truth_llama8b_metadata():
    w = synth.build("llama8b")
    o = OracleStore.for_shape(w.shape, capacity=57344, with_payload=False)
    st_toks, st_offs = w.store_batch()
    rc, m, _, _ = o.insert(st_toks, st_offs, w.passage_blocks)
    assert rc == ORC_OK and o.count == 57344 and (m == 224).all()
    m, _ = o.lookup(w.tokens, w.offsets, w.max_blocks)
    expect = np.where(np.isin(w.req_passage, w.stored), 224, 0)
    np.testing.assert_array_equal(m, expect)


def test_ground_truth_trie_small():
    cap = 6000
    w = synth.build("trie", capacity=cap, n_requests=400, chunk_walks=2048)
    o = OracleStore.for_shape(w.shape, capacity=cap, with_payload=False)
    rc, m_ins, _, _ = o.insert(w.store_tokens, w.store_offsets, w.depth)
    assert o.count == cap
    # resident nodes = the first `cap` distinct tree nodes in walk order
    flat = w.store_paths.ravel()
    uniq, first = np.unique(flat, return_index=True)
    resident = set(uniq[np.argsort(first)][:cap].tolist())
    m, _ = o.lookup(w.tokens, w.offsets, w.depth)
    for r in range(w.n_requests):
        k = 0
        while k < w.depth and int(w.req_paths[r, k]) in resident:
            k += 1
        assert m[r] == k


# --------------------------------------------------------------------------
# edge cases and argument checks
# --------------------------------------------------------------------------

def test_empty_batch_and_empty_requests():
    o = small_store(4, 10)
    m, ids = o.lookup(np.zeros(0, np.int32), np.zeros(1, np.int64), 3)
    assert m.shape == (0,) and ids.shape == (0, 3)
    rc, m, ids, cr = o.insert(np.zeros(0, np.int32), np.zeros(1, np.int64), 3)
    assert rc == ORC_OK and o.count == 0
    toks, offs = synth.concat_requests([np.zeros(0, np.int32), np.arange(3, dtype=np.int32)])
    rc, m, ids, cr = o.insert(toks, offs, 3)
    assert m.tolist() == [0, 0] and o.count == 0


def test_full_match_and_max_blocks_truncation():
    o = small_store(2, 100)
    toks, offs = synth.concat_requests([np.arange(10, dtype=np.int32)])
    rc, m, ids, cr = o.insert(toks, offs, 3)  # only 3 of 5 blocks considered
    assert m.tolist() == [3] and o.count == 3
    m, ids = o.lookup(toks, offs, 5)
    assert m.tolist() == [3]
    m, ids = o.lookup(toks[:6], np.array([0, 6]), 5)  # full match: m == n
    assert m.tolist() == [3] and ids[0, :3].tolist() == [0, 1, 2]


def test_capacity_zero():
    o = small_store(2, 0)
    toks, offs = synth.concat_requests([np.arange(4, dtype=np.int32)])
    rc, m, ids, cr = o.insert(toks, offs, 2)
    assert rc == ORC_ERR_FULL and m.tolist() == [0] and o.count == 0


def test_invalid_arguments():
    o = small_store(2, 10)
    with pytest.raises(ValueError):
        o.lookup(np.arange(4, dtype=np.int32), np.array([0, 4]), 0)
    with pytest.raises(ValueError):
        o.lookup(np.arange(4, dtype=np.int32), np.array([3, 1]), 2)  # decreasing offsets
