"""Eviction mode: GPU library vs the CPU oracle, element by element.

The store evicts leaf blocks by frequency (Section 4.1, "Access
pattern-aware eviction policy"; the exact reading is the one the oracle and
tests/golden/eviction.json pin). Every step compares the outputs of insert,
lookup and gather, and after it the access counts and priorities of every
block, the clock, the number of evictions, the block metadata and the pool.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from workloads import synth
from tests.helpers import load_golden, spell_batch, random_block_batch, block_table_identity

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2607_22648_amd import ptstore as P
    from tests.twin import Twin, host

    EVICT = P.PTSTORE_FLAG_EVICT


def _atoms(rng, n, bt, vocab):
    while True:
        a = rng.integers(0, vocab, size=(n, bt), dtype=np.int32)
        if len({r.tobytes() for r in a}) == n:
            return a


@pytest.mark.parametrize("case", load_golden("eviction.json")["cases"], ids=lambda c: c["name"])
def test_golden_eviction(case):
    g = load_golden("eviction.json")
    t = Twin(1, 1, 8, g["block_tokens"], case["capacity"], flags=EVICT)
    maxb = case["max_blocks"]
    for step in case["steps"]:
        toks, offs = spell_batch(step["batch"], g["blocks"])
        if step["op"] == "insert":
            (m, ids, cr), _ = t.insert(toks, offs, maxb)
            assert host(cr).tolist() == step["created"], step["why"]
        else:
            (m, ids), _ = t.lookup(toks, offs, maxb)
        assert host(m).tolist() == step["m"], step["why"]
        assert host(ids).tolist() == step["ids"], step["why"]
        t.check_evict()
        f, h = t.gpu.evict_tensors()
        f, h = host(f), host(h)
        for nid, (ef, eh) in step["nodes"].items():
            assert (f[int(nid)], h[int(nid)]) == (ef, eh), (step["why"], nid)
        if "clock" in step:
            st = t.gpu.stats()
            assert st["clock"] == step["clock"] and st["evictions"] == step["evictions"], step["why"]
        t.check_meta()
    t.close()


def _random_evict(seed, bt, n_atoms, max_len, capacity, maxb, rounds, n_req, flags=0,
                  index_slots=0, p_lookup=0.4, layers=1, heads=1, dim=8):
    rng = np.random.default_rng(seed)
    atoms = _atoms(rng, n_atoms, bt, 1000)
    t = Twin(layers, heads, dim, bt, capacity, flags=EVICT | flags, index_slots=index_slots)
    for i in range(rounds):
        toks, offs = random_block_batch(rng, int(rng.integers(1, n_req + 1)), atoms, max_len)
        R = len(offs) - 1
        if rng.random() < p_lookup:
            t.lookup_gather(toks, offs, maxb, block_table_identity(R, maxb), R * maxb)
        else:
            (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, maxb)
            t.scatter_random(ids, cr, rids, rcr, block_table_identity(R, maxb), seed=seed * 1000 + i)
        t.check_evict()
    t.check_meta()
    t.check_pool()
    st = t.gpu.stats()
    t.close()
    return st


@pytest.mark.parametrize("bt", [2, 16, 5])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_random_evict(seed, bt):
    st = _random_evict(seed, bt, n_atoms=3, max_len=6, capacity=9, maxb=6, rounds=30, n_req=8)
    assert st["evictions"] > 0


@pytest.mark.parametrize("seed", [3, 4])
def test_random_evict_weak_hash(seed):
    """8-bit index keys: key collisions everywhere, together with deleted slots."""
    st = _random_evict(seed, 4, n_atoms=5, max_len=8, capacity=24, maxb=8, rounds=30, n_req=10,
                       flags=P.PTSTORE_FLAG_WEAK_HASH)
    assert st["evictions"] > 0


def test_index_rebuilds_keep_results():
    """A 16-slot index rebuilt every few inserts (deleted slots pile up fast)."""
    st = _random_evict(5, 2, n_atoms=4, max_len=6, capacity=8, maxb=6, rounds=60, n_req=6,
                       index_slots=16)
    assert st["index_rebuilds"] > 2 and st["evictions"] > 20


def test_long_requests_evict():
    """Requests of up to 150 blocks: matches and cuts span several 64-block windows."""
    rng = np.random.default_rng(77)
    bt, maxb, cap = 16, 160, 600
    t = Twin(1, 1, 8, bt, cap, flags=EVICT)
    base = [rng.integers(0, 50_000, size=150 * bt, dtype=np.int32) for _ in range(4)]
    for i in range(12):
        seqs = []
        for _ in range(6):
            s = base[int(rng.integers(4))]
            cut = int(rng.integers(1, 151)) * bt
            tail = rng.integers(0, 50_000, size=int(rng.integers(0, 40)) * bt, dtype=np.int32)
            seqs.append(np.concatenate([s[:cut], tail]))
        toks, offs = synth.concat_requests(seqs)
        R = len(offs) - 1
        if i % 3 == 2:
            t.lookup_gather(toks, offs, maxb, block_table_identity(R, maxb), R * maxb)
        else:
            (m, ids, cr), (rc, rm, rids, rcr) = t.insert(toks, offs, maxb)
            t.scatter_random(ids, cr, rids, rcr, block_table_identity(R, maxb), seed=500 + i)
        t.check_evict()
    t.check_meta()
    t.check_pool()
    assert t.gpu.stats()["evictions"] > 0
    t.close()


def test_capacity_zero_evict():
    t = Twin(1, 1, 8, 2, 0, flags=EVICT)
    toks, offs = spell_batch(["AB", "C"], {"A": [1, 2], "B": [3, 4], "C": [5, 6]})
    (m, ids, cr), (rc, *_) = t.insert(toks, offs, 3)
    assert host(m).tolist() == [0, 0]
    t.lookup(toks, offs, 3)
    t.close()


def test_stream_evict_small():
    """The question-length stream on a small pool: it fills, then evicts every round."""
    kv = synth.KVShape(2, 8, 128, 16, "bf16")
    sw = synth.build("stream_evict", n_rounds=8, per_round=24, pool_blocks=700, fresh_blocks=(8, 8),
                     base_override=dict(shape=kv, n_passages=24, passage_tokens=512,
                                        suffix_tokens=128, n_requests=24,
                                        stored_ranks=list(range(1, 13))))
    base = sw.base
    t = Twin.for_shape(kv, sw.pool_blocks, flags=EVICT)
    st_, so = base.store_batch()
    maxb = int(np.diff(base.offsets).max()) // 16
    (m, ids, cr), (rc, rm, rids, rcr) = t.insert(st_, so, base.passage_blocks)
    R0 = len(so) - 1
    t.scatter_random(ids, cr, rids, rcr, block_table_identity(R0, base.passage_blocks), seed=71)
    for i, rd in enumerate(sw.rounds):
        R = len(rd.lookup_offsets) - 1
        t.lookup_gather(rd.lookup_tokens, rd.lookup_offsets, maxb, block_table_identity(R, maxb),
                        R * maxb)
        Ri = len(rd.insert_offsets) - 1
        (m, ids, cr), (rc, rm, rids, rcr) = t.insert(rd.insert_tokens, rd.insert_offsets, maxb)
        t.scatter_random(ids, cr, rids, rcr, block_table_identity(Ri, maxb), seed=2000 + i)
        t.check_evict()
    t.check_pool()
    t.check_meta()
    assert t.gpu.stats()["evictions"] > 0
    t.close()
