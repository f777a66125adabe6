"""Pins of the oracle's eviction mode against things other than itself (no GPU).

Section 4.1 ("Access pattern-aware eviction policy") asks for a
frequency-based, GDSF-style eviction; the exact reading (leaf-only victims,
H = L + F, protection of the batch's matches, the tie-break, the id reuse
order) is written out in tests/golden/eviction.json. Pins:

- that golden sequence, derived by hand, for the oracle and for the brute
  force of oracle/brute.py (prefix tuples in a dict, no trie);
- oracle == brute force on random interleavings of inserts and lookups on
  tiny stores that evict all the time, node statistics included;
- invariants: every id below the count holds a node, every parent is
  stored (prefix-closed), a parent's F and H are never below its child's;
- the equivalence the GPU selection relies on: the sequential leaf-by-leaf
  eviction takes exactly the first nodes of one global order over all
  unprotected nodes;
- payloads: after evictions and id reuse, a gather returns the bytes that
  were scattered for that very prefix.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import OracleStore, ORC_ERR_FULL, brute
from tests.helpers import load_golden, spell_batch, random_block_batch, cache_view

GOLDEN = "eviction.json"


def evict_store(block_tokens, capacity, layers=1, heads=1, dim=8, payload=True):
    return OracleStore(layers, heads, dim, block_tokens, 2, capacity, payload, evict=True)


def _run_golden(case, make):
    g = load_golden(GOLDEN)
    blocks = g["blocks"]
    st = make(g["block_tokens"], case["capacity"])
    maxb = case["max_blocks"]
    for step in case["steps"]:
        toks, offs = spell_batch(step["batch"], blocks)
        if step["op"] == "insert":
            full, m, ids, created = st.insert(toks, offs, maxb)
            assert full == step["rc_full"], step["why"]
            assert created.tolist() == step["created"], step["why"]
        else:
            m, ids = st.lookup(toks, offs, maxb)
        assert m.tolist() == step["m"], step["why"]
        assert ids.tolist() == step["ids"], step["why"]
        for nid, (f, h) in step["nodes"].items():
            assert st.stats_of(int(nid))[:2] == (f, h), (step["why"], nid)
        if "clock" in step:
            assert st.clock == step["clock"], step["why"]
            assert st.evictions == step["evictions"], step["why"]


class _OracleAdapter:
    def __init__(self, bt, cap):
        self.o = evict_store(bt, cap)

    def insert(self, toks, offs, maxb):
        rc, m, ids, created = self.o.insert(toks, offs, maxb)
        return rc == ORC_ERR_FULL, m, ids, created

    def lookup(self, toks, offs, maxb):
        return self.o.lookup(toks, offs, maxb)

    def stats_of(self, nid):
        return self.o.node_stats(nid)[:2]

    @property
    def clock(self):
        return self.o.clock

    @property
    def evictions(self):
        return self.o.evictions


class _BruteAdapter:
    def __init__(self, bt, cap):
        self.b = brute.BruteEvictStore(bt, cap)

    def insert(self, toks, offs, maxb):
        return self.b.insert(toks, offs, maxb)

    def lookup(self, toks, offs, maxb):
        return self.b.lookup(toks, offs, maxb)

    def stats_of(self, nid):
        return self.b.by_id()[nid][:2]

    @property
    def clock(self):
        return self.b.clock

    @property
    def evictions(self):
        return self.b.evictions


@pytest.mark.parametrize("case", load_golden(GOLDEN)["cases"], ids=lambda c: c["name"])
def test_golden_eviction_oracle(case):
    _run_golden(case, _OracleAdapter)


@pytest.mark.parametrize("case", load_golden(GOLDEN)["cases"], ids=lambda c: c["name"])
def test_golden_eviction_brute(case):
    _run_golden(case, _BruteAdapter)


# --------------------------------------------------------------------------
# oracle == brute force on random interleavings
# --------------------------------------------------------------------------

def _atoms(rng, n_atoms, bt, vocab):
    while True:
        a = rng.integers(0, vocab, size=(n_atoms, bt), dtype=np.int32)
        if len({r.tobytes() for r in a}) == n_atoms:
            return a


def _node_table(o: OracleStore):
    """id -> (parent, tokens, F, H, depth) of every id below the count."""
    out = {}
    for i in range(o.count):
        parent, toks = o.node(i)
        f, h, _, d = o.node_stats(i)
        out[i] = (parent, tuple(int(t) for t in toks), f, h, d)
    return out


def _brute_table(b: brute.BruteEvictStore):
    out = {}
    for key, (nid, f, h) in b.nodes.items():
        parent = -1 if len(key) == 1 else b.nodes[key[:-1]][0]
        out[nid] = (parent, key[-1], f, h, len(key) - 1)
    return out


def check_evict_against_brute(seed, bt, n_atoms, max_len, capacity, max_blocks, rounds=12,
                              n_req=6, p_lookup=0.4):
    rng = np.random.default_rng(seed)
    atoms = _atoms(rng, n_atoms, bt, 1000)
    o = evict_store(bt, capacity)
    b = brute.BruteEvictStore(bt, capacity)
    for _ in range(rounds):
        toks, offs = random_block_batch(rng, int(rng.integers(1, n_req + 1)), atoms, max_len)
        if rng.random() < p_lookup:
            mo, io = o.lookup(toks, offs, max_blocks)
            mb, ib = b.lookup(toks, offs, max_blocks)
            assert (mo == mb).all() and (io == ib).all()
        else:
            rc, mo, io, co = o.insert(toks, offs, max_blocks)
            full, mb, ib, cb = b.insert(toks, offs, max_blocks)
            assert (rc == ORC_ERR_FULL) == full
            assert (mo == mb).all() and (io == ib).all() and (co == cb).all()
        assert o.count == b.next_id
        assert o.clock == b.clock and o.evictions == b.evictions
        assert _node_table(o) == _brute_table(b)


@pytest.mark.parametrize("seed", range(12))
def test_evict_random_vs_brute(seed):
    check_evict_against_brute(seed, bt=2, n_atoms=3, max_len=5, capacity=6, max_blocks=5)


@pytest.mark.parametrize("seed", range(6))
def test_evict_random_vs_brute_wider(seed):
    check_evict_against_brute(100 + seed, bt=4, n_atoms=4, max_len=7, capacity=11, max_blocks=6,
                              rounds=16, n_req=8)


def test_evict_random_vs_brute_capacity_one():
    check_evict_against_brute(7, bt=2, n_atoms=3, max_len=3, capacity=1, max_blocks=3)


# --------------------------------------------------------------------------
# invariants and the global-order equivalence
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(8))
def test_evict_invariants(seed):
    rng = np.random.default_rng(1000 + seed)
    bt, cap, maxb = 2, 9, 6
    atoms = _atoms(rng, 4, bt, 50)
    o = evict_store(bt, cap)
    for _ in range(20):
        toks, offs = random_block_batch(rng, int(rng.integers(1, 7)), atoms, 6)
        if rng.random() < 0.4:
            o.lookup(toks, offs, maxb)
        else:
            o.insert(toks, offs, maxb)
        t = _node_table(o)
        assert len(t) == o.count <= cap  # no holes below the count
        for i, (parent, _, f, h, d) in t.items():
            if parent < 0:
                assert d == 0
                continue
            pp, _, pf, ph, pd = t[parent]
            assert pd == d - 1
            assert pf >= f and ph >= h  # a child is never accessed without its parent
            assert h <= o.clock + f  # priorities are set with a clock that only grows


@pytest.mark.parametrize("seed", range(10))
def test_sequential_leaf_eviction_is_a_global_order(seed):
    """The leaves taken one at a time are the first nodes of the order
    (H, deeper first, id) over all unprotected nodes: a child never ranks
    after its parent, and the unprotected nodes include every descendant of
    each of their members."""
    rng = np.random.default_rng(2000 + seed)
    bt, cap, maxb = 2, 7, 5
    atoms = _atoms(rng, 3, bt, 50)
    b = brute.BruteEvictStore(bt, cap)
    seen = 0
    for _ in range(30):
        toks, offs = random_block_batch(rng, int(rng.integers(1, 6)), atoms, 5)
        if rng.random() < 0.4:
            b.lookup(toks, offs, maxb)
            continue
        before = {k: list(v) for k, v in b.nodes.items()}
        protected = set()
        for r in range(len(offs) - 1):
            blocks = brute.request_blocks(toks, offs, r, bt, maxb)
            for j in range(len(blocks)):
                if tuple(blocks[:j + 1]) in before:
                    protected.add(tuple(blocks[:j + 1]))
        b.insert(toks, offs, maxb)
        order = sorted((k for k in before if k not in protected),
                       key=lambda k: (before[k][2], -len(k), before[k][0]))
        assert b.last_victims == order[:len(b.last_victims)]
        seen += len(b.last_victims)
    assert seen > 0


# --------------------------------------------------------------------------
# payload under id reuse
# --------------------------------------------------------------------------

def _payload_of(prefix_tokens: np.ndarray, nbytes: int) -> np.ndarray:
    """Bytes standing for the KV of one prefix: a function of its tokens only."""
    h = np.uint64(1469598103934665603)
    for t in prefix_tokens.tolist():
        h = np.uint64((int(h) ^ (t & 0xFFFFFFFF)) * 1099511628211 % (1 << 64))
    r = np.random.default_rng(int(h))
    return r.integers(0, 256, size=nbytes, dtype=np.uint8)


@pytest.mark.parametrize("seed", range(4))
def test_evict_gather_returns_the_prefix_payload(seed):
    rng = np.random.default_rng(3000 + seed)
    L, H, D, bt, cap, maxb = 2, 1, 8, 2, 5, 4
    o = OracleStore(L, H, D, bt, 2, cap, True, evict=True)
    chunk = H * bt * D * 2
    atoms = _atoms(rng, 3, bt, 50)
    for _ in range(12):
        toks, offs = random_block_batch(rng, int(rng.integers(1, 5)), atoms, 4, tail_p=0.0)
        R = len(offs) - 1
        nb = R * maxb
        bt_tab = np.arange(nb, dtype=np.int32).reshape(R, maxb)
        cache = np.zeros(L * 2 * nb * chunk, dtype=np.uint8)
        cv = cache_view(cache, L, nb, chunk)
        # the cache holds each block's payload as a function of its prefix
        for r in range(R):
            seq = toks[offs[r]:offs[r + 1]]
            for j in range(min(len(seq) // bt, maxb)):
                p = _payload_of(seq[:(j + 1) * bt], L * 2 * chunk).reshape(L, 2, chunk)
                cv[:, :, bt_tab[r, j]] = p
        rc, m, ids, created = o.insert(toks, offs, maxb)
        o.scatter(ids, created, bt_tab, cache, nb)
        # look up again and gather into a cleared cache
        m2, ids2 = o.lookup(toks, offs, maxb)
        assert (m2 == m).all() and (ids2 == ids).all()
        out = np.zeros_like(cache)
        o.gather(ids2, m2, bt_tab, out, nb)
        ov = cache_view(out, L, nb, chunk)
        for r in range(R):
            seq = toks[offs[r]:offs[r + 1]]
            for j in range(m2[r]):
                p = _payload_of(seq[:(j + 1) * bt], L * 2 * chunk).reshape(L, 2, chunk)
                assert (ov[:, :, bt_tab[r, j]] == p).all()
    assert o.evictions > 0


# --------------------------------------------------------------------------
# hot set (replication of popular prefixes)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
def test_hot_set_is_top_priorities(seed):
    """The oracle's hot set of an id range = the k nodes of the brute force with
    the highest H, ties to the smaller id (a plain sort of the definition)."""
    rng = np.random.default_rng(4000 + seed)
    bt, cap, maxb = 2, 12, 6
    atoms = _atoms(rng, 4, bt, 50)
    o = evict_store(bt, cap)
    b = brute.BruteEvictStore(bt, cap)
    for step in range(25):
        toks, offs = random_block_batch(rng, int(rng.integers(1, 7)), atoms, 6)
        if rng.random() < 0.5:
            o.lookup(toks, offs, maxb)
            b.lookup(toks, offs, maxb)
        else:
            o.insert(toks, offs, maxb)
            b.insert(toks, offs, maxb)
        stats = b.by_id()
        for lo, hi, k in ((0, cap, 3), (4, cap, 2), (2, 9, 5), (0, cap, cap + 3), (5, 6, 1)):
            pool = sorted((i for i in stats if lo <= i < hi), key=lambda i: (-stats[i][1], i))
            assert o.hot_set(lo, hi, k).tolist() == sorted(pool[:k]), (step, lo, hi, k)
