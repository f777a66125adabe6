"""Run the same store operations on the GPU library and the CPU oracle.

Every call goes through the C ABI on the GPU side and through the oracle on
the CPU side with the same seeded inputs; ``check_*`` compare outputs
element by element (all of this work is integer, index and copy work, so
the bar is bit-exact).
"""
from __future__ import annotations

from typing import Optional

import numpy as np
import torch

from oracle import OracleStore, ORC_ERR_FULL
from paper_2607_22648_amd.ptstore import PrefixStore, StoreShape, PTSTORE_FLAG_EVICT

DEV = torch.device("cuda:0")


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy()


def random_bytes(n: int, seed: int) -> torch.Tensor:
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return torch.randint(0, 256, (n,), dtype=torch.uint8, device=DEV, generator=g)


class Twin:
    def __init__(self, layers, kv_heads, head_dim, block_tokens, capacity, *, elem_bytes=2,
                 index_slots=0, hash_seed=0x5EED, flags=0, payload=True, host_blocks=0,
                 replica_blocks=0, layer_chunk_bytes=None):
        lcb = tuple(layer_chunk_bytes) if layer_chunk_bytes else None
        self.shape = StoreShape(layers, kv_heads, head_dim, block_tokens, elem_bytes, lcb)
        self.gpu = PrefixStore(self.shape, capacity, index_slots=index_slots, hash_seed=hash_seed,
                               flags=flags, host_blocks=host_blocks, replica_blocks=replica_blocks)
        cap = self.gpu.stats()["capacity"]
        self.evict = bool(flags & PTSTORE_FLAG_EVICT)
        self.ref = OracleStore(layers, kv_heads, head_dim, block_tokens, elem_bytes, cap, payload,
                               evict=self.evict, layer_chunk_bytes=lcb)
        self.capacity = cap
        self.payload = payload

    @classmethod
    def for_shape(cls, kv, capacity, **kw) -> "Twin":
        return cls(kv.layers, kv.kv_heads, kv.head_dim, kv.block_tokens, capacity,
                   elem_bytes=kv.elem_bytes, **kw)

    def close(self):
        self.gpu.close()
        self.ref.close()

    # ---- operations -------------------------------------------------------
    def insert(self, tokens: np.ndarray, offsets: np.ndarray, max_blocks: int, check=True):
        full0 = self.gpu.stats()["full_events"] if check else 0
        m, ids, created = self.gpu.insert(to_dev(tokens), to_dev(offsets), max_blocks)
        rc, rm, rids, rcr = self.ref.insert(tokens, offsets, max_blocks)
        if check:
            torch.cuda.synchronize()
            np.testing.assert_array_equal(host(m), rm, err_msg="insert m")
            np.testing.assert_array_equal(host(ids), rids, err_msg="insert ids")
            np.testing.assert_array_equal(host(created), rcr, err_msg="insert created")
            st = self.gpu.stats()
            assert st["blocks_stored"] == self.ref.count
            # a full event exactly when the oracle refused a block
            assert st["full_events"] - full0 == (1 if rc == ORC_ERR_FULL else 0)
        return (m, ids, created), (rc, rm, rids, rcr)

    def lookup(self, tokens, offsets, max_blocks, check=True):
        m, ids = self.gpu.lookup(to_dev(tokens), to_dev(offsets), max_blocks)
        rm, rids = self.ref.lookup(tokens, offsets, max_blocks)
        if check:
            torch.cuda.synchronize()
            np.testing.assert_array_equal(host(m), rm, err_msg="lookup m")
            np.testing.assert_array_equal(host(ids), rids, err_msg="lookup ids")
        return (m, ids), (rm, rids)

    def scatter_random(self, ids_dev, created_dev, rids, rcreated, block_table: np.ndarray,
                       seed: int, cache_blocks: Optional[int] = None, layers=None):
        """Fill a cache with seeded random bytes and scatter the created blocks
        (only layers[0] .. layers[1]-1 if given)."""
        nb = int(block_table.max()) + 1 if block_table.size else 1
        nb = max(nb, cache_blocks or 0)
        cache = random_bytes(nb * self.shape.block_bytes, seed)
        self.gpu.scatter(ids_dev, created_dev, to_dev(block_table), cache, layers=layers)
        self.ref.scatter(rids, rcreated, block_table, host(cache), nb, layers=layers)

    def lookup_gather(self, tokens, offsets, max_blocks, block_table: np.ndarray, cache_blocks: int,
                      sentinel=0xA5, check=True):
        n = cache_blocks * self.shape.block_bytes
        dst = torch.full((n,), sentinel, dtype=torch.uint8, device=DEV)
        m, ids = self.gpu.lookup_gather(to_dev(tokens), to_dev(offsets), max_blocks,
                                        to_dev(block_table), dst)
        rm, rids = self.ref.lookup(tokens, offsets, max_blocks)
        rdst = np.full(n, sentinel, dtype=np.uint8)
        self.ref.gather(rids, rm, block_table, rdst, cache_blocks)
        if check:
            torch.cuda.synchronize()
            np.testing.assert_array_equal(host(m), rm, err_msg="lookup_gather m")
            np.testing.assert_array_equal(host(ids), rids, err_msg="lookup_gather ids")
            got = host(dst)
            if not np.array_equal(got, rdst):
                bad = np.flatnonzero(got != rdst)
                raise AssertionError(f"gathered bytes differ at {bad.size} positions, first {bad[:8]}")
        return (m, ids, dst), (rm, rids, rdst)

    def gather_layers(self, m_dev, ids_dev, rm, rids, block_table: np.ndarray, cache_blocks: int,
                      layers, dst: Optional[torch.Tensor] = None, rdst: Optional[np.ndarray] = None,
                      sentinel=0xA5):
        """Gather layers[0] .. layers[1]-1 of already-looked-up blocks on both sides
        into caches (new sentinel-filled ones unless given) and compare all bytes."""
        n = cache_blocks * self.shape.block_bytes
        if dst is None:
            dst = torch.full((n,), sentinel, dtype=torch.uint8, device=DEV)
            rdst = np.full(n, sentinel, dtype=np.uint8)
        self.gpu.gather(ids_dev, m_dev, to_dev(block_table), dst, layers=layers)
        self.ref.gather(rids, rm, block_table, rdst, cache_blocks, layers=layers)
        torch.cuda.synchronize()
        got = host(dst)
        if not np.array_equal(got, rdst):
            bad = np.flatnonzero(got != rdst)
            raise AssertionError(f"layers {layers}: bytes differ at {bad.size} positions, first {bad[:8]}")
        return dst, rdst

    def check_pool(self):
        """Every block's home bytes (device or host tier) equal the oracle's pool."""
        torch.cuda.synchronize()
        n = self.ref.count
        got = host(self.gpu.block_bytes_of(np.arange(n)))
        exp = self.ref.pool()[:n]
        if not np.array_equal(got, exp):
            bad = np.flatnonzero((got != exp).any(axis=1))
            raise AssertionError(f"pool blocks differ: {bad[:10]} ({bad.size} blocks)")

    def check_meta(self):
        torch.cuda.synchronize()
        n = self.ref.count
        par, tok = self.gpu.meta_tensors()
        par, tok = host(par[:n]), host(tok[:n])
        for i in range(n):
            p, t = self.ref.node(i)
            assert par[i] == p, f"parent of {i}"
            np.testing.assert_array_equal(tok[i], t, err_msg=f"tokens of {i}")

    def check_evict(self):
        """Access counts, priorities, clock and eviction count equal the oracle's."""
        torch.cuda.synchronize()
        n = self.ref.count
        f, h = self.gpu.evict_tensors()
        f, h = host(f[:n]), host(h[:n])
        exp = np.array([self.ref.node_stats(i)[:2] for i in range(n)], dtype=np.int64).reshape(n, 2)
        np.testing.assert_array_equal(f, exp[:, 0], err_msg="access counts")
        np.testing.assert_array_equal(h, exp[:, 1], err_msg="priorities")
        st = self.gpu.stats()
        assert st["clock"] == self.ref.clock, (st["clock"], self.ref.clock)
        assert st["evictions"] == self.ref.evictions, (st["evictions"], self.ref.evictions)

    def check_replicas(self, hot_set=True):
        """Replica bytes equal their blocks' home bytes; right after a replicate,
        the replicated blocks are the oracle's hot set of the host tier."""
        torch.cuda.synchronize()
        st = self.gpu.stats()
        owned, R = st["device_blocks"], self.gpu._replicas
        rep = host(self.gpu.replica_map())
        have = np.flatnonzero(rep >= 0)
        assert len(have) == st["replicas"] <= R
        assert len(set(rep[have].tolist())) == len(have), "two blocks share a replica slot"
        if len(have):
            dev = self.gpu.pool_tensor()
            got = host(dev[torch.from_numpy(owned + rep[have].astype(np.int64)).to(DEV)])
            exp = host(self.gpu.block_bytes_of(owned + have))
            np.testing.assert_array_equal(got, exp, err_msg="replica bytes")
        if hot_set:
            want = self.ref.hot_set(owned, self.ref.count, R)
            np.testing.assert_array_equal(owned + have, want, err_msg="replica set")
