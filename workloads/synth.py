"""Seeded generators for the five prefix-store workloads.

Every workload is long-passage question answering in shape: a long shared
passage followed by a short request-specific suffix (the paper evaluates on
WikiQA and SQuAD, Section 6.1; neither dataset is used here, these synthetic
token streams stand in for them). Popularity of passages follows a finite Zipf
law P(rank k) ~ k^-s, k = 1..N (the paper samples documents with a power law,
Section 6.1, "Metrics"). Tokens are uniform int32 in [0, 32000).

All arrays are numpy. Token sequences of a batch are packed as CSR:
``tokens`` (int32, concatenated) and ``offsets`` (int64, length R+1).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import pandas as pd

VOCAB = 32000

@dataclass(frozen=True)
class KVShape:
    """Shape of the KV payload of one block of ``block_tokens`` tokens."""

    layers: int
    kv_heads: int
    head_dim: int
    block_tokens: int = 16
    dtype: str = "bf16"
    layer_kv_heads: Optional[Tuple[int, ...]] = None  # per-layer KV heads (hybrid models)

    @property
    def elem_bytes(self) -> int:
        return 2

    @property
    def layer_chunk_bytes(self) -> Optional[Tuple[int, ...]]:
        """Per-layer slab bytes when layers differ, else None."""
        if self.layer_kv_heads is None:
            return None
        return tuple(h * self.block_tokens * self.head_dim * self.elem_bytes
                     for h in self.layer_kv_heads)

    @property
    def chunk_bytes(self) -> int:
        """Bytes of one (layer, K|V) slab of a block: heads x slots x dim (layer 0's)."""
        if self.layer_kv_heads is not None:
            return self.layer_chunk_bytes[0]
        return self.kv_heads * self.block_tokens * self.head_dim * self.elem_bytes

    @property
    def block_bytes(self) -> int:
        if self.layer_kv_heads is not None:
            return 2 * sum(self.layer_chunk_bytes)
        return self.layers * 2 * self.chunk_bytes


def zipf_probs(n: int, s: float) -> np.ndarray:
    k = np.arange(1, n + 1, dtype=np.float64)
    p = k ** (-s)
    return p / p.sum()


def concat_requests(seqs: Sequence[np.ndarray]) -> Tuple[np.ndarray, np.ndarray]:
    """Pack a list of int32 token arrays into (tokens, offsets) CSR."""
    lens = np.array([len(s) for s in seqs], dtype=np.int64)
    offsets = np.zeros(len(seqs) + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    if len(seqs):
        tokens = np.concatenate([np.asarray(s, dtype=np.int32) for s in seqs])
    else:
        tokens = np.zeros(0, dtype=np.int32)
    return tokens.astype(np.int32, copy=False), offsets


def _fresh(rng: np.random.Generator, n: int) -> np.ndarray:
    return rng.integers(0, VOCAB, size=n, dtype=np.int32)


# ---------------------------------------------------------------------------
# Passage workloads (tiny, 8B-shaped, 70B-shaped shard)
# ---------------------------------------------------------------------------


@dataclass
class PassageWorkload:
    """Requests = Zipf-chosen passage + fresh suffix; store = some passages."""

    name: str
    shape: KVShape
    passages: np.ndarray  # [P, passage_tokens] int32; index i has rank i+1
    stored: np.ndarray  # passage indices held by the store, in insert order
    req_passage: np.ndarray  # [R] passage index behind each request
    tokens: np.ndarray  # requests, CSR
    offsets: np.ndarray
    sub_batch: int  # requests per lookup+gather call
    seed: int

    @property
    def n_requests(self) -> int:
        return len(self.offsets) - 1

    @property
    def max_blocks(self) -> int:
        lens = np.diff(self.offsets)
        return int(lens.max() // self.shape.block_tokens) if len(lens) else 0

    @property
    def passage_blocks(self) -> int:
        return self.passages.shape[1] // self.shape.block_tokens

    def store_batch(self) -> Tuple[np.ndarray, np.ndarray]:
        """The stored passages as an insert batch (tokens, offsets)."""
        return concat_requests([self.passages[i] for i in self.stored])

    def sub_batches(self) -> List[Tuple[int, int]]:
        R = self.n_requests
        return [(s, min(R, s + self.sub_batch)) for s in range(0, R, self.sub_batch)]

    def request_slice(self, lo: int, hi: int) -> Tuple[np.ndarray, np.ndarray]:
        o = self.offsets
        toks = self.tokens[o[lo]:o[hi]]
        return toks, (o[lo:hi + 1] - o[lo]).astype(np.int64)


def _draw_passages(rng, n_passages: int, passage_tokens: int, block_tokens: int) -> np.ndarray:
    """Uniform random passages, re-drawn until all first blocks differ."""
    P = _fresh(rng, n_passages * passage_tokens).reshape(n_passages, passage_tokens)
    seen: Dict[bytes, int] = {}
    for i in range(n_passages):
        while True:
            key = P[i, :block_tokens].tobytes()
            if key not in seen:
                seen[key] = i
                break
            P[i] = _fresh(rng, passage_tokens)
    return P


def make_passage_workload(
    name: str,
    shape: KVShape,
    n_passages: int,
    passage_tokens: int,
    suffix_tokens: int,
    n_requests: int,
    zipf_s: float,
    stored_ranks: Sequence[int],
    sub_batch: int,
    seed: int = 1234,
    store_order_seed: Optional[int] = None,
    tiers: Optional[dict] = None,
) -> PassageWorkload:
    rng = np.random.default_rng(seed)
    P = _draw_passages(rng, n_passages, passage_tokens, shape.block_tokens)
    probs = zipf_probs(n_passages, zipf_s)
    req_passage = rng.choice(n_passages, size=n_requests, p=probs).astype(np.int64)
    seqs = [np.concatenate([P[p], _fresh(rng, suffix_tokens)]) for p in req_passage]
    tokens, offsets = concat_requests(seqs)
    stored = np.asarray([r - 1 for r in stored_ranks], dtype=np.int64)
    if store_order_seed is not None:  # a store filled over time is not sorted by popularity
        stored = np.random.default_rng(store_order_seed).permutation(stored)
    w = PassageWorkload(name, shape, P, stored, req_passage, tokens, offsets, sub_batch, seed)
    w.tiers = tiers
    return w


# ---------------------------------------------------------------------------
# Divergent trie workload
# ---------------------------------------------------------------------------

_M64 = (1 << 64) - 1


def _splitmix64(x: np.ndarray) -> np.ndarray:
    """SplitMix64 finaliser (Steele, Lea, Flood 2014), vectorised over uint64."""
    with np.errstate(over="ignore"):
        z = (x + np.uint64(0x9E3779B97F4A7C15)).astype(np.uint64)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


@dataclass
class TrieWorkload:
    """Random walks down an implicit prefix tree.

    A tree node is named by a 64-bit path hash. Node ``h`` has ``fanout``
    children with probability ``branch_p`` and one child otherwise (a
    counter-based draw keyed by ``h``). Each child carries one block of
    tokens derived from its own path hash. A walk picks a child uniformly at
    every level for ``depth`` levels.
    """

    shape: KVShape
    depth: int
    branch_p: float
    fanout: int
    capacity: int  # stored blocks the store is filled to
    store_tokens: np.ndarray  # walks inserted into the store, CSR
    store_offsets: np.ndarray
    store_paths: np.ndarray  # [W, depth] uint64 path hash of each visited node
    tokens: np.ndarray  # request walks, CSR
    offsets: np.ndarray
    req_paths: np.ndarray  # [R, depth] uint64
    seed: int

    @property
    def n_requests(self) -> int:
        return len(self.offsets) - 1

    @property
    def max_blocks(self) -> int:
        return self.depth


def _trie_paths(root: np.uint64, n: int, depth: int, branch_p: float, fanout: int,
                rng: np.random.Generator) -> np.ndarray:
    """[n, depth] path hashes of n random walks from the root."""
    h = np.full(n, root, dtype=np.uint64)
    paths = np.empty((n, depth), dtype=np.uint64)
    thresh = np.uint64(int(branch_p * 2.0 ** 64) & _M64)
    for lvl in range(depth):
        u = _splitmix64(h ^ np.uint64(0xA0761D6478BD642F))
        nchild = np.where(u < thresh, fanout, 1).astype(np.int64)
        pick = (rng.random(n) * nchild).astype(np.int64)
        with np.errstate(over="ignore"):
            h = _splitmix64(h * np.uint64(0x100000001B3) + pick.astype(np.uint64) + np.uint64(1))
        paths[:, lvl] = h
    return paths


def _node_tokens(h: np.ndarray, block_tokens: int) -> np.ndarray:
    """The block of tokens a tree node carries, a function of its path hash."""
    tj = np.arange(1, block_tokens + 1, dtype=np.uint64) * np.uint64(0xD1B54A32D192ED03)
    t = _splitmix64(h.reshape(-1)[:, None] ^ tj[None, :])
    return (t % np.uint64(VOCAB)).astype(np.int32)


def _walk_tokens(paths: np.ndarray, block_tokens: int) -> np.ndarray:
    """Tokens of walks, [n * depth * block_tokens], computed once per distinct node."""
    codes, uniq = pd.factorize(paths.reshape(-1))
    table = _node_tokens(np.asarray(uniq, dtype=np.uint64), block_tokens)
    return table[codes].reshape(-1)


def make_trie_workload(
    shape: KVShape,
    n_requests: int = 8192,
    depth: int = 64,
    branch_p: float = 0.1,
    fanout: int = 4,
    capacity: int = 1_000_000,
    seed: int = 1234,
    chunk_walks: int = 65536,
) -> TrieWorkload:
    """Draw store walks until they visit at least ``capacity`` distinct nodes."""
    rng = np.random.default_rng(seed)
    root = np.uint64(int(rng.integers(0, 2**63)))
    chunks = []
    seen = pd.Index(np.zeros(0, dtype=np.uint64))
    distinct = 0
    while distinct < capacity:
        p = _trie_paths(root, chunk_walks, depth, branch_p, fanout, rng)
        chunks.append(p)
        seen = seen.append(pd.Index(pd.unique(p.reshape(-1)))).unique()
        distinct = len(seen)
    paths = np.concatenate(chunks)
    # keep only the walks needed to reach `capacity` distinct nodes in walk order
    first = ~pd.Index(paths.reshape(-1)).duplicated(keep="first")
    new_per_walk = first.reshape(paths.shape).sum(axis=1)
    W = int(np.searchsorted(np.cumsum(new_per_walk), capacity) + 1)
    paths = paths[:W]
    bt = shape.block_tokens
    store_tokens = _walk_tokens(paths, bt)
    store_offsets = np.arange(W + 1, dtype=np.int64) * (depth * bt)
    rp = _trie_paths(root, n_requests, depth, branch_p, fanout, rng)
    tokens = _walk_tokens(rp, bt)
    offsets = np.arange(n_requests + 1, dtype=np.int64) * (depth * bt)
    return TrieWorkload(shape, depth, branch_p, fanout, capacity, store_tokens, store_offsets,
                        paths, tokens, offsets, rp, seed)


# ---------------------------------------------------------------------------
# Streaming insert + lookup workload
# ---------------------------------------------------------------------------


@dataclass
class StreamRound:
    lookup_tokens: np.ndarray
    lookup_offsets: np.ndarray
    insert_tokens: np.ndarray
    insert_offsets: np.ndarray


@dataclass
class StreamWorkload:
    """Rounds of (lookups, inserts) on top of a passage store.

    Lookups: with probability 1/2 an earlier inserted sequence padded with
    fresh tokens to the request length, else passage + fresh question.
    Inserts: a stored sequence (Zipf by passage, then uniform among the
    sequences grown from it) cut at a uniform block depth d >= 1, extended
    with ``fresh_blocks`` = (lo, hi) fresh blocks, uniform in lo..hi (1 or 2
    by default; 32, a 512-token question, in the reading where every insert
    stores a whole question); with probability 1/4 an exact repeat of an
    earlier insert.
    """

    base: PassageWorkload
    rounds: List[StreamRound]
    pool_blocks: int
    seed: int


def make_stream_workload(base: PassageWorkload, n_rounds: int = 100, per_round: int = 128,
                         pool_blocks: int = 76293, seed: int = 4321,
                         repeat_p: float = 0.25, history_p: float = 0.5,
                         fresh_blocks: Tuple[int, int] = (1, 2)) -> StreamWorkload:
    rng = np.random.default_rng(seed)
    bt = base.shape.block_tokens
    req_len = int(np.diff(base.offsets).max())
    stored = list(base.stored)
    st_probs = zipf_probs(len(stored), 1.1)
    all_probs = zipf_probs(base.passages.shape[0], 1.1)
    suffix = req_len - base.passages.shape[1]
    branches: Dict[int, List[np.ndarray]] = {}
    history: List[np.ndarray] = []
    rounds: List[StreamRound] = []
    for _ in range(n_rounds):
        prev = list(history)
        lk: List[np.ndarray] = []
        for _ in range(per_round):
            if prev and rng.random() < history_p:
                s = prev[int(rng.integers(len(prev)))]
                pad = max(0, req_len - len(s))
                lk.append(np.concatenate([s, _fresh(rng, pad)]))
            else:
                p = int(rng.choice(len(all_probs), p=all_probs))
                lk.append(np.concatenate([base.passages[p], _fresh(rng, suffix)]))
        ins: List[np.ndarray] = []
        for _ in range(per_round):
            if history and rng.random() < repeat_p:
                s = history[int(rng.integers(len(history)))]
                ins.append(s.copy())
                continue
            p = stored[int(rng.choice(len(stored), p=st_probs))]
            cands = [base.passages[p]] + branches.get(p, [])
            src = cands[int(rng.integers(len(cands)))]
            nb = len(src) // bt
            d = int(rng.integers(1, nb + 1))
            k = int(rng.integers(fresh_blocks[0], fresh_blocks[1] + 1))
            s = np.concatenate([src[: d * bt], _fresh(rng, k * bt)])
            branches.setdefault(p, []).append(s)
            history.append(s)
            ins.append(s)
        lt, lo = concat_requests(lk)
        it, io = concat_requests(ins)
        rounds.append(StreamRound(lt, lo, it, io))
    return StreamWorkload(base, rounds, pool_blocks, seed)


# ---------------------------------------------------------------------------
# KV payload
# ---------------------------------------------------------------------------


def kv_payload_numpy(n_blocks: int, shape: KVShape, seed: int) -> np.ndarray:
    """``n_blocks`` blocks of N(0,1) KV in the shape's dtype, as raw bytes.

    Returns uint8 [n_blocks, block_bytes]. bf16 is fp32 with the low 16 bits
    dropped (the payload is opaque to the store; only its bytes matter).
    """
    rng = np.random.default_rng(seed)
    n = n_blocks * shape.block_bytes // 2
    x = rng.standard_normal(n, dtype=np.float32)
    if shape.dtype == "fp16":
        b = x.astype(np.float16).view(np.uint16)
    else:
        b = (x.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    return b.view(np.uint8).reshape(n_blocks, shape.block_bytes)


# ---------------------------------------------------------------------------
# The five configurations at full size
# ---------------------------------------------------------------------------

SHAPE_TINY = KVShape(2, 8, 128, 16, "fp16")
SHAPE_8B = KVShape(32, 8, 128, 16, "bf16")
SHAPE_70B = KVShape(80, 8, 128, 16, "bf16")
SHAPE_TRIE = KVShape(1, 8, 128, 16, "fp16")
# a hybrid 32-layer model: full-attention layers (8 KV heads) alternate with
# layers of 2 KV heads, so slabs alternate 32 KiB and 8 KiB (1.25 MiB blocks)
SHAPE_HYBRID = KVShape(32, 8, 128, 16, "bf16", layer_kv_heads=tuple([8, 2] * 16))

CONFIGS = {
    # 64 requests x 1024 tokens: one of 32 passages of 768 tokens (Zipf 1.0)
    # + 256 fresh tokens; store holds the 16 most popular passages.
    "tiny": dict(kind="passage", shape=SHAPE_TINY, n_passages=32, passage_tokens=768,
                 suffix_tokens=256, n_requests=64, zipf_s=1.0,
                 stored_ranks=list(range(1, 17)), sub_batch=64),
    # 256 requests x 4096 tokens: one of 512 passages of 3584 tokens (Zipf 1.1)
    # + 512 fresh tokens; store holds the 256 most popular passages.
    "llama8b": dict(kind="passage", shape=SHAPE_8B, n_passages=512, passage_tokens=3584,
                    suffix_tokens=512, n_requests=256, zipf_s=1.1,
                    stored_ranks=list(range(1, 257)), sub_batch=128),
    # 64 requests x 32768 tokens: one of 64 passages of 30720 tokens (Zipf 1.2)
    # + 2048 fresh tokens. The 32 most popular passages need 322 GB of KV, more
    # than one GPU holds; one GPU keeps the odd ranks 1,3,..,31 (half of a
    # two-way split of the store).
    "llama70b_shard": dict(kind="passage", shape=SHAPE_70B, n_passages=64, passage_tokens=30720,
                           suffix_tokens=2048, n_requests=64, zipf_s=1.2,
                           stored_ranks=list(range(1, 33, 2)), sub_batch=4),
    # The 8B-shaped workload on the hybrid shape (per-layer slab sizes).
    "hybrid8b": dict(kind="passage", shape=SHAPE_HYBRID, n_passages=512, passage_tokens=3584,
                     suffix_tokens=512, n_requests=256, zipf_s=1.1,
                     stored_ranks=list(range(1, 257)), sub_batch=128),
    # All 32 passages of the 70B-shaped configuration (322 GB) on one GPU:
    # 48,640 blocks (237.5 GiB) in device memory, one passage's worth of device
    # replica slots, the remaining 12,800 blocks (62.5 GiB) in pinned host
    # memory. Passages are inserted in a seeded random order, so hot ones can
    # land on the host tier; one request per call keeps the paged cache at
    # 10 GiB.
    "llama70b_full": dict(kind="passage", shape=SHAPE_70B, n_passages=64, passage_tokens=30720,
                          suffix_tokens=2048, n_requests=64, zipf_s=1.2,
                          stored_ranks=list(range(1, 33)), sub_batch=1, store_order_seed=7,
                          tiers=dict(device_blocks=48640, replica_blocks=1920, host_blocks=12800)),
    # 8192 walks of a 64-level tree (fanout 4 with p=0.1), store = 1M blocks.
    "trie": dict(kind="trie", shape=SHAPE_TRIE, n_requests=8192, depth=64, branch_p=0.1,
                 fanout=4, capacity=1_000_000),
    # 100 rounds of 128 lookups + 128 inserts on the 8B-shaped store, pool of
    # 160 GB (76,293 blocks of 2 MiB).
    "stream": dict(kind="stream", base="llama8b", n_rounds=100, per_round=128,
                   pool_blocks=76293),
    # the same with every insert storing a 512-token question (32 fresh
    # blocks): the pool fills within a few rounds and the store must evict.
    "stream_evict": dict(kind="stream", base="llama8b", n_rounds=100, per_round=128,
                         pool_blocks=76293, fresh_blocks=(32, 32)),
}


def build(name: str, seed: int = 1234, **override):
    """Build a named configuration; keyword overrides shrink it for tests."""
    cfg = dict(CONFIGS[name])
    kind = cfg.pop("kind")
    if kind == "passage":
        cfg.update(override)
        return make_passage_workload(name, seed=seed, **cfg)
    if kind == "trie":
        cfg.update(override)
        return make_trie_workload(seed=seed, **cfg)
    base_over = override.pop("base_override", {})
    base = build(cfg.pop("base"), seed=seed, **base_over)
    cfg.update(override)
    return make_stream_workload(base, seed=seed + 1, **cfg)
