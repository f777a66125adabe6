"""Small helpers shared by the tests (no store arithmetic here)."""
from __future__ import annotations

import json
import os
from typing import Dict, List, Sequence, Tuple

import numpy as np

from workloads.synth import concat_requests

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_golden(name: str) -> dict:
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def spell(word: str, blocks: Dict[str, List[int]]) -> np.ndarray:
    """'AB+9' -> tokens of block A, block B, then the lone token 9."""
    if "+" in word:
        head, tail = word.split("+", 1)
        extra = [int(t) for t in tail.split(",") if t]
    else:
        head, extra = word, []
    toks: List[int] = []
    for ch in head:
        toks.extend(blocks[ch])
    toks.extend(extra)
    return np.asarray(toks, dtype=np.int32)


def spell_batch(words: Sequence[str], blocks) -> Tuple[np.ndarray, np.ndarray]:
    return concat_requests([spell(w, blocks) for w in words])


def random_block_batch(rng: np.random.Generator, n_req: int, atoms: np.ndarray, max_len: int,
                       tail_p: float = 0.3) -> Tuple[np.ndarray, np.ndarray]:
    """Requests made of blocks drawn from a small alphabet ``atoms`` [A, bt].

    A small alphabet makes shared prefixes, branches and repeats dense.
    Some requests get a partial trailing block.
    """
    bt = atoms.shape[1]
    seqs = []
    for _ in range(n_req):
        n = int(rng.integers(0, max_len + 1))
        pick = rng.integers(0, atoms.shape[0], size=n)
        s = atoms[pick].reshape(-1)
        if rng.random() < tail_p:
            s = np.concatenate([s, rng.integers(0, 5, size=int(rng.integers(1, bt)) if bt > 1 else 0,
                                                dtype=np.int32)])
        seqs.append(s.astype(np.int32))
    return concat_requests(seqs)


def block_table_identity(R: int, max_blocks: int) -> np.ndarray:
    return np.arange(R * max_blocks, dtype=np.int32).reshape(R, max_blocks)


def cache_view(cache: np.ndarray, layers: int, cache_blocks: int, chunk_bytes: int) -> np.ndarray:
    """[layer][K|V][cache block][chunk bytes] view of a flat paged cache."""
    return cache.reshape(layers, 2, cache_blocks, chunk_bytes)


def pool_view(pool: np.ndarray, layers: int, chunk_bytes: int) -> np.ndarray:
    """[id][layer][K|V][chunk bytes] view of a flat pool."""
    return pool.reshape(-1, layers, 2, chunk_bytes)
