"""Brute-force definitions for tiny inputs (test infrastructure only).

Nothing here shares code with the C oracle: prefixes are whole token tuples
in a dict and a list, not trie nodes.

- ``lcp_blocks``: the longest common prefix, in whole blocks, of a request
  with every stored object, taken as a maximum over all of them (Section 4.1:
  the LCP is sought "among all previously stored objects").
- ``BruteStore.insert``: each distinct block-prefix is stored once (Section 1,
  redundancy-free growth) and gets the next id the first time it is seen in
  request order; a request inherits the ids of what is already stored and
  appends ids for its increment (Section 4.1).
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np


def request_blocks(tokens: np.ndarray, offsets: np.ndarray, r: int, block_tokens: int,
                   max_blocks: int) -> List[Tuple[int, ...]]:
    seq = tokens[offsets[r]:offsets[r + 1]]
    n = min(len(seq) // block_tokens, max_blocks)
    return [tuple(int(t) for t in seq[b * block_tokens:(b + 1) * block_tokens]) for b in range(n)]


def lcp_blocks(req: Sequence[Tuple[int, ...]], stored: Sequence[Sequence[Tuple[int, ...]]]) -> int:
    best = 0
    for s in stored:
        k = 0
        while k < len(req) and k < len(s) and req[k] == s[k]:
            k += 1
        best = max(best, k)
    return best


class BruteStore:
    def __init__(self, block_tokens: int, capacity: int):
        self.block_tokens = block_tokens
        self.capacity = capacity
        self.prefix_id: Dict[Tuple[Tuple[int, ...], ...], int] = {}
        self.objects: List[List[Tuple[int, ...]]] = []  # resident part of each inserted request

    @property
    def count(self) -> int:
        return len(self.prefix_id)

    def insert(self, tokens, offsets, max_blocks):
        R = len(offsets) - 1
        m = np.zeros(R, dtype=np.int32)
        ids = np.full((R, max_blocks), -1, dtype=np.int32)
        created = np.zeros((R, max_blocks), dtype=np.uint8)
        full = False
        for r in range(R):
            blocks = request_blocks(tokens, offsets, r, self.block_tokens, max_blocks)
            k = 0
            for b in range(len(blocks)):
                key = tuple(blocks[:b + 1])
                if key not in self.prefix_id:
                    if len(self.prefix_id) >= self.capacity:
                        full = True
                        break
                    self.prefix_id[key] = len(self.prefix_id)
                    created[r, b] = 1
                ids[r, b] = self.prefix_id[key]
                k = b + 1
            m[r] = k
            self.objects.append(blocks[:k])
        return full, m, ids, created

    def lookup(self, tokens, offsets, max_blocks):
        R = len(offsets) - 1
        m = np.zeros(R, dtype=np.int32)
        ids = np.full((R, max_blocks), -1, dtype=np.int32)
        for r in range(R):
            blocks = request_blocks(tokens, offsets, r, self.block_tokens, max_blocks)
            k = lcp_blocks(blocks, self.objects)
            m[r] = k
            for b in range(k):
                ids[r, b] = self.prefix_id[tuple(blocks[:b + 1])]
        return m, ids
