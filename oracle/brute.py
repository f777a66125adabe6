"""Brute-force definitions for tiny inputs (test infrastructure only).

Nothing here shares code with the C oracle: prefixes are whole token tuples
in a dict and a list, not trie nodes.

- ``lcp_blocks``: the longest common prefix, in whole blocks, of a request
  with every stored object, taken as a maximum over all of them (Section 4.1:
  the LCP is taken over every object stored so far).
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


class BruteEvictStore:
    """Store with frequency-based leaf eviction, written from the definition.

    Nodes are whole prefixes (tuples of blocks) in a dict; a node is a leaf
    when no stored prefix is one block longer and starts with it. Section 4.1
    ("Access pattern-aware eviction policy") asks for frequency-based,
    GDSF-style eviction; the exact rules read from it:

    - an access of a node adds one to its frequency F and sets its priority
      to H = L + F, with L the clock (the largest priority evicted so far);
    - a lookup accesses every node of each request's match; an insert
      accesses every node of each request's resident path, after its
      evictions;
    - an insert that needs more ids than were never handed out evicts, one
      at a time, the unprotected leaf with the lowest (H, deeper first, id);
      the nodes matched by the batch are protected;
    - new prefixes take never-used ids first, then the freed ids from the
      smallest up, in order of first appearance in the batch.
    """

    def __init__(self, block_tokens: int, capacity: int):
        self.block_tokens = block_tokens
        self.capacity = capacity
        self.nodes: Dict[Tuple[Tuple[int, ...], ...], List[int]] = {}  # prefix -> [id, F, H]
        self.next_id = 0
        self.clock = 0
        self.evictions = 0
        self.last_victims: List[Tuple[Tuple[int, ...], ...]] = []  # in eviction order

    def _touch(self, key):
        rec = self.nodes[key]
        rec[1] += 1
        rec[2] = self.clock + rec[1]

    def _is_leaf(self, key) -> bool:
        n = len(key)
        return not any(len(k) == n + 1 and k[:n] == key for k in self.nodes)

    def by_id(self) -> Dict[int, Tuple[int, int, int]]:
        """id -> (F, H, depth) of every stored node."""
        return {rec[0]: (rec[1], rec[2], len(k) - 1) for k, rec in self.nodes.items()}

    def lookup(self, tokens, offsets, max_blocks):
        R = len(offsets) - 1
        m = np.zeros(R, dtype=np.int32)
        ids = np.full((R, max_blocks), -1, dtype=np.int32)
        for r in range(R):
            blocks = request_blocks(tokens, offsets, r, self.block_tokens, max_blocks)
            k = 0
            while k < len(blocks) and tuple(blocks[:k + 1]) in self.nodes:
                key = tuple(blocks[:k + 1])
                ids[r, k] = self.nodes[key][0]
                self._touch(key)
                k += 1
            m[r] = k
        return m, ids

    def insert(self, tokens, offsets, max_blocks):
        R = len(offsets) - 1
        paths, protected, new, creator = [], set(), [], {}
        for r in range(R):
            blocks = request_blocks(tokens, offsets, r, self.block_tokens, max_blocks)
            keys = [tuple(blocks[:b + 1]) for b in range(len(blocks))]
            for key in keys:
                if key in self.nodes:
                    protected.add(key)
                elif key not in creator:
                    creator[key] = r
                    new.append(key)
            paths.append(keys)
        fresh = self.capacity - self.next_id
        want = max(0, len(new) - fresh)
        self.last_victims = []
        freed = []
        while len(self.last_victims) < want:
            leaves = [k for k in self.nodes if k not in protected and self._is_leaf(k)]
            if not leaves:
                break
            v = min(leaves, key=lambda k: (self.nodes[k][2], -len(k), self.nodes[k][0]))
            self.clock = max(self.clock, self.nodes[v][2])
            self.last_victims.append(v)
            freed.append(self.nodes.pop(v)[0])
            self.evictions += 1
        freed.sort()
        avail = list(range(self.next_id, self.capacity)) + freed
        made = set()
        for k, key in enumerate(new):
            if k < len(avail):
                self.nodes[key] = [avail[k], 0, 0]
                made.add(key)
        self.next_id = min(self.capacity, self.next_id + len(new))
        m = np.zeros(R, dtype=np.int32)
        ids = np.full((R, max_blocks), -1, dtype=np.int32)
        created = np.zeros((R, max_blocks), dtype=np.uint8)
        for r, keys in enumerate(paths):
            k = 0
            while k < len(keys) and keys[k] in self.nodes:
                ids[r, k] = self.nodes[keys[k]][0]
                created[r, k] = 1 if (keys[k] in made and creator[keys[k]] == r) else 0
                k += 1
            m[r] = k
        for r, keys in enumerate(paths):
            for key in keys[:m[r]]:
                self._touch(key)
        full = len(made) < len(new)
        return full, m, ids, created
