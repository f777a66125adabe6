"""ctypes wrapper of the C oracle (test infrastructure only).

Each method follows the function of the same purpose in ``ptstore_oracle.c``;
see that file for which passage of the paper each one restates.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ptstore_oracle.c")
# PTSTORE_ORACLE_LIB names another build of the same source (the sanitized
# build a CPU test runs the pins against); the default is built on demand.
_LIB = os.environ.get("PTSTORE_ORACLE_LIB") or os.path.join(_HERE, "libptstore_oracle.so")
# library OracleStore loads when no path is given (the mutation tests swap it)
DEFAULT_LIB = _LIB

ORC_OK, ORC_ERR_INVALID, ORC_ERR_FULL, ORC_ERR_NOMEM = 0, 1, 2, 3


def build_oracle(out: str = _LIB, extra_flags=(), src: str = _SRC) -> str:
    """Compile the oracle with gcc into a shared library; returns its path.

    The library is written under a temporary name and renamed into place, so
    that a process loading it meanwhile never sees a partial file."""
    tmp = f"{out}.{os.getpid()}.tmp"
    cmd = ["gcc", "-O2", "-g", "-std=c99", "-Wall", "-Wextra", "-shared", "-fPIC",
           *extra_flags, "-o", tmp, src]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


_lib_cache = {}


def _load(path: str = _LIB):
    if path in _lib_cache:
        return _lib_cache[path]
    if path == _LIB and (not os.path.exists(path)
                         or os.path.getmtime(path) < os.path.getmtime(_SRC)):
        build_oracle(path)
    lib = C.CDLL(path)
    p, i32, i64, u8p = C.c_void_p, C.c_int32, C.c_int64, C.c_void_p
    lib.orc_create.restype = p
    lib.orc_create.argtypes = [i32, i32, i32, i32, i32, i64, i32]
    lib.orc_create_layers.restype = p
    lib.orc_create_layers.argtypes = [i32, i32, p, i64, i32]
    lib.orc_gather_layers.argtypes = [p, p, p, p, i32, i32, i32, i32, u8p, i64]
    lib.orc_scatter_layers.argtypes = [p, p, p, p, i32, i32, i32, i32, u8p, i64]
    lib.orc_gather_layers.restype = C.c_int
    lib.orc_scatter_layers.restype = C.c_int
    lib.orc_destroy.argtypes = [p]
    lib.orc_lookup.argtypes = [p, p, p, i32, i32, p, p]
    lib.orc_gather.argtypes = [p, p, p, p, i32, i32, u8p, i64]
    lib.orc_insert.argtypes = [p, p, p, i32, i32, p, p, p]
    lib.orc_scatter.argtypes = [p, p, p, p, i32, i32, u8p, i64]
    lib.orc_count.restype = i64
    lib.orc_count.argtypes = [p]
    lib.orc_bad_entries.restype = i64
    lib.orc_bad_entries.argtypes = [p]
    lib.orc_block_bytes.restype = i64
    lib.orc_block_bytes.argtypes = [p]
    lib.orc_pool.restype = C.POINTER(C.c_uint8)
    lib.orc_pool.argtypes = [p]
    lib.orc_node.argtypes = [p, i64, C.POINTER(C.c_int32), p]
    lib.orc_set_evict.argtypes = [p, i32]
    lib.orc_hot_set.restype = i64
    lib.orc_hot_set.argtypes = [p, i64, i64, i64, p]
    lib.orc_clock.restype = i64
    lib.orc_clock.argtypes = [p]
    lib.orc_evictions.restype = i64
    lib.orc_evictions.argtypes = [p]
    lib.orc_node_stats.argtypes = [p, i64, C.POINTER(C.c_int64), C.POINTER(C.c_int64),
                                   C.POINTER(C.c_int32), C.POINTER(C.c_int32)]
    for f in (lib.orc_lookup, lib.orc_gather, lib.orc_insert, lib.orc_scatter, lib.orc_node,
              lib.orc_node_stats):
        f.restype = C.c_int
    _lib_cache[path] = lib
    return lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


class OracleStore:
    """A store of ``capacity`` blocks of ``layers x 2 x heads x block_tokens x head_dim`` elements,
    or, with ``layer_chunk_bytes``, of ``layers x 2`` slabs whose size depends on the layer."""

    def __init__(self, layers: int, kv_heads: int, head_dim: int, block_tokens: int = 16,
                 elem_bytes: int = 2, capacity: int = 1 << 16, with_payload: bool = True,
                 lib_path: Optional[str] = None, evict: bool = False, layer_chunk_bytes=None):
        self._lib = _load(lib_path or DEFAULT_LIB)
        self.layers, self.kv_heads, self.head_dim = layers, kv_heads, head_dim
        self.block_tokens, self.elem_bytes, self.capacity = block_tokens, elem_bytes, capacity
        if layer_chunk_bytes is None:
            self.layer_chunk_bytes = [kv_heads * block_tokens * head_dim * elem_bytes] * layers
            self._h = self._lib.orc_create(layers, kv_heads, head_dim, block_tokens, elem_bytes,
                                           capacity, 1 if with_payload else 0)
        else:
            self.layer_chunk_bytes = [int(c) for c in layer_chunk_bytes]
            arr = np.asarray(self.layer_chunk_bytes, dtype=np.int64)
            self._h = self._lib.orc_create_layers(layers, block_tokens, _ptr(arr), capacity,
                                                  1 if with_payload else 0)
        self.chunk_bytes = self.layer_chunk_bytes[0]
        self.block_bytes = 2 * sum(self.layer_chunk_bytes)
        if not self._h:
            raise MemoryError("oracle store allocation failed")
        self.with_payload = with_payload
        self.evict = evict
        self._lib.orc_set_evict(self._h, 1 if evict else 0)

    @classmethod
    def for_shape(cls, shape, capacity: int, with_payload: bool = True, **kw) -> "OracleStore":
        kw.setdefault("layer_chunk_bytes", getattr(shape, "layer_chunk_bytes", None))
        return cls(shape.layers, shape.kv_heads, shape.head_dim, shape.block_tokens,
                   shape.elem_bytes, capacity, with_payload, **kw)

    def close(self):
        if self._h:
            self._lib.orc_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- the four operations -------------------------------------------------
    def lookup(self, tokens: np.ndarray, offsets: np.ndarray, max_blocks: int
               ) -> Tuple[np.ndarray, np.ndarray]:
        tokens = np.ascontiguousarray(tokens, dtype=np.int32)
        offsets = np.ascontiguousarray(offsets, dtype=np.int64)
        R = len(offsets) - 1
        m = np.zeros(R, dtype=np.int32)
        ids = np.zeros((R, max_blocks), dtype=np.int32)
        rc = self._lib.orc_lookup(self._h, _ptr(tokens), _ptr(offsets), R, max_blocks,
                                  _ptr(m), _ptr(ids))
        if rc:
            raise ValueError(f"orc_lookup failed: {rc}")
        return m, ids

    def insert(self, tokens: np.ndarray, offsets: np.ndarray, max_blocks: int
               ) -> Tuple[int, np.ndarray, np.ndarray, np.ndarray]:
        tokens = np.ascontiguousarray(tokens, dtype=np.int32)
        offsets = np.ascontiguousarray(offsets, dtype=np.int64)
        R = len(offsets) - 1
        m = np.zeros(R, dtype=np.int32)
        ids = np.zeros((R, max_blocks), dtype=np.int32)
        created = np.zeros((R, max_blocks), dtype=np.uint8)
        rc = self._lib.orc_insert(self._h, _ptr(tokens), _ptr(offsets), R, max_blocks,
                                  _ptr(m), _ptr(ids), _ptr(created))
        if rc not in (ORC_OK, ORC_ERR_FULL):
            raise ValueError(f"orc_insert failed: {rc}")
        return rc, m, ids, created

    def gather(self, ids: np.ndarray, m: np.ndarray, block_table: np.ndarray,
               cache: np.ndarray, cache_blocks: int, layers: Optional[Tuple[int, int]] = None) -> None:
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        m = np.ascontiguousarray(m, dtype=np.int32)
        bt = np.ascontiguousarray(block_table, dtype=np.int32)
        assert cache.dtype == np.uint8 and cache.flags.c_contiguous
        assert cache.size == cache_blocks * self.block_bytes
        R, maxb = ids.shape
        l0, l1 = layers if layers is not None else (0, self.layers)
        rc = self._lib.orc_gather_layers(self._h, _ptr(ids), _ptr(m), _ptr(bt), R, maxb, l0, l1,
                                         _ptr(cache), cache_blocks)
        if rc:
            raise ValueError(f"orc_gather failed: {rc}")

    def scatter(self, ids: np.ndarray, created: np.ndarray, block_table: np.ndarray,
                cache: np.ndarray, cache_blocks: int, layers: Optional[Tuple[int, int]] = None) -> None:
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        created = np.ascontiguousarray(created, dtype=np.uint8)
        bt = np.ascontiguousarray(block_table, dtype=np.int32)
        assert cache.dtype == np.uint8 and cache.flags.c_contiguous
        assert cache.size == cache_blocks * self.block_bytes
        R, maxb = ids.shape
        l0, l1 = layers if layers is not None else (0, self.layers)
        rc = self._lib.orc_scatter_layers(self._h, _ptr(ids), _ptr(created), _ptr(bt), R, maxb,
                                          l0, l1, _ptr(cache), cache_blocks)
        if rc:
            raise ValueError(f"orc_scatter failed: {rc}")

    # -- inspection ----------------------------------------------------------
    @property
    def count(self) -> int:
        return int(self._lib.orc_count(self._h))

    @property
    def bad_entries(self) -> int:
        return int(self._lib.orc_bad_entries(self._h))

    @property
    def clock(self) -> int:
        """Eviction clock L (the largest priority evicted so far)."""
        return int(self._lib.orc_clock(self._h))

    @property
    def evictions(self) -> int:
        return int(self._lib.orc_evictions(self._h))

    def hot_set(self, lo: int, hi: int, k: int) -> np.ndarray:
        """Ids in [lo, hi) of the k nodes with the highest priority (ties: smaller
        id), ascending."""
        out = np.zeros(max(k, 1), dtype=np.int32)
        n = int(self._lib.orc_hot_set(self._h, lo, hi, k, _ptr(out)))
        return out[:n].copy()

    def node_stats(self, node_id: int) -> Tuple[int, int, int, int]:
        """(frequency, priority, children holding an id, depth) of a node."""
        f, p = C.c_int64(0), C.c_int64(0)
        lc, d = C.c_int32(0), C.c_int32(0)
        rc = self._lib.orc_node_stats(self._h, node_id, C.byref(f), C.byref(p), C.byref(lc),
                                      C.byref(d))
        if rc:
            raise KeyError(node_id)
        return int(f.value), int(p.value), int(lc.value), int(d.value)

    def node(self, node_id: int) -> Tuple[int, np.ndarray]:
        parent = C.c_int32(0)
        toks = np.zeros(self.block_tokens, dtype=np.int32)
        rc = self._lib.orc_node(self._h, node_id, C.byref(parent), _ptr(toks))
        if rc:
            raise KeyError(node_id)
        return int(parent.value), toks

    def pool(self) -> np.ndarray:
        """The pool as a uint8 [capacity, block_bytes] view (no copy)."""
        if not self.with_payload:
            raise ValueError("store built without payload")
        p = self._lib.orc_pool(self._h)
        return np.ctypeslib.as_array(p, shape=(self.capacity * self.block_bytes,)).reshape(
            self.capacity, self.block_bytes)
