"""Python binding of the C ABI in include/ptstore.h (argument marshalling only).

The functions carry the C names and forward device pointers of torch tensors
plus the current HIP stream; every step of the work runs in the HIP library
``libptstore.so``. If the library has not been built this module raises at
import time: there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libptstore.so")

PTSTORE_OK, PTSTORE_ERR_INVALID, PTSTORE_ERR_FULL, PTSTORE_ERR_HIP, PTSTORE_ERR_NOMEM = 0, 1, 2, 3, 4
PTSTORE_FLAG_WEAK_HASH, PTSTORE_FLAG_COUNTERS, PTSTORE_FLAG_TIMING = 1, 2, 4
PTSTORE_FLAG_EVICT = 8
PTSTORE_FLAG_WEAK_TAGS = 16
PTSTORE_NOALLOC_MAX_ENTRIES = 1 << 20
KIND_GATHER, KIND_LOOKUP, KIND_SCATTER, KIND_INSERT, KIND_SELECT, KIND_EVICT = 0, 1, 2, 3, 4, 5
KIND_REPLICATE = 6


class ptstore_config_t(C.Structure):
    _fields_ = [("num_layers", C.c_int32), ("num_kv_heads", C.c_int32), ("head_dim", C.c_int32),
                ("block_tokens", C.c_int32), ("elem_bytes", C.c_int32),
                ("pool_blocks", C.c_int64), ("index_slots", C.c_int64),
                ("hash_seed", C.c_uint64), ("flags", C.c_uint32),
                ("host_blocks", C.c_int64), ("replica_blocks", C.c_int64),
                ("layer_chunk_bytes", C.c_void_p)]


class ptstore_stats_t(C.Structure):
    _fields_ = [(n, C.c_int64) for n in (
        "blocks_stored", "capacity", "index_slots", "block_bytes", "chunk_bytes", "full_events",
        "bad_entries", "probes", "token_compares", "cas_attempts", "cas_failures",
        "insert_fallbacks", "evictions", "clock", "index_rebuilds", "device_blocks", "replicas",
        "replica_copies")]


class ptstore_buffers_t(C.Structure):
    _fields_ = [("pool", C.c_void_p), ("parent", C.c_void_p), ("tokens", C.c_void_p),
                ("slots", C.c_void_p), ("capacity", C.c_int64), ("index_slots", C.c_int64),
                ("freq", C.c_void_p), ("prio", C.c_void_p), ("host_pool", C.c_void_p),
                ("host_blocks", C.c_int64), ("device_blocks", C.c_int64), ("replica_of", C.c_void_p)]


class PTStoreError(RuntimeError):
    def __init__(self, fn: str, code: int, detail: str):
        super().__init__(f"{fn} failed: code {code} ({detail})")
        self.code = code


EXPORTS = ("ptstore_create", "ptstore_destroy", "ptstore_lookup", "ptstore_gather",
           "ptstore_lookup_gather", "ptstore_insert", "ptstore_scatter", "ptstore_stats",
           "ptstore_reset_counters", "ptstore_get_buffers", "ptstore_kernel_times",
           "ptstore_set_copy_shape", "ptstore_strerror", "ptstore_last_error",
           "ptstore_bandwidth_probe", "ptstore_replicate", "ptstore_gather_layers",
           "ptstore_scatter_layers", "ptstore_gather_prepare", "ptstore_gather_prepared",
           "ptstore_set_counters", "ptstore_set_timing", "ptstore_lookup_gather_noalloc",
           "ptstore_set_timing_kinds",
           "ptstore_insert_sync")


def _load() -> C.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it first (python -m "
                          "paper_2607_22648_amd.build or __graft_entry__.build())")
    lib = C.CDLL(LIB_PATH)
    p, i32, i64, d = C.c_void_p, C.c_int32, C.c_int64, C.c_double
    sig = {
        "ptstore_create": [C.POINTER(ptstore_config_t), C.POINTER(C.c_void_p)],
        "ptstore_destroy": [p],
        "ptstore_lookup": [p, p, p, i64, i32, i32, p, p, p],
        "ptstore_gather": [p, p, p, p, i32, i32, p, i64, p],
        "ptstore_lookup_gather": [p, p, p, i64, i32, i32, p, p, p, p, i64, p],
        "ptstore_lookup_gather_noalloc": [p, p, p, i64, i32, i32, p, p, p, p, i64, p],
        "ptstore_insert": [p, p, p, i64, i32, i32, p, p, p, p],
        "ptstore_insert_sync": [p, p, p, i64, i32, i32, p, p, p, p],
        "ptstore_scatter": [p, p, p, p, i32, i32, p, i64, p],
        "ptstore_stats": [p, C.POINTER(ptstore_stats_t)],
        "ptstore_reset_counters": [p],
        "ptstore_set_counters": [p, C.c_int],
        "ptstore_set_timing": [p, C.c_int],
        "ptstore_set_timing_kinds": [p, C.c_uint32],
        "ptstore_get_buffers": [p, C.POINTER(ptstore_buffers_t)],
        "ptstore_kernel_times": [p, i32, C.POINTER(d), C.POINTER(i64)],
        "ptstore_set_copy_shape": [p, i32, i32, i32],
        "ptstore_bandwidth_probe": [i32, p, p, i64, p],
        "ptstore_replicate": [p, p],
        "ptstore_gather_layers": [p, p, p, p, i32, i32, i32, i32, p, i64, p],
        "ptstore_scatter_layers": [p, p, p, p, i32, i32, i32, i32, p, i64, p],
        "ptstore_gather_prepare": [p, p, p, p, i32, i32, i64, p],
        "ptstore_gather_prepared": [p, i32, i32, p, i64, p],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = C.c_int
    lib.ptstore_strerror.argtypes = [C.c_int]
    lib.ptstore_strerror.restype = C.c_char_p
    lib.ptstore_last_error.argtypes = []
    lib.ptstore_last_error.restype = C.c_char_p
    return lib


_lib = _load()


def lib() -> C.CDLL:
    return _lib


def _check(fn: str, rc: int):
    if rc != PTSTORE_OK:
        raise PTStoreError(fn, rc, _lib.ptstore_last_error().decode())


def _dev(t: Optional[torch.Tensor], dtype, name: str) -> int:
    if t is None:
        return 0
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous device tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def _need(t: Optional[torch.Tensor], n: int, name: str) -> None:
    """The device arrays a call reads or writes are sized by R and max_blocks;
    the library cannot see an allocation's size, so it is checked here."""
    if t is None:
        if n:
            raise ValueError(f"{name} is required")
        return
    if t.numel() < n:
        raise ValueError(f"{name} holds {t.numel()} elements, the call needs {n}")


def _rows(ids: torch.Tensor, name: str = "ids") -> Tuple[int, int]:
    if ids.dim() != 2:
        raise ValueError(f"{name} must be [R, max_blocks], got shape {tuple(ids.shape)}")
    return int(ids.shape[0]), int(ids.shape[1])


def _requests(offsets: torch.Tensor) -> int:
    if offsets.dim() != 1 or offsets.numel() < 1:
        raise ValueError("offsets must be a 1-D tensor of R + 1 entries")
    return offsets.numel() - 1


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


# ---------------------------------------------------------------------------
# C entry points under their own names
# ---------------------------------------------------------------------------

def ptstore_create(cfg: ptstore_config_t) -> C.c_void_p:
    h = C.c_void_p()
    _check("ptstore_create", _lib.ptstore_create(C.byref(cfg), C.byref(h)))
    return h


def ptstore_destroy(h) -> None:
    _check("ptstore_destroy", _lib.ptstore_destroy(h))


def ptstore_lookup(h, tokens, offsets, max_blocks, m, ids, stream=None) -> None:
    R = _requests(offsets)
    _need(m, R, "m")
    _need(ids, R * max_blocks, "ids")
    _check("ptstore_lookup", _lib.ptstore_lookup(
        h, _dev(tokens, torch.int32, "tokens"), _dev(offsets, torch.int64, "offsets"),
        tokens.numel(), R, max_blocks, _dev(m, torch.int32, "m"), _dev(ids, torch.int32, "ids"),
        _stream(stream)))


def _cache_blocks(cache: torch.Tensor, block_bytes: int) -> int:
    """Cache blocks a flat paged cache holds (every layer's slabs of one block)."""
    nbytes = cache.numel() * cache.element_size()
    per = block_bytes
    if nbytes % per:
        raise ValueError("cache size is not a whole number of blocks")
    return nbytes // per


def ptstore_gather(h, ids, m, block_table, cache, cache_blocks, stream=None) -> None:
    R, maxb = _rows(ids)
    _need(m, R, "m")
    _need(block_table, R * maxb, "block_table")
    _check("ptstore_gather", _lib.ptstore_gather(
        h, _dev(ids, torch.int32, "ids"), _dev(m, torch.int32, "m"),
        _dev(block_table, torch.int32, "block_table"), R, maxb, _dev(cache, None, "cache"),
        cache_blocks, _stream(stream)))


def ptstore_gather_layers(h, ids, m, block_table, layer_begin, layer_end, cache, cache_blocks,
                          stream=None) -> None:
    R, maxb = _rows(ids)
    _need(m, R, "m")
    _need(block_table, R * maxb, "block_table")
    _check("ptstore_gather_layers", _lib.ptstore_gather_layers(
        h, _dev(ids, torch.int32, "ids"), _dev(m, torch.int32, "m"),
        _dev(block_table, torch.int32, "block_table"), R, maxb, layer_begin, layer_end,
        _dev(cache, None, "cache"), cache_blocks, _stream(stream)))


def ptstore_gather_prepare(h, ids, m, block_table, cache_blocks, stream=None) -> None:
    R, maxb = _rows(ids)
    _need(m, R, "m")
    _need(block_table, R * maxb, "block_table")
    _check("ptstore_gather_prepare", _lib.ptstore_gather_prepare(
        h, _dev(ids, torch.int32, "ids"), _dev(m, torch.int32, "m"),
        _dev(block_table, torch.int32, "block_table"), R, maxb, cache_blocks, _stream(stream)))


def ptstore_gather_prepared(h, layer_begin, layer_end, cache, cache_blocks, stream=None) -> None:
    _check("ptstore_gather_prepared", _lib.ptstore_gather_prepared(
        h, layer_begin, layer_end, _dev(cache, None, "cache"), cache_blocks, _stream(stream)))


def ptstore_scatter_layers(h, ids, created, block_table, layer_begin, layer_end, cache,
                           cache_blocks, stream=None) -> None:
    R, maxb = _rows(ids)
    _need(created, R * maxb, "created")
    _need(block_table, R * maxb, "block_table")
    _check("ptstore_scatter_layers", _lib.ptstore_scatter_layers(
        h, _dev(ids, torch.int32, "ids"), _dev(created, torch.uint8, "created"),
        _dev(block_table, torch.int32, "block_table"), R, maxb, layer_begin, layer_end,
        _dev(cache, None, "cache"), cache_blocks, _stream(stream)))


def ptstore_lookup_gather(h, tokens, offsets, max_blocks, m, ids, block_table, cache, cache_blocks,
                          stream=None) -> None:
    R = _requests(offsets)
    _need(m, R, "m")
    _need(ids, R * max_blocks, "ids")
    _need(block_table, R * max_blocks, "block_table")
    _check("ptstore_lookup_gather", _lib.ptstore_lookup_gather(
        h, _dev(tokens, torch.int32, "tokens"), _dev(offsets, torch.int64, "offsets"),
        tokens.numel(), R, max_blocks, _dev(m, torch.int32, "m"), _dev(ids, torch.int32, "ids"),
        _dev(block_table, torch.int32, "block_table"), _dev(cache, None, "cache"), cache_blocks,
        _stream(stream)))


def ptstore_lookup_gather_noalloc(h, tokens, offsets, max_blocks, m, ids, block_table, cache,
                                  cache_blocks, stream=None) -> None:
    R = _requests(offsets)
    _need(m, R, "m")
    _need(ids, R * max_blocks, "ids")
    _need(block_table, R * max_blocks, "block_table")
    _check("ptstore_lookup_gather_noalloc", _lib.ptstore_lookup_gather_noalloc(
        h, _dev(tokens, torch.int32, "tokens"), _dev(offsets, torch.int64, "offsets"),
        tokens.numel(), R, max_blocks, _dev(m, torch.int32, "m"), _dev(ids, torch.int32, "ids"),
        _dev(block_table, torch.int32, "block_table"), _dev(cache, None, "cache"), cache_blocks,
        _stream(stream)))


def ptstore_insert(h, tokens, offsets, max_blocks, m_out, ids, created, stream=None) -> None:
    R = _requests(offsets)
    _need(m_out, R, "m_out")
    _need(ids, R * max_blocks, "ids")
    _need(created, R * max_blocks, "created")
    _check("ptstore_insert", _lib.ptstore_insert(
        h, _dev(tokens, torch.int32, "tokens"), _dev(offsets, torch.int64, "offsets"),
        tokens.numel(), R, max_blocks, _dev(m_out, torch.int32, "m_out"),
        _dev(ids, torch.int32, "ids"), _dev(created, torch.uint8, "created"), _stream(stream)))


def ptstore_insert_sync(h, tokens, offsets, max_blocks, m_out, ids, created, stream=None) -> int:
    """Returns PTSTORE_OK, or PTSTORE_ERR_FULL when the insert refused blocks
    (its outputs are written either way); raises on any other error."""
    R = _requests(offsets)
    _need(m_out, R, "m_out")
    _need(ids, R * max_blocks, "ids")
    _need(created, R * max_blocks, "created")
    rc = _lib.ptstore_insert_sync(
        h, _dev(tokens, torch.int32, "tokens"), _dev(offsets, torch.int64, "offsets"),
        tokens.numel(), R, max_blocks, _dev(m_out, torch.int32, "m_out"),
        _dev(ids, torch.int32, "ids"), _dev(created, torch.uint8, "created"), _stream(stream))
    if rc != PTSTORE_ERR_FULL:
        _check("ptstore_insert_sync", rc)
    return rc


def ptstore_scatter(h, ids, created, block_table, cache, cache_blocks, stream=None) -> None:
    R, maxb = _rows(ids)
    _need(created, R * maxb, "created")
    _need(block_table, R * maxb, "block_table")
    _check("ptstore_scatter", _lib.ptstore_scatter(
        h, _dev(ids, torch.int32, "ids"), _dev(created, torch.uint8, "created"),
        _dev(block_table, torch.int32, "block_table"), R, maxb, _dev(cache, None, "cache"),
        cache_blocks, _stream(stream)))


def ptstore_stats(h) -> dict:
    s = ptstore_stats_t()
    _check("ptstore_stats", _lib.ptstore_stats(h, C.byref(s)))
    return {n: getattr(s, n) for n, _ in s._fields_}


def ptstore_replicate(h, stream=None) -> None:
    _check("ptstore_replicate", _lib.ptstore_replicate(h, _stream(stream)))


def ptstore_reset_counters(h) -> None:
    _check("ptstore_reset_counters", _lib.ptstore_reset_counters(h))


def ptstore_set_counters(h, on: bool) -> None:
    _check("ptstore_set_counters", _lib.ptstore_set_counters(h, 1 if on else 0))


def ptstore_set_timing(h, on: bool) -> None:
    _check("ptstore_set_timing", _lib.ptstore_set_timing(h, 1 if on else 0))


def ptstore_set_timing_kinds(h, kinds: int) -> None:
    _check("ptstore_set_timing_kinds", _lib.ptstore_set_timing_kinds(h, kinds))


def ptstore_get_buffers(h) -> ptstore_buffers_t:
    b = ptstore_buffers_t()
    _check("ptstore_get_buffers", _lib.ptstore_get_buffers(h, C.byref(b)))
    return b


def ptstore_kernel_times(h, kind: int) -> Tuple[float, int]:
    ms, n = C.c_double(), C.c_int64()
    _check("ptstore_kernel_times", _lib.ptstore_kernel_times(h, kind, C.byref(ms), C.byref(n)))
    return ms.value, n.value


def ptstore_set_copy_shape(h, chunks_per_group: int = 0, threads: int = 0, grid: int = 0) -> None:
    _check("ptstore_set_copy_shape", _lib.ptstore_set_copy_shape(h, chunks_per_group, threads,
                                                                  grid))


def ptstore_bandwidth_probe(kind: int, a, b, nbytes: int, stream=None) -> None:
    """a, b: device tensors, or integer addresses the device can access (such as
    the pinned host tier)."""
    pa = a if isinstance(a, int) else _dev(a, None, "a")
    pb = b if isinstance(b, int) else _dev(b, None, "b")
    _check("ptstore_bandwidth_probe", _lib.ptstore_bandwidth_probe(kind, pa, pb, nbytes,
                                                                   _stream(stream)))


def ptstore_strerror(code: int) -> str:
    return _lib.ptstore_strerror(code).decode()


def ptstore_last_error() -> str:
    return _lib.ptstore_last_error().decode()


# ---------------------------------------------------------------------------
# Convenience wrapper
# ---------------------------------------------------------------------------

@dataclass
class StoreShape:
    layers: int
    kv_heads: int
    head_dim: int
    block_tokens: int = 16
    elem_bytes: int = 2
    layer_chunk_bytes: Optional[Tuple[int, ...]] = None  # per-layer slab sizes, or uniform

    @property
    def chunk_bytes(self) -> int:
        """Slab bytes of layer 0 (of every layer when they are uniform)."""
        if self.layer_chunk_bytes:
            return int(self.layer_chunk_bytes[0])
        return self.kv_heads * self.block_tokens * self.head_dim * self.elem_bytes

    @property
    def block_bytes(self) -> int:
        if self.layer_chunk_bytes:
            return 2 * int(sum(self.layer_chunk_bytes))
        return self.layers * 2 * self.chunk_bytes


class PrefixStore:
    """A store on the current device; methods take device tensors."""

    def __init__(self, shape: StoreShape, pool_blocks: int, index_slots: int = 0,
                 hash_seed: int = 0x5EED, flags: int = 0, host_blocks: int = 0,
                 replica_blocks: int = 0):
        self.shape = shape
        lcb = None
        if shape.layer_chunk_bytes:
            lcb = (C.c_int64 * shape.layers)(*[int(x) for x in shape.layer_chunk_bytes])
        cfg = ptstore_config_t(shape.layers, shape.kv_heads, shape.head_dim, shape.block_tokens,
                               shape.elem_bytes, pool_blocks, index_slots, hash_seed, flags,
                               host_blocks, replica_blocks,
                               C.cast(lcb, C.c_void_p) if lcb is not None else None)
        self.h = ptstore_create(cfg)  # the slab-size array is read here and not kept
        self._replicas = replica_blocks

    def close(self):
        if getattr(self, "h", None):
            ptstore_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self) -> "PrefixStore":
        return self

    def __exit__(self, *exc) -> None:
        self.close()

    def cache_blocks(self, cache: torch.Tensor) -> int:
        return _cache_blocks(cache, self.shape.block_bytes)

    def lookup(self, tokens, offsets, max_blocks, m=None, ids=None, stream=None):
        R = offsets.numel() - 1
        dev = offsets.device
        m = torch.empty(R, dtype=torch.int32, device=dev) if m is None else m
        ids = torch.empty((R, max_blocks), dtype=torch.int32, device=dev) if ids is None else ids
        ptstore_lookup(self.h, tokens, offsets, max_blocks, m, ids, stream)
        return m, ids

    def gather(self, ids, m, block_table, cache, stream=None, layers=None):
        """layers = (begin, end): only those layers' slabs (None: all)."""
        if layers is None:
            ptstore_gather(self.h, ids, m, block_table, cache, self.cache_blocks(cache), stream)
        else:
            ptstore_gather_layers(self.h, ids, m, block_table, layers[0], layers[1], cache,
                                  self.cache_blocks(cache), stream)

    def lookup_gather(self, tokens, offsets, max_blocks, block_table, cache, m=None, ids=None,
                      stream=None):
        R = offsets.numel() - 1
        dev = offsets.device
        m = torch.empty(R, dtype=torch.int32, device=dev) if m is None else m
        ids = torch.empty((R, max_blocks), dtype=torch.int32, device=dev) if ids is None else ids
        ptstore_lookup_gather(self.h, tokens, offsets, max_blocks, m, ids, block_table, cache,
                              self.cache_blocks(cache), stream)
        return m, ids

    def lookup_gather_noalloc(self, tokens, offsets, max_blocks, block_table, cache, m, ids,
                              stream=None):
        """ptstore_lookup_gather_noalloc: the caller brings every output buffer."""
        ptstore_lookup_gather_noalloc(self.h, tokens, offsets, max_blocks, m, ids, block_table,
                                      cache, self.cache_blocks(cache), stream)
        return m, ids

    def insert(self, tokens, offsets, max_blocks, stream=None):
        R = offsets.numel() - 1
        dev = offsets.device
        m = torch.empty(R, dtype=torch.int32, device=dev)
        ids = torch.empty((R, max_blocks), dtype=torch.int32, device=dev)
        created = torch.empty((R, max_blocks), dtype=torch.uint8, device=dev)
        ptstore_insert(self.h, tokens, offsets, max_blocks, m, ids, created, stream)
        return m, ids, created

    def insert_sync(self, tokens, offsets, max_blocks, stream=None):
        """(rc, m, ids, created): rc is PTSTORE_OK or PTSTORE_ERR_FULL."""
        R = offsets.numel() - 1
        dev = offsets.device
        m = torch.empty(R, dtype=torch.int32, device=dev)
        ids = torch.empty((R, max_blocks), dtype=torch.int32, device=dev)
        created = torch.empty((R, max_blocks), dtype=torch.uint8, device=dev)
        rc = ptstore_insert_sync(self.h, tokens, offsets, max_blocks, m, ids, created, stream)
        return rc, m, ids, created

    def gather_prepare(self, ids, m, block_table, cache, stream=None):
        """List once the blocks a gather of (ids, m, block_table) into `cache` moves."""
        ptstore_gather_prepare(self.h, ids, m, block_table, self.cache_blocks(cache), stream)

    def gather_prepared(self, cache, layers, stream=None):
        """Copy layers[0] .. layers[1]-1 of the prepared blocks into `cache`."""
        ptstore_gather_prepared(self.h, layers[0], layers[1], cache, self.cache_blocks(cache), stream)

    def scatter(self, ids, created, block_table, cache, stream=None, layers=None):
        """layers = (begin, end): only those layers' slabs (None: all)."""
        if layers is None:
            ptstore_scatter(self.h, ids, created, block_table, cache, self.cache_blocks(cache),
                            stream)
        else:
            ptstore_scatter_layers(self.h, ids, created, block_table, layers[0], layers[1], cache,
                                   self.cache_blocks(cache), stream)

    def replicate(self, stream=None):
        ptstore_replicate(self.h, stream)

    def stats(self) -> dict:
        return ptstore_stats(self.h)

    def reset_counters(self):
        ptstore_reset_counters(self.h)

    def set_counters(self, on: bool):
        ptstore_set_counters(self.h, on)

    def set_timing(self, on: bool):
        ptstore_set_timing(self.h, on)

    def set_timing_kinds(self, kinds: int):
        """Events around the kernels of the kinds whose bit is set only."""
        ptstore_set_timing_kinds(self.h, kinds)

    def kernel_times(self, kind: int) -> Tuple[float, int]:
        return ptstore_kernel_times(self.h, kind)

    def set_copy_shape(self, chunks_per_group: int = 0, threads: int = 0, grid: int = 0):
        ptstore_set_copy_shape(self.h, chunks_per_group, threads, grid)

    def buffers(self) -> ptstore_buffers_t:
        return ptstore_get_buffers(self.h)

    def pool_tensor(self) -> torch.Tensor:
        """The device pool as a uint8 [rows, block_bytes] device tensor (no copy): the
        home of ids below device_blocks, then the replica slots."""
        b = self.buffers()
        rows = b.device_blocks + self._replicas
        n = rows * self.shape.block_bytes
        return _wrap_device(b.pool, n, torch.uint8).view(rows, self.shape.block_bytes)

    def host_tensor(self) -> torch.Tensor:
        """The pinned host tier as a uint8 [host_blocks, block_bytes] CPU tensor (no
        copy); row j holds block id device_blocks + j."""
        b = self.buffers()
        if not b.host_pool:
            raise ValueError("store has no host tier")
        n = b.host_blocks * self.shape.block_bytes
        arr = (C.c_uint8 * n).from_address(b.host_pool)
        return torch.frombuffer(arr, dtype=torch.uint8).view(b.host_blocks, self.shape.block_bytes)

    def block_bytes_of(self, ids) -> torch.Tensor:
        """Home bytes of the given block ids, [len(ids), block_bytes] on the device
        (device tier rows and host tier rows alike; a test helper)."""
        b = self.buffers()
        ids = torch.as_tensor(ids, dtype=torch.int64)
        dev = self.pool_tensor()
        on_dev = ids < b.device_blocks
        if bool(on_dev.all()):
            return dev[ids.to(dev.device)]
        out = torch.empty((ids.numel(), self.shape.block_bytes), dtype=torch.uint8, device=dev.device)
        if bool(on_dev.any()):
            out[on_dev.to(dev.device)] = dev[ids[on_dev].to(dev.device)]
        if bool((~on_dev).any()):
            torch.cuda.synchronize()  # host-tier rows are written by device kernels
            host = self.host_tensor()
            out[(~on_dev).to(dev.device)] = host[ids[~on_dev] - b.device_blocks].to(dev.device)
        return out

    def replica_map(self) -> torch.Tensor:
        """[host_blocks] int32 device tensor: replica slot of each host-tier block, or -1."""
        b = self.buffers()
        if not b.replica_of:
            raise ValueError("store has no replica slots")
        return _wrap_device(b.replica_of, b.host_blocks, torch.int32)

    def meta_tensors(self) -> Tuple[torch.Tensor, torch.Tensor]:
        """(parent [capacity] int32, tokens [capacity, block_tokens] int32), device, no copy."""
        b = self.buffers()
        par = _wrap_device(b.parent, b.capacity, torch.int32)
        tok = _wrap_device(b.tokens, b.capacity * self.shape.block_tokens, torch.int32)
        return par, tok.view(b.capacity, self.shape.block_tokens)

    def evict_tensors(self) -> Tuple[torch.Tensor, torch.Tensor]:
        """(access counts F, priorities H), each [capacity] int64, device, no copy
        (the values are unsigned 64-bit; they stay far below 2^63)."""
        b = self.buffers()
        if not b.freq:
            raise ValueError("store created without PTSTORE_FLAG_EVICT")
        return (_wrap_device(b.freq, b.capacity, torch.int64),
                _wrap_device(b.prio, b.capacity, torch.int64))


class _CudaArray:
    def __init__(self, ptr: int, n: int, typestr: str):
        self.__cuda_array_interface__ = {"shape": (n,), "typestr": typestr, "data": (ptr, False),
                                         "version": 2, "strides": None}


def _wrap_device(ptr: int, n: int, dtype) -> torch.Tensor:
    typestr = {torch.uint8: "|u1", torch.int32: "<i4", torch.int64: "<i8"}[dtype]
    return torch.as_tensor(_CudaArray(ptr, n, typestr), device="cuda")
