"""The C-ABI library loads and exports every function include/ptstore.h declares (no GPU)."""
from __future__ import annotations

import ctypes as C
import os
import re
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ptstore.h")
LIB = os.path.join(ROOT, "paper_2607_22648_amd", "libptstore.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ptstore_[a-z_]+)\s*\(", text)))


def test_header_declares_the_api():
    names = declared_functions()
    for n in ("ptstore_create", "ptstore_destroy", "ptstore_lookup", "ptstore_gather",
              "ptstore_lookup_gather", "ptstore_insert", "ptstore_scatter", "ptstore_stats"):
        assert n in names


def test_library_exports_every_declared_symbol():
    assert os.path.exists(LIB), "build the library first (__graft_entry__.build())"
    lib = C.CDLL(LIB)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_fails_loudly_without_the_library(tmp_path):
    """Importing the binding from a copy of the package that has no built
    library raises at import: there is no fallback path."""
    import shutil
    pkg = tmp_path / "paper_2607_22648_amd"
    pkg.mkdir()
    for f in ("__init__.py", "ptstore.py"):
        shutil.copy(os.path.join(ROOT, "paper_2607_22648_amd", f), pkg / f)
    code = ("import sys; sys.path.insert(0, %r)\n"
            "try:\n    from paper_2607_22648_amd import ptstore\n"
            "except ImportError as e:\n    print('ImportError', e)\n"
            "else:\n    print('loaded')\n") % str(tmp_path)
    out = subprocess.run(["python", "-c", code], capture_output=True, text=True, timeout=300,
                         cwd=str(tmp_path))
    assert out.returncode == 0, out.stderr
    assert out.stdout.startswith("ImportError") and "libptstore.so is missing" in out.stdout


def test_binding_names_match_header():
    from paper_2607_22648_amd import ptstore as P
    assert sorted(P.EXPORTS) == declared_functions()
    for n in P.EXPORTS:
        assert hasattr(P, n), n


def test_strerror_without_gpu():
    lib = C.CDLL(LIB)
    lib.ptstore_strerror.restype = C.c_char_p
    assert lib.ptstore_strerror(0) == b"ok"
    assert lib.ptstore_strerror(1) == b"invalid argument"


def _c_layout(tmp_path, struct, fields):
    """sizeof and offsetof of `fields` in `struct`, as gcc lays out the header."""
    lines = [f'printf("%zu\\n", sizeof({struct}));']
    lines += [f'printf("%zu\\n", offsetof({struct}, {f}));' for f in fields]
    src = tmp_path / "layout.c"
    src.write_text("#include <stddef.h>\n#include <stdio.h>\n#include \"ptstore.h\"\n"
                   "int main(void) {\n" + "\n".join(lines) + "\nreturn 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.dirname(HEADER), "-o", str(exe), str(src)],
                   check=True)
    out = [int(x) for x in subprocess.run([str(exe)], check=True, capture_output=True,
                                          text=True).stdout.split()]
    return out[0], out[1:]


def test_struct_layouts_match_header(tmp_path):
    """The ctypes mirrors have the size and field offsets gcc gives the C structs."""
    from paper_2607_22648_amd import ptstore as P
    for cls, name in ((P.ptstore_config_t, "ptstore_config_t"), (P.ptstore_stats_t, "ptstore_stats_t"),
                      (P.ptstore_buffers_t, "ptstore_buffers_t")):
        fields = [f for f, _ in cls._fields_]
        size, offs = _c_layout(tmp_path, name, fields)
        assert C.sizeof(cls) == size, name
        assert [getattr(cls, f).offset for f in fields] == offs, name



def test_create_refuses_bad_shapes_without_gpu():
    """Shape checks run on the host before any HIP call: slab sizes whose
    product overflows 64 bits, slabs over 1 GiB, pools beyond 2^56 bytes."""
    from paper_2607_22648_amd import ptstore as P
    lib = C.CDLL(LIB)
    lib.ptstore_last_error.restype = C.c_char_p

    def create(**kw):
        base = dict(num_layers=2, num_kv_heads=8, head_dim=128, block_tokens=16, elem_bytes=2,
                    pool_blocks=16, index_slots=0, hash_seed=1, flags=0, host_blocks=0,
                    replica_blocks=0, layer_chunk_bytes=None)
        base.update(kw)
        cfg = P.ptstore_config_t(**base)
        h = C.c_void_p()
        rc = lib.ptstore_create(C.byref(cfg), C.byref(h))
        return rc, h.value, lib.ptstore_last_error().decode()

    refused = [
        dict(num_layers=0), dict(num_layers=(1 << 20) + 1), dict(block_tokens=65),
        dict(elem_bytes=0), dict(pool_blocks=-1), dict(pool_blocks=1 << 31),
        # 2^16 * 64 * 2^21 * 2^21 = 2^64: zero in 64-bit arithmetic
        dict(num_kv_heads=1 << 16, block_tokens=64, head_dim=1 << 21, elem_bytes=1 << 21),
        # a 2 GiB slab
        dict(num_kv_heads=64, block_tokens=64, head_dim=1 << 16, elem_bytes=8),
        # 1 GiB slabs x 2^20 layers x 2^20 blocks = 2^71 bytes of pool
        dict(num_layers=1 << 20, num_kv_heads=1 << 14, block_tokens=16, head_dim=1 << 10,
             elem_bytes=4, pool_blocks=1 << 20),
        # the same blocks in a host tier
        dict(num_layers=1 << 20, num_kv_heads=1 << 14, block_tokens=16, head_dim=1 << 10,
             elem_bytes=4, pool_blocks=0, host_blocks=1 << 20),
        dict(replica_blocks=1),  # replicas need a host tier and eviction
        dict(index_slots=3),
        dict(num_kv_heads=1, block_tokens=8, head_dim=1, elem_bytes=1),  # 8-byte slab
    ]
    for kw in refused:
        rc, h, msg = create(**kw)
        assert rc == P.PTSTORE_ERR_INVALID and h is None, (kw, rc, msg)
        assert msg.startswith("ptstore_create"), (kw, msg)


def test_binding_checks_array_sizes_without_gpu():
    """The binding refuses arrays smaller than R and max_blocks require before
    anything reaches the library (which cannot see allocation sizes)."""
    import pytest
    import torch
    from paper_2607_22648_amd import ptstore as P
    offs = torch.tensor([0, 32, 64], dtype=torch.int64)
    toks = torch.zeros(64, dtype=torch.int32)
    m = torch.zeros(2, dtype=torch.int32)
    ids = torch.zeros((2, 4), dtype=torch.int32)
    with pytest.raises(ValueError, match="ids holds 7"):
        P.ptstore_lookup(None, toks, offs, 4, m, ids.view(-1)[:7])
    with pytest.raises(ValueError, match="m holds 1"):
        P.ptstore_lookup(None, toks, offs, 4, m[:1], ids)
    with pytest.raises(ValueError, match="block_table holds 4"):
        P.ptstore_gather(None, ids, m, ids[:1], None, 0)
    with pytest.raises(ValueError, match="created holds 6"):
        P.ptstore_scatter(None, ids, torch.zeros(6, dtype=torch.uint8), ids, None, 0)
    with pytest.raises(ValueError, match=r"must be \[R, max_blocks\]"):
        P.ptstore_gather(None, ids.view(-1), m, ids, None, 0)
    with pytest.raises(ValueError, match="created holds 4"):
        P.ptstore_insert(None, toks, offs, 4, m, ids, torch.zeros(4, dtype=torch.uint8))
    with pytest.raises(ValueError, match="block_table holds 2"):
        P.ptstore_lookup_gather(None, toks, offs, 4, m, ids, ids.view(-1)[:2], None, 0)
    with pytest.raises(ValueError, match="offsets"):
        P.ptstore_lookup(None, toks, offs[:0], 4, m, ids)


def test_binding_constants_match_header():
    """Every PTSTORE_* enum constant of the header (error codes, flags) has
    the same value in the binding, and the binding defines none the header
    lacks."""
    from paper_2607_22648_amd import ptstore as P
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    header = {n: int(v) for n, v in re.findall(r"\b(PTSTORE_[A-Z_]+)\s*=\s*(\d+)u?\b", text)}
    assert "PTSTORE_FLAG_WEAK_TAGS" in header and "PTSTORE_ERR_NOMEM" in header
    for n, v in header.items():
        assert getattr(P, n, None) == v, n
    binding = {n for n in dir(P) if re.fullmatch(r"PTSTORE_(ERR|FLAG|OK|NOALLOC)[A-Z_]*", n)}
    assert binding == set(header), binding ^ set(header)
