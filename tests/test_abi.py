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
