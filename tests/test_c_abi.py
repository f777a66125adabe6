"""The C ABI used from plain C (tests/c/abi_demo.c): built on the CPU, run on the GPU."""
from __future__ import annotations

import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c", "abi_demo.c")
OUT_DIR = os.path.join(ROOT, "tests", "c", "_build")
EXE = os.path.join(OUT_DIR, "abi_demo")
LIBDIR = os.path.join(ROOT, "paper_2607_22648_amd")


def build_demo() -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include", SRC,
           "-L", LIBDIR, "-lptstore", "-L", "/opt/rocm/lib", "-lamdhip64",
           f"-Wl,-rpath,{LIBDIR}", "-Wl,-rpath,/opt/rocm/lib", "-o", EXE]
    subprocess.run(cmd, check=True)
    return EXE


def test_header_compiles_as_c_and_links():
    assert os.path.exists(build_demo())


@pytest.mark.gpu
def test_demo_runs_on_gpu():
    exe = build_demo()  # always against the current header and library
    p = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert p.returncode == 0, p.stderr
    assert "abi_demo ok" in p.stdout
