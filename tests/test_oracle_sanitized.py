"""The oracle's pins, run against a build of the oracle under AddressSanitizer
and UndefinedBehaviorSanitizer (host code on the CPU): an out-of-bounds
access, use after free, overflow of a signed integer or other undefined
behaviour in the oracle aborts the run instead of passing by luck."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

from oracle.ref import build_oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SANITIZE = ("-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer")


def _asan_runtime():
    out = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True)
    p = out.stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


@pytest.mark.skipif(_asan_runtime() is None, reason="gcc has no AddressSanitizer runtime")
def test_oracle_pins_under_sanitizers(tmp_path):
    lib = str(tmp_path / "libptstore_oracle_sanitized.so")
    build_oracle(lib, extra_flags=SANITIZE)
    # the sanitizer runtime goes first; any preload already set stays after it
    preload = ":".join(x for x in (_asan_runtime(), os.environ.get("LD_PRELOAD", "")) if x)
    env = dict(os.environ, LD_PRELOAD=preload, PTSTORE_ORACLE_LIB=lib,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    tests = ["tests/test_oracle.py", "tests/test_oracle_eviction.py", "tests/test_oracle_layers.py"]
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu", *tests], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=1200)
    assert r.returncode == 0, (r.stdout[-4000:], r.stderr[-4000:])
    assert " passed" in r.stdout
