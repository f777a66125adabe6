"""CPU oracle of the prefix store -- TEST INFRASTRUCTURE ONLY.

A plain single-threaded C implementation (``ptstore_oracle.c``: a pointer
trie compared token by token, plus ``memcpy``) behind a ctypes wrapper, and a
pure-Python brute force over whole prefixes for tiny inputs. Only the tests,
the smoke check and the bench's CPU-baseline leg may import this package; the
GPU library never links or calls it and shares no source with it.
"""
from .ref import OracleStore, build_oracle, ORC_OK, ORC_ERR_INVALID, ORC_ERR_FULL  # noqa: F401
from . import brute  # noqa: F401
