"""Seeded synthetic inputs shared by the tests, the bench and the smoke check.

This package draws token sequences, block tables and KV payloads. It holds
none of the prefix store's arithmetic (no hashing of blocks, no matching, no
id assignment): both the CPU oracle and the GPU path are fed from here and
compared with each other.
"""
from .synth import (  # noqa: F401
    KVShape,
    PassageWorkload,
    TrieWorkload,
    StreamRound,
    StreamWorkload,
    CONFIGS,
    concat_requests,
    zipf_probs,
    make_passage_workload,
    make_trie_workload,
    make_stream_workload,
    kv_payload_numpy,
)
