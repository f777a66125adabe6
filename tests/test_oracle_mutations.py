"""Planted mistakes in a copy of the oracle must each fail some pin.

Each mutant is the oracle's C source with one plausible slip (a dropped
term, a wrong index, a transposed layout, an off-by-one), compiled to a
temporary library. The pins of test_oracle.py run against it and at least
one must fail; this shows the pins would catch such a slip in the oracle
itself. All on the CPU; each mutant runs in a child process so that a
mutant which corrupts memory cannot take the test session down.
"""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

import oracle.ref as ref
from tests import test_oracle as pins
from tests import test_oracle_eviction as evpins
from tests import test_oracle_layers as lpins

MUTANTS = {
    "match_first_token_only": ("if (memcmp(c->tokens, blk, nbytes) == 0)",
                               "if (memcmp(c->tokens, blk, sizeof(int32_t)) == 0)"),
    "lookup_m_off_by_one": ("        m[r] = b;\n        for (int32_t j = b; j < max_blocks; j++) row[j] = -1;\n    }\n    return ORC_OK;",
                            "        m[r] = b > 0 ? b - 1 : 0;\n        for (int32_t j = b; j < max_blocks; j++) row[j] = -1;\n    }\n    return ORC_OK;"),
    "created_never_set": ("                crow[b] = 1;\n", "                crow[b] = 0;\n"),
    "capacity_off_by_one": ("if (s->count >= s->capacity) { full = 1; break; }",
                            "if (s->count + 1 >= s->capacity) { full = 1; break; }"),
    "cache_layout_transposed": ("return cache_blocks * s->lbase[l] + ((int64_t)kv * cache_blocks + cb) * s->chunk[l];",
                                "return cb * s->block_bytes + s->lbase[l] + (int64_t)kv * s->chunk[l];"),
    "pool_kv_layer_swapped": ("return id * s->block_bytes + s->lbase[l] + (int64_t)kv * s->chunk[l];",
                              "return id * s->block_bytes + (int64_t)kv * (s->block_bytes / 2) + s->lbase[l] / 2;"),
    "layer_base_off_by_one": ("s->lbase[l + 1] = s->lbase[l] + 2 * chunk_bytes[l];",
                              "s->lbase[l + 1] = s->lbase[l] + 2 * chunk_bytes[l > 0 ? l - 1 : 0];"),
    "layer_range_end_inclusive": ("            for (int32_t l = l0; l < l1; l++)\n                for (int32_t kv = 0; kv < 2; kv++)\n                    memcpy(cache",
                                  "            for (int32_t l = l0; l <= l1 && l < s->layers; l++)\n                for (int32_t kv = 0; kv < 2; kv++)\n                    memcpy(cache"),
    "partial_block_counted": ("int64_t n = len / s->block_tokens;",
                              "int64_t n = (len + s->block_tokens - 1) / s->block_tokens;"),
    "ids_start_at_one": ("c->id = (int32_t)s->count;", "c->id = (int32_t)s->count + 1;"),
    "scatter_every_occurrence": ("if (!created[k]) continue;", "if (ids[k] < 0) continue;"),
    "root_children_by_parent_ignored": ("        onode_t *node = &s->root;\n        int32_t b = 0;\n        for (; b < n; b++) {\n            const int32_t *blk",
                                        "        onode_t *node = &s->root;\n        int32_t b = 0;\n        for (; b < n; b++) {\n            node = &s->root;\n            const int32_t *blk"),
    # eviction mode
    "evict_ties_ignore_depth": ("    if (a->depth != b->depth) return a->depth > b->depth;\n", ""),
    "evict_clock_never_raised": ("if (best->prio > s->clock) s->clock = best->prio;", ";"),
    "evict_no_protection": ("c->protect = s->epoch;", "c->protect = 0;"),
    "evict_ids_in_eviction_order": ("qsort(victims, (size_t)nv, sizeof(int32_t), cmp_i32);", ";"),
    "evict_lookup_not_an_access": ("if (s->evict) touch(s, c);", ";"),
    "evict_plain_lfu": ("n->prio = s->clock + n->freq;", "n->prio = n->freq;"),
    "evict_no_cascade": ("if (best->parent != &s->root) best->parent->live_children--;", ";"),
    "hot_set_ties_to_larger_id": ("return (x->id > y->id) - (x->id < y->id);",
                                  "return (x->id < y->id) - (x->id > y->id);"),
    "evict_created_for_every_user": ("if (c->born == s->epoch && c->creator == r) crow[b] = 1;",
                                     "if (c->born == s->epoch) crow[b] = 1;"),
}

# pins that need no mutable global state; each gets a fresh store
PIN_CALLS = [
    lambda: [pins.test_golden_oracle(c) for c in pins.load_golden("incremental_ids.json")["cases"]],
    lambda: pins._check_against_brute(5, 2, 3, 4, 6, 6, 30, rounds=3, n_req=20),
    lambda: pins._check_against_brute(9, 16, 2, 4, 5, 4, 1000, rounds=3, n_req=20),
    lambda: pins._check_against_brute(8, 16, 3, 4, 8, 8, 1000, rounds=3, n_req=20, shared_head=True),
    pins.test_invariants_after_inserts,
    pins.test_gather_scatter_layout_and_sentinel,
    pins.test_ground_truth_tiny,
    pins.test_full_match_and_max_blocks_truncation,
    pins.test_capacity_zero,
    lambda: [evpins.test_golden_eviction_oracle(c) for c in pins.load_golden("eviction.json")["cases"]],
    lambda: [evpins.test_evict_random_vs_brute(k) for k in range(4)],
    lambda: [evpins.test_evict_invariants(k) for k in range(2)],
    lambda: [evpins.test_hot_set_is_top_priorities(k) for k in range(3)],
    lambda: lpins.test_variable_slabs_scatter_then_gather(lpins.CHUNKS),
    lambda: [lpins.test_layer_range_gather_writes_only_its_layers(a, b) for a, b in ((1, 3), (4, 5))],
]


def run_battery(lib: str) -> int:
    """Number of pins that fail against the library at ``lib``."""
    ref.DEFAULT_LIB = lib
    caught = 0
    for call in PIN_CALLS:
        try:
            call()
        except (AssertionError, KeyError, ValueError):
            caught += 1
    return caught


_CHILD = """
import sys
sys.path.insert(0, {root!r})
from tests import test_oracle_mutations as t
n = t.run_battery({lib!r})
print("CAUGHT", n)
"""


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(ref._SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    msrc = tmp_path / "mutant.c"
    msrc.write_text(src.replace(old, new))
    lib = str(tmp_path / "libmutant.so")
    ref.build_oracle(lib, src=str(msrc))
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    p = subprocess.run([sys.executable, "-c", _CHILD.format(root=root, lib=lib)],
                       capture_output=True, text=True, timeout=300)
    if p.returncode != 0:
        # the mutant crashed the child: it did not pass unnoticed either
        assert p.returncode != 0
        return
    line = [l for l in p.stdout.splitlines() if l.startswith("CAUGHT")][-1]
    assert int(line.split()[1]) > 0, f"no pin caught mutant {name}"


def test_unmutated_passes_battery():
    for call in PIN_CALLS:
        call()
