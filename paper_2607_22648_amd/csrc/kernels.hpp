// Launch interface between the host runtime (api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.hpp"

namespace ptsd {

// View of the store used by the lookup kernels (read-only but for the
// access counts).
struct IndexView {
    const Slot* slots;
    uint64_t slot_mask;
    const int32_t* parent;   // [capacity]
    const int32_t* tokens;   // [capacity][block_tokens]
    const HashTables* ht;
    DevState* state;
    uint64_t* freq;          // [capacity] access counts, or null: no accounting
    uint64_t* prio;          // [capacity] priorities H = L + F
    int32_t block_tokens;
    int32_t counters;        // 1: count probes and comparisons
};

// One block to move: physical row (see TierView) <-> cache block cb.
struct Pair {
    int32_t row;
    int32_t cb;
};

// Where block bytes live. Physical rows 0 .. dev_rows-1 are rows of the
// device pool (rows below `owned` are the home of ids below `owned`, the
// rest are replica slots); rows dev_rows + j are rows of the pinned host
// tier, the home of id owned + j.
struct TierView {
    uint8_t* host;        // host tier base (device-accessible), null if none
    int64_t owned;        // ids below live in device memory
    int64_t dev_rows;     // device pool rows: owned + replica slots
    int64_t host_blocks;
    int32_t* rep_of;      // [host_blocks] replica slot or -1; null without replicas
    int32_t* rep_id;      // [replicas] host-tier index (id - owned) held, or -1
    int64_t replicas;
    uint64_t* enter_mask; // [ceil(host_blocks / 64)] blocks entering the hot set
    int32_t* free_list;   // [replicas] free slots, ascending (replicate scratch)
    int32_t* enter_list;  // [replicas] entering host-tier indices, ascending
    Pair* copies;         // [replicas] {host row, replica row} to copy
};

// Most workgroups of a selection pass.
constexpr int kSelGroups = 256;

// Per-block eviction state and the scratch of the victim selection
// (allocated with the store when eviction is on).
struct EvictView {
    uint64_t* freq;     // [capacity] F
    uint64_t* prio;     // [capacity] H
    int32_t* live;      // [capacity] children that hold an id
    int32_t* prot;      // [capacity] last insert epoch (DevState::ev_epoch) whose batch
                        // matched the block
    int32_t* depth;     // [capacity] 0 for a child of the root
    uint64_t* nkey;     // [capacity] index key, to rebuild the index
    uint32_t* spos;     // [capacity] index slot, to delete the entry
    uint64_t* wmask;    // [words] victims of the running insert, one bit per id
    uint32_t* wcnt;     // [words] victims per word
    uint32_t* wbase;    // [words] exclusive scan of wcnt
    int32_t* victims;   // [capacity] freed ids, ascending
    uint32_t* hist;     // [kSelPasses][kSelBins] digit histograms
    uint64_t* part;     // [kSelGroups][8] per-workgroup partials of the range pass
    int64_t words;      // ceil(capacity / 64)
    int32_t on;         // 0: eviction disabled, nothing here is touched
    TierView tier;      // an evicted host-tier block loses its replica
};

struct Batch {
    const int32_t* tokens;
    const int64_t* offsets;
    int64_t n_tokens;
    int32_t R;
    int32_t max_blocks;
};

// lookup.hip
hipError_t launch_lookup(const IndexView& ix, const Batch& b, int32_t* m, int32_t* ids,
                         hipStream_t s);
hipError_t launch_hash_all(const IndexView& ix, const Batch& b, uint64_t* keys, hipStream_t s);

// copy.hip
struct CopyPlan {
    uint8_t* pool;
    int64_t block_bytes;
    int64_t chunk_bytes;
    int32_t chunks_per_block;  // 2 * layers
    int32_t chunks_per_group;  // chunks one copy unit moves
    int32_t threads;           // workgroup size of the copy kernel
    int32_t grid;              // workgroups of the copy kernel, 0 = chosen per call
    int32_t gather_grid;       // most workgroups of a gather (one per unit below that)
    int32_t loop_grid;         // workgroups of a looping (sparse) copy
    int32_t host_grid;         // workgroups of the looping copy of host-tier rows
    DevState* state;
    TierView tier;
    // per-layer slab sizes (null when every layer has chunk_bytes): the
    // device table lbase[l] = 2 * (sum of the slab sizes of layers 0..l-1),
    // L + 1 entries, and the host's copy of it
    const int64_t* lbase;
    const int64_t* lbase_host;
};

// Most layers a store with per-layer slab sizes may have.
constexpr int kMaxVarLayers = 1024;


// A block a gather reads once, and the cache blocks it writes it to:
// dests[base .. base + n), 1 <= n <= kSliceDests. 16-byte aligned, so that a
// kernel reads one with a single load.
struct alignas(16) Slice {
    int32_t row;
    int32_t base;
    int32_t n;
    int32_t pad;
};
constexpr int kSliceDests = 64;  // one per lane of a wave

// Descriptor list of one gather / scatter call: the blocks whose row is in
// device memory first (*total of them), then those whose row is in the host
// tier (*total_h), each part in (request, block) order. A gather turns it
// into slices: each distinct row once, with the cache blocks that need it
// (device-row slices from 0, host-row slices from *total, in the order of
// the first request that needs the row). The row table groups the list's
// entries by row; it sits at the start of the scratch, table_cap slots that
// every call leaves empty, and a call uses its first table_mask + 1.
struct CopyScratch {
    unsigned long long* tkey;    // [table_cap] (row + 1) << 32 | entries so far; 0: empty
    int32_t* tbase;              // [table_cap] where the row's cache blocks start in dests
    uint64_t table_mask;
    Pair* pairs;                 // [R * max_blocks]
    Slice* slices;               // [R * max_blocks]
    int32_t* dests;              // [R * max_blocks]
    int32_t* pslot;              // [R * max_blocks] table slot of each list entry
    int32_t* prank;              // [R * max_blocks] its place among the row's cache blocks
    int32_t* row_cnt;            // [R] device-row blocks of each request
    int32_t* row_cnt_h;          // [R] host-row blocks of each request
    int64_t* row_base;           // [R] exclusive scan of row_cnt
    int64_t* row_base_h;         // [R] exclusive scan of row_cnt_h
    unsigned long long* total;   // device-row pairs
    unsigned long long* total_h; // host-row pairs (after the device-row ones)
    unsigned long long* nslices;   // device-row slices
    unsigned long long* nslices_h; // host-row slices (from slices + *total)
    unsigned long long* ndests;    // cache blocks of device-row slices handed out
    unsigned long long* ndests_h;  // the same for host-row slices (from dests + *total)
};
// Row-table slots a call needs (a power of two >= 2 R max_blocks, at least
// 64), and the scratch bytes of a call after a table region of table_cap
// slots; the carve lays a call out in such a scratch.
uint64_t copy_table_slots(int32_t R, int32_t max_blocks);
size_t copy_scratch_bytes(int32_t R, int32_t max_blocks, uint64_t table_cap);
void copy_scratch_carve(void* base, int32_t R, int32_t max_blocks, uint64_t table_cap,
                        CopyScratch* out);
// Empty row table: zeroes the first `bytes` of a new scratch.
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);

hipError_t launch_gather_select(const CopyPlan& p, const CopyScratch& sc, const int32_t* ids,
                                const int32_t* m, const int32_t* block_table, int32_t R,
                                int32_t max_blocks, int64_t cache_blocks, hipStream_t s);
hipError_t launch_scatter_select(const CopyPlan& p, const CopyScratch& sc, const int32_t* ids,
                                 const uint8_t* created, const int32_t* block_table, int32_t R,
                                 int32_t max_blocks, int64_t cache_blocks, hipStream_t s);
// Copies of layers l0 .. l1-1 of the listed blocks.
hipError_t launch_gather_copy(const CopyPlan& p, const CopyScratch& sc, uint8_t* cache,
                              int64_t cache_blocks, int32_t R, int32_t max_blocks, int32_t l0,
                              int32_t l1, hipStream_t s);
hipError_t launch_scatter_copy(const CopyPlan& p, const CopyScratch& sc, const uint8_t* cache,
                               int64_t cache_blocks, int32_t R, int32_t max_blocks, int32_t l0,
                               int32_t l1, hipStream_t s);
// Whole-block copies between rows: pairs[k] = {source row, destination row}.
hipError_t launch_copy_rows(const CopyPlan& p, const Pair* pairs, const unsigned long long* total,
                            int64_t max_pairs, hipStream_t s);

// insert.hip
struct BatchEntry;  // defined in insert.hip
struct InsertScratch {
    uint64_t* keys;       // [R][max_blocks]
    int32_t* m0;          // [R] match length before the insert
    int32_t* label;       // [R][max_blocks] batch-table slot of each new block
    int32_t* cnt;         // [R] blocks each request is the first to need
    int32_t* base;        // [R] exclusive scan of cnt
    void* table;          // batch table, table_mask + 1 entries of 16 bytes
    uint64_t table_mask;
    unsigned int* collision;  // set when the fast claim must be redone exactly
};
size_t insert_scratch_bytes(int32_t R, int32_t max_blocks, uint64_t* table_entries);
void insert_scratch_carve(void* base, int32_t R, int32_t max_blocks, InsertScratch* out);

struct InsertTarget {
    Slot* slots;
    int32_t* parent;
    int32_t* tokens;
    int64_t capacity;
};
// An insert is enqueued in three parts: match (lookup .. id scan), then,
// with eviction on, launch_evict, then commit (assign, publish, accesses).
hipError_t launch_insert_match(const IndexView& ix, const InsertTarget& tgt, const EvictView& ev,
                               const Batch& b, const InsertScratch& sc, int32_t* m_out, int32_t* ids,
                               uint8_t* created, hipStream_t s);
hipError_t launch_insert_commit(const IndexView& ix, const InsertTarget& tgt, const EvictView& ev,
                                const Batch& b, const InsertScratch& sc, int32_t* m_out, int32_t* ids,
                                uint8_t* created, hipStream_t s);

// evict.hip: victim selection and index maintenance of an insert (between
// its match and its commit), and the accesses of its resident paths (at the
// end of its commit).
hipError_t launch_evict(const IndexView& ix, const InsertTarget& tgt, const EvictView& ev,
                        hipStream_t s);
hipError_t launch_touch_paths(const IndexView& ix, const EvictView& ev, const int32_t* m,
                              const int32_t* ids, int32_t R, int32_t max_blocks, hipStream_t s);

// evict.hip: make the replica slots hold the hot set of the host tier.
hipError_t launch_replicate(const IndexView& ix, const EvictView& ev, const CopyPlan& p,
                            hipStream_t s);

// api.hip helpers
hipError_t launch_fill_slots(Slot* slots, int64_t n, hipStream_t s);

}  // namespace ptsd
