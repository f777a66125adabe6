/*
 * ptstore.h -- C ABI of the GPU-resident prefix store (MI355X / gfx950).
 *
 * The store keeps KV-cache prefixes at block granularity, each distinct
 * block-prefix exactly once, so that stored prefixes grow without redundancy
 * in divergent directions like a trie (PTStore, Section 1 "Contributions").
 * Every stored block has a dense unique id; an object's metadata is the flat
 * list of the ids on its path, inherited from its longest common prefix with
 * what is stored plus new ids for its own increment (Section 4.1,
 * "Co-optimized compact metadata and fast prefix queries"). The calls below
 * are the prefix query (LCP lookup), the load of the tensors behind a list
 * of ids into application-supplied GPU memory (gather), and the store of a
 * new object's increment (insert + scatter), as in Section 4.1 and the
 * client API of Section 5.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - A block is `block_tokens` consecutive int32 tokens. Only whole blocks
 *    count; a trailing partial block is never matched or stored. Only the
 *    first `max_blocks` blocks of a request are considered.
 *  - A batch of R requests is CSR: `tokens` (int32, device) and `offsets`
 *    (int64, device, R+1 entries); request r is tokens[offsets[r] ..
 *    offsets[r+1]). `n_tokens` is the length of `tokens`. A request whose
 *    offsets are decreasing, negative or beyond n_tokens is treated as empty
 *    and counted in `bad_entries`.
 *  - Per-(request, block) arrays are row-major [R][max_blocks].
 *  - KV payload of one block: [layer][K|V][head][slot][dim] elements of
 *    `elem_bytes` bytes; a (layer, K|V) slab of head*slot*dim elements is a
 *    "chunk". The store's pool is [pool_blocks][layer][K|V][head][slot][dim]
 *    (each block contiguous). The caller's paged cache is
 *    [layer][K|V][cache_blocks][head][slot][dim]. Payload bytes are copied
 *    verbatim: no arithmetic is done on them.
 *  - Every pointer argument except `cfg`/`out`/`stats` is a DEVICE pointer
 *    owned by the caller. `stream` is a hipStream_t (NULL = default stream).
 *    Calls only enqueue work on `stream` and return; outputs are valid once
 *    the stream has reached that point.
 *  - Streams: lookups and loads (lookup, gather, gather_layers,
 *    lookup_gather) may run on several streams of one store at once, up to
 *    16 streams per store: each stream has its own descriptor scratch. Every
 *    other call (insert, scatter, scatter_layers, replicate, gather_prepare,
 *    gather_prepared) must be ordered by the caller with respect to all
 *    other calls on the store (one stream, or events across streams); a
 *    lookup sees exactly the inserts ordered before it. Calls on one store
 *    come from one host thread at a time.
 *  - A call takes at most 2^29 (request, block) entries: R * max_blocks
 *    <= 2^29, else INVALID.
 *  - Return codes: PTSTORE_OK, or an error found on the host before any
 *    work is enqueued. Conditions only the device can see (a full store,
 *    out-of-range entries) are counted and reported by ptstore_stats();
 *    ptstore_insert_sync waits for its stream and returns PTSTORE_ERR_FULL
 *    when that insert refused blocks. Without waiting, a caller sees a cut
 *    in the outputs: request r was cut exactly when m_out[r] is below its
 *    number of whole blocks (at most max_blocks).
 *  - HIP graphs: once a call has grown the store's scratch to a batch size
 *    (for a load: the scratch of the capture's stream, or, for a capture
 *    stream that has made no call, that of the first stream that did),
 *    lookup, gather, gather_layers, lookup_gather, insert (with or without
 *    PTSTORE_FLAG_EVICT), scatter and scatter_layers of that size or
 *    smaller only launch kernels: no allocation, no wait, no memset. They
 *    may be captured and replayed; a replay works on the store as it is
 *    then. A later call with a larger batch regrows the scratch, after which
 *    earlier captures must not be replayed; a captured call that would need
 *    a larger scratch (or whose scratch a failed call left to be cleared
 *    by the next uncaptured call) returns INVALID and allocates nothing. A load captured
 *    on a stream that had made no call shares the first stream's scratch:
 *    its replays must not overlap loads enqueued on that stream. A capture
 *    keeps the counting state (ptstore_set_counters) it was made with.
 *    ptstore_lookup_gather_noalloc
 *    never allocates, whatever the batch (up to its limit).
 */
#ifndef PTSTORE_H
#define PTSTORE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ptstore ptstore_t;

enum {
    PTSTORE_OK = 0,
    PTSTORE_ERR_INVALID = 1, /* bad argument (null pointer, negative size, misaligned, ...) */
    PTSTORE_ERR_FULL = 2,    /* ptstore_insert_sync: the insert refused blocks for lack of room */
    PTSTORE_ERR_HIP = 3,     /* a HIP runtime call failed (see ptstore_last_error) */
    PTSTORE_ERR_NOMEM = 4    /* device or host allocation failed */
};

/* Configuration flags. */
enum {
    /* Mask index keys to 8 bits so that hash collisions are the rule: used
     * to test that results never depend on the hash (every hit is verified
     * on tokens and parent). Slow; for tests only. */
    PTSTORE_FLAG_WEAK_HASH = 1u,
    /* Count probes, token comparisons and compare-and-swap attempts. */
    PTSTORE_FLAG_COUNTERS = 2u,
    /* Record HIP events around every gather / scatter / lookup kernel so
     * that ptstore_kernel_times() can report their durations. */
    PTSTORE_FLAG_TIMING = 4u,
    /* Evict instead of refusing once the store is full (Section 4.1,
     * "Access pattern-aware eviction policy": frequency-based, GDSF adapted
     * to shared prefixes). Every lookup and insert counts accesses: an
     * access adds 1 to a block's frequency F and sets its priority
     * H = L + F, L being the store's clock. An insert that needs more new
     * blocks than the never-used ids left frees the difference first: it
     * evicts, one at a time, a block with no resident child that no request
     * of the batch matched, the one with the lowest H, then the deepest,
     * then the smallest id, and raises L to that block's H. What stays
     * resident is therefore always a set of whole prefixes. New blocks take
     * never-used ids first, then the freed ids from the smallest up; blocks
     * still without an id are refused as without this flag. Costs 44 bytes
     * of device memory per pool block. */
    PTSTORE_FLAG_EVICT = 8u,
    /* Name a new block in an insert's batch table by its key and only the
     * parity of its depth, so that blocks of one request at different
     * depths share entries: used to test that such sharing is detected and
     * the insert takes its exact path, with the same results. Slow; for
     * tests only. */
    PTSTORE_FLAG_WEAK_TAGS = 16u
};

typedef struct {
    int32_t num_layers;    /* L, 1 .. 2^20 */
    int32_t num_kv_heads;  /* H >= 1 */
    int32_t head_dim;      /* D >= 1 */
    int32_t block_tokens;  /* tokens per block, 1..64 */
    int32_t elem_bytes;    /* bytes per KV element (2 for fp16 / bf16) */
    int64_t pool_blocks;   /* blocks the pool can hold, 0 .. 2^31-4 */
    int64_t index_slots;   /* hash index slots (power of two) or 0 for
                              the smallest power of two >= 2*pool_blocks.
                              The store holds at most min(pool_blocks,
                              index_slots/2) blocks. */
    uint64_t hash_seed;    /* results never depend on it */
    uint32_t flags;        /* PTSTORE_FLAG_* */
    /* Tiers (Section 4.1, "Fine-grain multi-level caching" and "Replication
     * of popular prefixes"). Block ids 0 .. pool_blocks-replica_blocks-1
     * live in device memory; the next host_blocks ids live in pinned host
     * memory that the same copy kernels read and write over the host link.
     * replica_blocks of the pool_blocks device slots hold copies of hot
     * host-tier blocks (see ptstore_replicate); at most pool_blocks/2, and
     * only with PTSTORE_FLAG_EVICT (the hot set is ranked by its access
     * counts). Where a block's bytes are read from never changes a result. */
    int64_t host_blocks;     /* 0: no host tier */
    int64_t replica_blocks;  /* 0: no replicas */
    /* Per-layer slab sizes (Section 5: prefixes are combinations of tensors
     * of variable sizes): NULL, or num_layers (at most 1024) byte counts, each
     * a positive multiple of 16, read at create time. Layer l's K and V slabs of a block
     * are then layer_chunk_bytes[l] bytes each (num_kv_heads, head_dim and
     * elem_bytes are ignored); a pool block is layer after layer, and layer l
     * of the paged cache takes 2 * cache_blocks * layer_chunk_bytes[l] bytes
     * after all earlier layers, as [K|V][cache block][slab]. */
    const int64_t *layer_chunk_bytes;
} ptstore_config_t;

typedef struct {
    int64_t blocks_stored;  /* blocks (trie nodes) held, = next id */
    int64_t capacity;       /* maximum blocks_stored */
    int64_t index_slots;
    int64_t block_bytes;    /* L * 2 * H * block_tokens * D * elem_bytes (2 * sum of the
                               per-layer slab sizes when those are given) */
    int64_t chunk_bytes;    /* H * block_tokens * D * elem_bytes (layer 0's slab size
                               when per-layer sizes are given) */
    int64_t full_events;    /* inserts that refused blocks for lack of room */
    int64_t bad_entries;    /* skipped malformed requests, ids or cache blocks */
    int64_t probes;         /* index slots read (PTSTORE_FLAG_COUNTERS) */
    int64_t token_compares; /* candidate blocks compared token by token */
    int64_t cas_attempts;   /* compare-and-swap attempts by inserts */
    int64_t cas_failures;
    int64_t insert_fallbacks; /* inserts whose key collisions sent them to the exact
                                 sequential claim (results are the same either way) */
    int64_t evictions;      /* blocks evicted so far (PTSTORE_FLAG_EVICT) */
    int64_t clock;          /* eviction clock L: the largest priority evicted so far */
    int64_t index_rebuilds; /* times the index was rebuilt to clear deleted slots */
    int64_t device_blocks;  /* ids below this live in device memory */
    int64_t replicas;       /* host-tier blocks with a device copy now */
    int64_t replica_copies; /* blocks copied into replica slots so far */
} ptstore_stats_t;

/* Device buffers of a store, for inspection by tests (read-only use). */
typedef struct {
    void *pool;             /* [capacity][block_bytes] */
    const int32_t *parent;  /* [capacity] parent id, -1 for a root child */
    const int32_t *tokens;  /* [capacity][block_tokens] */
    const void *slots;      /* [index_slots] of {uint64 key, int32 id, int32 parent} */
    int64_t capacity;
    int64_t index_slots;
    const uint64_t *freq;   /* [capacity] access counts F (NULL without PTSTORE_FLAG_EVICT) */
    const uint64_t *prio;   /* [capacity] priorities H (NULL without PTSTORE_FLAG_EVICT) */
    void *host_pool;        /* [host_blocks][block_bytes] pinned host tier, or NULL; block
                               id device_blocks + j is row j. Device-accessible. */
    int64_t host_blocks;
    int64_t device_blocks;  /* ids below this are rows of `pool` */
    const int32_t *replica_of; /* [host_blocks] device replica slot of host-tier block j
                                  (its bytes are pool row device_blocks + slot), or -1 */
} ptstore_buffers_t;

/* ======================================================================
 * Store lifetime
 * ====================================================================== */

/*
 * Create a store on the current HIP device: allocates the pool, the block
 * metadata and the hash index, and waits until they are initialised.
 * On success *out owns them until ptstore_destroy(). Errors: INVALID (bad
 * shape, a (layer, K|V) slab not a multiple of 16 bytes or over 1 GiB, the
 * device pool or the host tier over 2^56 bytes, other sizes out of range;
 * returned before any HIP call), NOMEM, HIP.
 */
int ptstore_create(const ptstore_config_t *cfg, ptstore_t **out);

/* Wait for the device, then free everything the store owns. NULL is a no-op. */
int ptstore_destroy(ptstore_t *store);

/* ======================================================================
 * The prefix query and the load (Section 4.1; Section 5)
 * ====================================================================== */

/*
 * LCP query (Section 4.1): for each request r, m[r] = the largest k such that
 * its blocks 0..k-1 are a stored prefix (blocks beyond max_blocks ignored),
 * and ids[r][b] = the id of the stored block at depth b for b < m[r], -1
 * beyond. Outputs: m [R] int32, ids [R][max_blocks] int32. With
 * PTSTORE_FLAG_EVICT every matched block of every request counts one access.
 * Errors: INVALID (store NULL, R < 0, max_blocks < 1, R * max_blocks >
 * 2^29, n_tokens < 0 or >= 2^32, a NULL pointer with R > 0), HIP.
 */
int ptstore_lookup(ptstore_t *store, const int32_t *tokens, const int64_t *offsets,
                   int64_t n_tokens, int32_t R, int32_t max_blocks,
                   int32_t *m, int32_t *ids, void *stream);

/*
 * Load (Section 4.1: iterate over an object's ids and bring their tensors
 * into application-supplied GPU memory): for every r and b < m[r] with
 * block_table[r][b] >= 0, copy each (layer, K|V) chunk of pool block
 * ids[r][b] into cache[layer][K|V][block_table[r][b]]. Entries with an id
 * outside [0, blocks_stored) or a cache block >= cache_blocks are skipped
 * and counted in bad_entries. Destinations must be distinct (two entries
 * naming the same cache block race). `cache` must be 16-byte aligned.
 * The call first builds a dense list of the blocks to copy in store-owned
 * scratch of `stream` (about 60 bytes per (request, block) plus 24 per
 * request, grown on demand; growing waits for `stream`), then copies only
 * those blocks. With R >= 2 the list groups the entries by stored block, so
 * that a block several requests need is read once per call and written to
 * each of their cache blocks. Blocks read from device memory are copied on
 * the full device, blocks read from the host tier by a quarter of the
 * compute units (they move at the host link's rate whatever the grid, and
 * the rest of the device stays free for device-memory copies, of this call
 * or of loads on other streams). Errors: INVALID (store
 * NULL, R < 0, max_blocks < 1, R * max_blocks > 2^29, cache_blocks < 0, a
 * NULL pointer with R > 0, `cache` not 16-byte aligned), NOMEM (scratch),
 * HIP.
 */
int ptstore_gather(ptstore_t *store, const int32_t *ids, const int32_t *m,
                   const int32_t *block_table, int32_t R, int32_t max_blocks,
                   void *cache, int64_t cache_blocks, void *stream);

/*
 * The hot path of a prefix-cache hit: the LCP query, then the load of the
 * matched prefix's tensors into the caller's paged cache (Section 4.1: a
 * load finds the longest stored prefix and iterates over its ids; Section 5:
 * the client issues an LCP query, then reads the tensors it names).
 * ptstore_lookup followed by ptstore_gather of its result, enqueued back to
 * back on `stream`. m and ids are written as by ptstore_lookup.
 * Errors: those of either call.
 */
int ptstore_lookup_gather(ptstore_t *store, const int32_t *tokens, const int64_t *offsets,
                          int64_t n_tokens, int32_t R, int32_t max_blocks,
                          int32_t *m, int32_t *ids, const int32_t *block_table,
                          void *cache, int64_t cache_blocks, void *stream);

/* ======================================================================
 * The store of an increment (Sections 1 and 4; Section 4.1)
 * ====================================================================== */

/*
 * Store (Sections 1 and 4): with the same result as taking the requests one
 * after another, each request reuses the stored blocks of its longest
 * common prefix (including blocks created by earlier requests of this
 * batch) and creates one new block per missing block, ids handed out
 * densely in (request, block) order. Once the store holds `capacity`
 * blocks nothing more is created (with PTSTORE_FLAG_EVICT: once no block can
 * be evicted, see there); a request then keeps only the blocks it
 * could reuse or create (the cut is always a prefix), full_events is
 * incremented and ptstore_insert_sync would return PTSTORE_ERR_FULL. With
 * PTSTORE_FLAG_EVICT, after the evictions every block on each request's
 * resident path counts one access. Outputs: m_out [R] = blocks of r
 * resident after the call;
 * ids [R][max_blocks] their ids (-1 beyond m_out); created [R][max_blocks]
 * = 1 exactly where request r created the block (a block shared by several
 * requests of the batch is created by the first of them).
 * Uses store-owned scratch sized for R * max_blocks, grown on demand (the
 * growth waits for `stream`). Errors as ptstore_lookup, plus NOMEM.
 */
int ptstore_insert(ptstore_t *store, const int32_t *tokens, const int64_t *offsets,
                   int64_t n_tokens, int32_t R, int32_t max_blocks,
                   int32_t *m_out, int32_t *ids, uint8_t *created, void *stream);

/*
 * ptstore_insert, then wait for `stream` and report whether that insert
 * refused blocks for lack of room (the capacity cut of ptstore_insert;
 * with PTSTORE_FLAG_EVICT, blocks left after every possible eviction).
 * Returns PTSTORE_ERR_FULL in that case, with every output written as
 * ptstore_insert writes it (the cut is a prefix of each request, the same
 * as the one-after-another insert gives), else PTSTORE_OK.
 * Errors: those of ptstore_insert, HIP; INVALID when `stream` is being
 * captured into a graph (nothing is enqueued; capture ptstore_insert).
 */
int ptstore_insert_sync(ptstore_t *store, const int32_t *tokens, const int64_t *offsets,
                        int64_t n_tokens, int32_t R, int32_t max_blocks,
                        int32_t *m_out, int32_t *ids, uint8_t *created, void *stream);

/*
 * Store the tensors of new blocks (Section 4: a store saves only the
 * increment beyond the longest common prefix; Section 4.1: the application
 * supplies pointers to the GPU memory holding the tensors of the object to
 * store): for every (r, b) with created[r][b] != 0 and block_table[r][b] >= 0,
 * copy each chunk of cache[layer][K|V][block_table[r][b]] into pool block
 * ids[r][b] (its home row: device pool or host tier). Out-of-range ids /
 * cache blocks are skipped and counted in bad_entries. Uses the same
 * store-owned descriptor scratch as ptstore_gather. The pool is not cleared
 * when the store is made, and an evicted id keeps its old bytes: a block's
 * tensors (or the layers of them ptstore_scatter_layers did not write) are
 * undefined until a scatter writes them, and a gather of them copies
 * whatever the row holds. Errors as ptstore_gather.
 */
int ptstore_scatter(ptstore_t *store, const int32_t *ids, const uint8_t *created,
                    const int32_t *block_table, int32_t R, int32_t max_blocks,
                    const void *cache, int64_t cache_blocks, void *stream);

/* ======================================================================
 * Layer granularity (Section 4.1: transfers overlap computation;
 * Section 5: subsets of tensors, tensors of variable sizes)
 * ====================================================================== */

/*
 * Load of a range of layers (Section 4.1: transfers overlap computation;
 * Section 5: clients read subsets of tensors): as ptstore_gather, but only
 * the K and V slabs of layers layer_begin .. layer_end-1 are copied; the
 * cache's other layers are not touched. A caller can so bring in layer l+1
 * while it computes on layer l. Errors as ptstore_gather, plus INVALID
 * unless 0 <= layer_begin < layer_end <= num_layers.
 */
int ptstore_gather_layers(ptstore_t *store, const int32_t *ids, const int32_t *m,
                          const int32_t *block_table, int32_t R, int32_t max_blocks,
                          int32_t layer_begin, int32_t layer_end, void *cache,
                          int64_t cache_blocks, void *stream);

/*
 * A load in layer steps without rebuilding its block list each step.
 * ptstore_gather_prepare lists, once, the blocks a gather of (ids, m,
 * block_table) moves (bad entries are counted here); each
 * ptstore_gather_prepared then copies layers layer_begin .. layer_end-1 of
 * those blocks into `cache`, exactly as ptstore_gather_layers with the
 * prepare's arguments would. The list lives in the scratch of the prepare's
 * stream (a prepared copy on another stream must be ordered after it); any
 * other call on the store except lookups (gather, gather_layers,
 * lookup_gather, scatter, scatter_layers, insert, replicate) discards it.
 * ptstore_gather_prepared returns INVALID when there is no list, or when
 * cache_blocks differs from the prepare's.
 */
int ptstore_gather_prepare(ptstore_t *store, const int32_t *ids, const int32_t *m,
                           const int32_t *block_table, int32_t R, int32_t max_blocks,
                           int64_t cache_blocks, void *stream);
int ptstore_gather_prepared(ptstore_t *store, int32_t layer_begin, int32_t layer_end, void *cache,
                            int64_t cache_blocks, void *stream);

/*
 * Store the tensors of a range of layers of new blocks (a prefill can hand
 * each layer's KV to the store as soon as it is computed): as
 * ptstore_scatter, but only layers layer_begin .. layer_end-1. Errors as
 * ptstore_scatter, plus INVALID for a bad range. A block's replica, if any,
 * is dropped as by ptstore_scatter.
 */
int ptstore_scatter_layers(ptstore_t *store, const int32_t *ids, const uint8_t *created,
                           const int32_t *block_table, int32_t R, int32_t max_blocks,
                           int32_t layer_begin, int32_t layer_end, const void *cache,
                           int64_t cache_blocks, void *stream);

/* ======================================================================
 * Tiers and replication (Section 4.1)
 * ====================================================================== */

/*
 * Replication of popular prefixes (Section 4.1): make the device replica
 * slots hold exactly the hot set of the host tier -- the replica_blocks
 * host-tier blocks with the highest priority H, ties going to the smaller
 * id. Replicas that left the hot set free their slots; blocks that entered
 * it are copied from host memory into free slots (lowest slot to lowest id).
 * Gathers then read those blocks from device memory. A scatter into a block
 * drops its replica; an eviction too. Enqueued on `stream`; errors: INVALID
 * (no replica tier), HIP.
 */
int ptstore_replicate(ptstore_t *store, void *stream);

/* ======================================================================
 * Status
 * ====================================================================== */

/*
 * Wait for the device and read the store's counters into *stats: what it
 * holds, and the conditions only the device sees while running the calls
 * above (blocks refused for lack of room, the Section 4.1 capacity limit;
 * skipped malformed entries; evictions and the eviction clock of Section 4.1's
 * access-pattern-aware policy; replicas). Errors: INVALID (a NULL argument),
 * HIP.
 */
int ptstore_stats(ptstore_t *store, ptstore_stats_t *stats);

/* Human-readable text for a return code. */
const char *ptstore_strerror(int code);

/* Text of the last error on this host thread ("" if none). */
const char *ptstore_last_error(void);

/* ======================================================================
 * Allocation-free variant (for callers that cannot allocate)
 * ====================================================================== */

/*
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, kernels and results as ptstore_lookup_gather, but the
 * gather's descriptor list and the row table that groups its entries by
 * stored block live in a static device array of the library (about 84 MiB
 * per device, held until the process ends) instead of store-owned scratch.
 * The call allocates nothing, frees nothing, creates no event and never
 * waits; it records no ptstore_kernel_times() entries and leaves a list
 * made by ptstore_gather_prepare intact.
 * Limit: R * max_blocks <= PTSTORE_NOALLOC_MAX_ENTRIES, else INVALID before
 * any work is enqueued. Every such call on one device shares that device's
 * array, whichever store it names: calls that overlap in time on one device
 * (other streams, other threads) race and must be ordered by the caller.
 * Errors: those of ptstore_lookup_gather (NOMEM excepted), plus INVALID for
 * a batch over the limit or a device index of 64 or more.
 */
enum { PTSTORE_NOALLOC_MAX_ENTRIES = 1048576 /* 2^20 (request, block) entries */ };
int ptstore_lookup_gather_noalloc(ptstore_t *store, const int32_t *tokens, const int64_t *offsets,
                                  int64_t n_tokens, int32_t R, int32_t max_blocks,
                                  int32_t *m, int32_t *ids, const int32_t *block_table,
                                  void *cache, int64_t cache_blocks, void *stream);

/* ======================================================================
 * Tuning and diagnostics: not store operations. Counters, timing, the
 * store's buffers for tests, copy launch shapes, and a bandwidth probe.
 * ====================================================================== */

/* Zero the event counters (probes, compares, CAS, full_events, bad_entries,
 * insert_fallbacks, index_rebuilds); blocks_stored, evictions and the clock
 * are state and stay. Waits for the device. Errors: INVALID (NULL), HIP. */
int ptstore_reset_counters(ptstore_t *store);

/* Turn the event counters (probes, token compares, CAS attempts and
 * failures) on (on != 0) or off for the calls enqueued after this one;
 * PTSTORE_FLAG_COUNTERS sets the state a store starts in. Counting costs
 * about a tenth of a lookup's kernel time when the lookup is bound by
 * probe latency, so a caller can measure with it off and count in a
 * separate pass. Host only: no device work, no wait. Errors: INVALID (NULL
 * store). */
int ptstore_set_counters(ptstore_t *store, int on);

/* Turn the HIP events around kernels (what ptstore_kernel_times() reports)
 * on (on != 0) or off for the calls enqueued after this one; pairs already
 * recorded stay until read. PTSTORE_FLAG_TIMING sets the state a store
 * starts in. Two events around each launch add a few microseconds to a
 * short call, so a caller can time back-to-back short calls with them off
 * and one event pair of its own around all of them. Host only: no device
 * work, no wait. Errors: INVALID (NULL store). The same as
 * ptstore_set_timing_kinds with every kind (0x7F) or none. */
int ptstore_set_timing(ptstore_t *store, int on);

/* The events of some kinds only: bit k of `kinds` turns on those around
 * the kernels of kind k (the kinds of ptstore_kernel_times), and a clear
 * bit turns them off, for the calls enqueued after this one. A caller that
 * times short calls back to back can so keep the events around the copy
 * kernel alone (kinds = 1) and leave the lookup and the descriptor-list
 * build without them. Host only. Errors: INVALID (NULL store, a bit above
 * 6). */
int ptstore_set_timing_kinds(ptstore_t *store, uint32_t kinds);

/* Device buffers of the store (see ptstore_buffers_t); no device work.
 * Errors: INVALID (a NULL argument). */
int ptstore_get_buffers(ptstore_t *store, ptstore_buffers_t *out);

/*
 * With events on (PTSTORE_FLAG_TIMING, ptstore_set_timing or
 * ptstore_set_timing_kinds): wait for the device, then return the summed
 * durations (ms) and launch counts of the kernels recorded since the last
 * call, for kind 0 = gather copy kernel, 1 = lookup, 2 = scatter copy
 * kernel, 3 = insert (all its kernels), 4 = descriptor-list build of gather
 * and scatter, 5 = the eviction part of an insert (PTSTORE_FLAG_EVICT;
 * included in kind 3), 6 = ptstore_replicate. Resets the records of that
 * kind. At most 65,536 launches
 * per kind are recorded between two calls.
 */
int ptstore_kernel_times(ptstore_t *store, int32_t kind, double *total_ms, int64_t *launches);

/* Launch shape of the copy kernels (gather and scatter); 0 keeps a field's
 * current value. chunks_per_group: (layer, K|V) chunks one unit moves (by
 * default the smallest divisor of 2 * num_layers that leaves at most 64
 * units per block, and a gather of a layer range of at most 4 chunks per
 * block moves the whole range as one unit; once set here, it applies to
 * every copy); threads: workgroup size, 64..1024, a multiple of 64
 * (default 1024); grid: workgroups of the copy kernels (by default a
 * gather launches one per possible unit, up to 512 times the workgroups
 * the device holds at once, and a scatter 16 times the workgroups the
 * device holds, looping; a grid once set replaces both until set again).
 * For tuning sweeps; results never depend on it. */
int ptstore_set_copy_shape(ptstore_t *store, int32_t chunks_per_group, int32_t threads,
                           int32_t grid);

/*
 * Streaming-bandwidth probe (not a store operation): enqueue on `stream` one
 * kernel that, with the access pattern of the copy kernels (16-byte
 * non-temporal vectors), reads `bytes` from `a` (kind 0), writes `bytes` to
 * `b` (kind 1) or copies `bytes` from `a` to `b` (kind 2). Time it with
 * events around the call to get the device's practical HBM ceiling.
 * `a`, `b`: device buffers of at least `bytes`, 16-byte aligned; `bytes` a
 * multiple of 16, at most 32 GiB. Errors: INVALID, HIP.
 */
int ptstore_bandwidth_probe(int32_t kind, const void *a, void *b, int64_t bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* PTSTORE_H */
