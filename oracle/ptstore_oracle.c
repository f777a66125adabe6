/*
 * CPU oracle of the prefix store -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, single-threaded C. It exists so that the GPU library can be
 * checked against something obviously correct; nothing on the product path
 * may link or call it. It shares no source with the GPU library.
 *
 * What it computes (PTStore, Section 4.1 "Co-optimized compact metadata and
 * fast prefix queries", and Section 1 "Contributions"):
 *
 *   - Stored objects are sequences of fixed-size token blocks. The store
 *     keeps each distinct block-prefix exactly once, as a node of a trie
 *     whose root is the empty prefix: prefixes that branch apart share what
 *     they have in common and nothing is stored twice (Section 1).
 *   - Every node has a dense unique id and a KV payload of block_bytes in
 *     a pool indexed by that id. An object's metadata is the flat list of
 *     the ids on its root path: it inherits the ids of its longest common
 *     prefix with what is stored and appends ids for its own increment
 *     (Section 4.1).
 *   - lookup: the longest common prefix, in whole blocks, of a request with
 *     everything stored (Section 4.1, the LCP query), plus the ids along it.
 *   - gather: a load iterates over those ids and copies their tensors into
 *     application-supplied memory (Section 4.1), here a paged cache laid out
 *     [layer][K|V][cache block][head][slot][dim]. A load may ask for a range
 *     of layers only (Section 5: clients read and write subsets of tensors),
 *     and layers may differ in size (Section 5: prefixes are combinations
 *     of tensors of variable sizes).
 *   - insert: a store saves only the increment beyond the LCP (Section 4),
 *     processing the batch one request after another; new nodes get the next
 *     free id. No node is created beyond the capacity.
 *   - scatter: copies the KV of the nodes an insert created from the paged
 *     cache into the pool.
 *   - eviction (optional, Section 4.1 "Access pattern-aware eviction
 *     policy"): when an insert needs more ids than remain, leaf nodes are
 *     evicted by frequency with a GDSF-style priority, so that the trie stays
 *     prefix-closed. The exact rules are spelt out at insert_evict() below.
 *   - hot set (Section 4.1, "Replication of popular prefixes"): the nodes of
 *     an id range with the highest priorities, those a faster tier keeps
 *     copies of. Where a block's bytes live never changes any result, so
 *     the oracle keeps one flat pool whatever the tiers.
 *
 * Trie representation: each node keeps a pointer to its parent, its first
 * child and its next sibling; a child is found by comparing the block's
 * tokens against each child in turn. No hashing is involved anywhere.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_ERR_INVALID 1
#define ORC_ERR_FULL 2
#define ORC_ERR_NOMEM 3

typedef struct onode {
    int32_t id;                 /* -1 for the root, -1 while tentative */
    struct onode *parent;
    struct onode *first_child;
    struct onode *next_sibling;
    int32_t *tokens;            /* block_tokens tokens of this block */
    /* eviction bookkeeping */
    int64_t freq;               /* accesses so far */
    int64_t prio;               /* clock + freq at the last access */
    int32_t live_children;      /* children that hold an id */
    int32_t protect;            /* epoch of the last insert whose match ran through it */
    int32_t depth;              /* 0 for a child of the root */
    int32_t creator;            /* request of the running insert that created it */
    int32_t born;               /* epoch of the insert that created it */
    int32_t dropped;            /* tentative node refused for lack of an id */
} onode_t;

typedef struct {
    int32_t layers, block_tokens;
    int64_t *chunk;             /* [layers] bytes of one (layer, K|V) slab of a block */
    int64_t *lbase;             /* [layers + 1] 2 * sum of chunk[0..l-1] */
    int64_t block_bytes;        /* lbase[layers] */
    int64_t capacity;           /* maximum number of nodes */
    int64_t count;              /* nodes created so far (= next id) */
    int64_t bad_entries;        /* skipped out-of-range ids / cache blocks */
    int32_t evict;              /* 1: inserts evict leaves when out of ids */
    int32_t epoch;              /* insert calls so far (eviction mode) */
    int64_t clock;              /* GDSF inflation value L */
    int64_t evictions;
    onode_t root;
    onode_t **by_id;            /* id -> node */
    uint8_t *pool;              /* capacity * block_bytes, or NULL */
} ostore_t;

/*
 * A store whose layer l keeps slabs of chunk_bytes[l] bytes per block, for
 * K and for V. Layers of one model may differ (Section 5: tensors of
 * variable size).
 */
ostore_t *orc_create_layers(int32_t layers, int32_t block_tokens, const int64_t *chunk_bytes,
                            int64_t capacity, int32_t with_payload)
{
    if (layers < 1 || block_tokens < 1 || capacity < 0 || !chunk_bytes) return NULL;
    for (int32_t l = 0; l < layers; l++)
        if (chunk_bytes[l] < 1) return NULL;
    ostore_t *s = (ostore_t *)calloc(1, sizeof(ostore_t));
    if (!s) return NULL;
    s->layers = layers;
    s->block_tokens = block_tokens;
    s->chunk = (int64_t *)malloc((size_t)layers * sizeof(int64_t));
    s->lbase = (int64_t *)malloc((size_t)(layers + 1) * sizeof(int64_t));
    if (!s->chunk || !s->lbase) abort();  /* test infrastructure: no recovery */
    s->lbase[0] = 0;
    for (int32_t l = 0; l < layers; l++) {
        s->chunk[l] = chunk_bytes[l];
        s->lbase[l + 1] = s->lbase[l] + 2 * chunk_bytes[l];
    }
    s->block_bytes = s->lbase[layers];
    s->capacity = capacity;
    s->root.id = -1;
    s->root.depth = -1;
    s->by_id = (onode_t **)calloc(capacity > 0 ? (size_t)capacity : 1, sizeof(onode_t *));
    if (!s->by_id) abort();
    if (with_payload && capacity > 0) {
        s->pool = (uint8_t *)calloc((size_t)capacity, (size_t)s->block_bytes);
        if (!s->pool) { free(s->by_id); free(s->chunk); free(s->lbase); free(s); return NULL; }
    }
    return s;
}

/* Every layer the same: slabs of kv_heads * block_tokens * head_dim elements. */
ostore_t *orc_create(int32_t layers, int32_t kv_heads, int32_t head_dim,
                     int32_t block_tokens, int32_t elem_bytes,
                     int64_t capacity, int32_t with_payload)
{
    if (layers < 1 || kv_heads < 1 || head_dim < 1 || block_tokens < 1 || elem_bytes < 1)
        return NULL;
    int64_t *c = (int64_t *)malloc((size_t)layers * sizeof(int64_t));
    if (!c) return NULL;
    for (int32_t l = 0; l < layers; l++) c[l] = (int64_t)kv_heads * block_tokens * head_dim * elem_bytes;
    ostore_t *s = orc_create_layers(layers, block_tokens, c, capacity, with_payload);
    free(c);
    return s;
}

void orc_destroy(ostore_t *s)
{
    if (!s) return;
    for (int64_t i = 0; i < s->count; i++) {
        if (!s->by_id[i]) continue;
        free(s->by_id[i]->tokens);
        free(s->by_id[i]);
    }
    free(s->by_id);
    free(s->pool);
    free(s->chunk);
    free(s->lbase);
    free(s);
}

/* The child of `node` whose block equals `blk`, or NULL. */
static onode_t *find_child(const ostore_t *s, const onode_t *node, const int32_t *blk)
{
    size_t nbytes = (size_t)s->block_tokens * sizeof(int32_t);
    for (onode_t *c = node->first_child; c; c = c->next_sibling)
        if (memcmp(c->tokens, blk, nbytes) == 0)
            return c;
    return NULL;
}

static onode_t *add_child(ostore_t *s, onode_t *node, const int32_t *blk)
{
    onode_t *c = (onode_t *)calloc(1, sizeof(onode_t));
    if (!c) return NULL;
    c->tokens = (int32_t *)malloc((size_t)s->block_tokens * sizeof(int32_t));
    if (!c->tokens) { free(c); return NULL; }
    memcpy(c->tokens, blk, (size_t)s->block_tokens * sizeof(int32_t));
    c->id = (int32_t)s->count;
    c->depth = node->depth + 1;
    c->parent = node;
    c->next_sibling = node->first_child;
    node->first_child = c;
    s->by_id[s->count++] = c;
    return c;
}

/* Number of whole blocks of request r that are considered. */
static int32_t request_blocks(const ostore_t *s, const int64_t *offsets, int32_t r,
                              int32_t max_blocks)
{
    int64_t len = offsets[r + 1] - offsets[r];
    int64_t n = len / s->block_tokens;
    return (int32_t)(n < max_blocks ? n : max_blocks);
}

static int check_batch(const int64_t *offsets, int32_t R, int32_t max_blocks)
{
    if (R < 0 || max_blocks < 1 || (R > 0 && !offsets)) return ORC_ERR_INVALID;
    for (int32_t r = 0; r < R; r++)
        if (offsets[r + 1] < offsets[r]) return ORC_ERR_INVALID;
    return ORC_OK;
}

/* One access of a node (eviction mode): the frequency grows and the
 * priority is refreshed with the current clock, H = L + F (GDSF with a
 * cost-over-size factor of 1, all blocks being the same size). */
static void touch(ostore_t *s, onode_t *n)
{
    n->freq += 1;
    n->prio = s->clock + n->freq;
}

/*
 * LCP query (Section 4.1): m[r] = the largest k such that blocks 0..k-1 of
 * request r form a path from the root; ids[r][b] = id of the b-th node on
 * it, -1 for b >= m[r]. Only the first max_blocks whole blocks count.
 * In eviction mode every matched node counts one access.
 */
int orc_lookup(ostore_t *s, const int32_t *tokens, const int64_t *offsets,
               int32_t R, int32_t max_blocks, int32_t *m, int32_t *ids)
{
    int rc = check_batch(offsets, R, max_blocks);
    if (rc) return rc;
    for (int32_t r = 0; r < R; r++) {
        int32_t n = request_blocks(s, offsets, r, max_blocks);
        const int32_t *seq = tokens + offsets[r];
        int32_t *row = ids + (int64_t)r * max_blocks;
        onode_t *node = &s->root;
        int32_t b = 0;
        for (; b < n; b++) {
            onode_t *c = find_child(s, node, seq + (int64_t)b * s->block_tokens);
            if (!c) break;
            row[b] = c->id;
            if (s->evict) touch(s, c);
            node = c;
        }
        m[r] = b;
        for (int32_t j = b; j < max_blocks; j++) row[j] = -1;
    }
    return ORC_OK;
}

/* Byte offset of (layer l, K|V kv, cache block cb) in the paged cache: layer
 * l occupies 2 * cache_blocks slabs of chunk[l] bytes, after all earlier
 * layers. */
static int64_t cache_off(const ostore_t *s, int64_t cache_blocks, int32_t l, int32_t kv,
                         int64_t cb)
{
    return cache_blocks * s->lbase[l] + ((int64_t)kv * cache_blocks + cb) * s->chunk[l];
}

/* Byte offset of (node id, layer l, K|V kv) in the pool. */
static int64_t pool_off(const ostore_t *s, int64_t id, int32_t l, int32_t kv)
{
    return id * s->block_bytes + s->lbase[l] + (int64_t)kv * s->chunk[l];
}

/*
 * Load (Section 4.1): for every matched block b < m[r] whose block-table
 * entry is >= 0, copy the (layer, K|V) slabs of layers l0 .. l1-1 of
 * pool[ids[r][b]] into cache[layer][K|V][block_table[r][b]]. Out-of-range
 * ids or cache blocks are skipped and counted in bad_entries.
 */
int orc_gather_layers(ostore_t *s, const int32_t *ids, const int32_t *m, const int32_t *block_table,
                      int32_t R, int32_t max_blocks, int32_t l0, int32_t l1, uint8_t *cache,
                      int64_t cache_blocks)
{
    if (!s->pool || R < 0 || max_blocks < 1 || cache_blocks < 0 || l0 < 0 || l1 > s->layers ||
        l0 >= l1)
        return ORC_ERR_INVALID;
    for (int32_t r = 0; r < R; r++) {
        int32_t mr = m[r] < max_blocks ? m[r] : max_blocks;
        for (int32_t b = 0; b < mr; b++) {
            int64_t id = ids[(int64_t)r * max_blocks + b];
            int64_t cb = block_table[(int64_t)r * max_blocks + b];
            if (cb < 0) continue;
            if (cb >= cache_blocks || id < 0 || id >= s->count || !s->by_id[id]) {
                s->bad_entries++;
                continue;
            }
            for (int32_t l = l0; l < l1; l++)
                for (int32_t kv = 0; kv < 2; kv++)
                    memcpy(cache + cache_off(s, cache_blocks, l, kv, cb),
                           s->pool + pool_off(s, id, l, kv), (size_t)s->chunk[l]);
        }
    }
    return ORC_OK;
}

int orc_gather(ostore_t *s, const int32_t *ids, const int32_t *m, const int32_t *block_table,
               int32_t R, int32_t max_blocks, uint8_t *cache, int64_t cache_blocks)
{
    return orc_gather_layers(s, ids, m, block_table, R, max_blocks, 0, s->layers, cache, cache_blocks);
}

/*
 * Store (Sections 1 and 4): requests are taken in batch order. Each one
 * walks its blocks from the root; existing nodes (stored earlier, or
 * created by an earlier request of this batch) are reused, a missing block
 * becomes a new node with the next id, unless the store already holds
 * `capacity` nodes, in which case the walk of this request stops there.
 * Outputs: m_out[r] = blocks of r resident after the call, ids[r][b] their
 * ids (-1 beyond), created[r][b] = 1 where request r created the node.
 * Returns ORC_ERR_FULL if some block was refused for lack of capacity.
 */
static int insert_evict(ostore_t *s, const int32_t *tokens, const int64_t *offsets, int32_t R,
                        int32_t max_blocks, int32_t *m_out, int32_t *ids, uint8_t *created);

int orc_insert(ostore_t *s, const int32_t *tokens, const int64_t *offsets, int32_t R,
               int32_t max_blocks, int32_t *m_out, int32_t *ids, uint8_t *created)
{
    int rc = check_batch(offsets, R, max_blocks);
    if (rc) return rc;
    if (s->evict) return insert_evict(s, tokens, offsets, R, max_blocks, m_out, ids, created);
    int full = 0;
    for (int32_t r = 0; r < R; r++) {
        int32_t n = request_blocks(s, offsets, r, max_blocks);
        const int32_t *seq = tokens + offsets[r];
        int32_t *row = ids + (int64_t)r * max_blocks;
        uint8_t *crow = created + (int64_t)r * max_blocks;
        memset(crow, 0, (size_t)max_blocks);
        onode_t *node = &s->root;
        int32_t b = 0;
        for (; b < n; b++) {
            const int32_t *blk = seq + (int64_t)b * s->block_tokens;
            onode_t *c = find_child(s, node, blk);
            if (!c) {
                if (s->count >= s->capacity) { full = 1; break; }
                c = add_child(s, node, blk);
                if (!c) return ORC_ERR_NOMEM;
                crow[b] = 1;
            }
            row[b] = c->id;
            node = c;
        }
        m_out[r] = b;
        for (int32_t j = b; j < max_blocks; j++) row[j] = -1;
    }
    return full ? ORC_ERR_FULL : ORC_OK;
}

/* Unlink `c` from its parent's list of children. */
static void unlink_child(onode_t *c)
{
    onode_t **pp = &c->parent->first_child;
    while (*pp != c) pp = &(*pp)->next_sibling;
    *pp = c->next_sibling;
}

/*
 * Insert with eviction (Section 4.1, "Access pattern-aware eviction
 * policy": frequency-based, GDSF adapted to shared prefixes; leaves only,
 * so that what stays is still a set of whole prefixes). Batch semantics:
 *  1. Every request is matched against the store as it was; the nodes on
 *     the matched paths are protected for this call.
 *  2. The blocks missing from the store are taken in request order; each
 *     distinct new prefix becomes one tentative node (later requests reuse
 *     the tentative nodes of earlier ones). Let N be their number.
 *  3. If N exceeds the ids never handed out (capacity - count), evict that
 *     many nodes, one after another: each time a leaf -- a node holding an
 *     id with no child holding one -- that is not protected, the one with
 *     the lowest priority; among equal priorities the deepest, then the
 *     smallest id. The clock becomes max(clock, priority of the victim).
 *     Stop early once no leaf qualifies.
 *  4. Tentative nodes get ids in their order: never-used ids first, then the
 *     victims' ids from the smallest up. Once ids run out, the remaining
 *     tentative nodes are refused (children come after parents in this
 *     order, so each request keeps a prefix).
 *  5. Every node on a request's resident path counts one access, with the
 *     clock as it stands after the evictions; a new node starts at 0.
 * Outputs as orc_insert; returns ORC_ERR_FULL if a node was refused.
 */
/* 1 if `a` is evicted before `b`: lower priority, then deeper, then smaller id. */
static int evicts_before(const onode_t *a, const onode_t *b)
{
    if (a->prio != b->prio) return a->prio < b->prio;
    if (a->depth != b->depth) return a->depth > b->depth;
    return a->id < b->id;
}

static int cmp_i32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

static int insert_evict(ostore_t *s, const int32_t *tokens, const int64_t *offsets, int32_t R,
                        int32_t max_blocks, int32_t *m_out, int32_t *ids, uint8_t *created)
{
    const int64_t rb = (int64_t)R * max_blocks;
    onode_t **path = (onode_t **)calloc(rb > 0 ? (size_t)rb : 1, sizeof(onode_t *));
    onode_t **tent = (onode_t **)calloc(rb > 0 ? (size_t)rb : 1, sizeof(onode_t *));
    int32_t *victims = (int32_t *)calloc(rb > 0 ? (size_t)rb : 1, sizeof(int32_t));
    if (!path || !tent || !victims) { free(path); free(tent); free(victims); return ORC_ERR_NOMEM; }
    s->epoch++;
    /* 1 + 2: match, protect, and create tentative nodes in request order */
    int64_t N = 0;
    for (int32_t r = 0; r < R; r++) {
        int32_t n = request_blocks(s, offsets, r, max_blocks);
        const int32_t *seq = tokens + offsets[r];
        onode_t *node = &s->root;
        for (int32_t b = 0; b < n; b++) {
            const int32_t *blk = seq + (int64_t)b * s->block_tokens;
            onode_t *c = find_child(s, node, blk);
            if (!c) {
                c = (onode_t *)calloc(1, sizeof(onode_t));
                int32_t *tk = (int32_t *)malloc((size_t)s->block_tokens * sizeof(int32_t));
                if (!c || !tk) abort();  /* test infrastructure: no recovery */
                c->tokens = tk;
                memcpy(c->tokens, blk, (size_t)s->block_tokens * sizeof(int32_t));
                c->id = -1;
                c->depth = node->depth + 1;
                c->creator = r;
                c->born = s->epoch;
                c->parent = node;
                c->next_sibling = node->first_child;
                node->first_child = c;
                tent[N++] = c;
            } else if (c->id >= 0) {
                c->protect = s->epoch;
            }
            path[(int64_t)r * max_blocks + b] = c;
            node = c;
        }
    }
    /* 3: evictions */
    const int64_t fresh = s->capacity - s->count;
    const int64_t want = N > fresh ? N - fresh : 0;
    int64_t nv = 0;
    while (nv < want) {
        onode_t *best = NULL;
        for (int64_t i = 0; i < s->count; i++) {
            onode_t *c = s->by_id[i];
            if (!c || c->live_children > 0 || c->protect == s->epoch) continue;
            if (!best || evicts_before(c, best)) best = c;
        }
        if (!best) break;
        if (best->prio > s->clock) s->clock = best->prio;
        if (best->parent != &s->root) best->parent->live_children--;
        unlink_child(best);
        s->by_id[best->id] = NULL;
        victims[nv++] = best->id;
        s->evictions++;
        free(best->tokens);
        free(best);
    }
    /* 4: ids for the tentative nodes */
    qsort(victims, (size_t)nv, sizeof(int32_t), cmp_i32);
    int full = 0;
    for (int64_t k = 0; k < N; k++) {
        onode_t *c = tent[k];
        int64_t id;
        if (k < fresh) id = s->count++;
        else if (k - fresh < nv) id = victims[k - fresh];
        else { full = 1; c->dropped = 1; continue; }
        c->id = (int32_t)id;
        s->by_id[id] = c;
        if (c->parent != &s->root) c->parent->live_children++;
    }
    /* outputs */
    for (int32_t r = 0; r < R; r++) {
        int32_t n = request_blocks(s, offsets, r, max_blocks);
        int32_t *row = ids + (int64_t)r * max_blocks;
        uint8_t *crow = created + (int64_t)r * max_blocks;
        memset(crow, 0, (size_t)max_blocks);
        int32_t b = 0;
        for (; b < n; b++) {
            onode_t *c = path[(int64_t)r * max_blocks + b];
            if (c->dropped) break;
            row[b] = c->id;
            /* created: this request made the node in this call */
            if (c->born == s->epoch && c->creator == r) crow[b] = 1;
        }
        m_out[r] = b;
        for (int32_t j = b; j < max_blocks; j++) row[j] = -1;
    }
    /* 5: accesses with the clock after the evictions */
    for (int32_t r = 0; r < R; r++)
        for (int32_t b = 0; b < m_out[r]; b++) touch(s, path[(int64_t)r * max_blocks + b]);
    /* drop refused tentative nodes (children before parents) */
    for (int64_t k = N - 1; k >= 0; k--) {
        onode_t *c = tent[k];
        if (!c->dropped) continue;
        unlink_child(c);
        free(c->tokens);
        free(c);
    }
    free(path);
    free(tent);
    free(victims);
    return full ? ORC_ERR_FULL : ORC_OK;
}

/*
 * Store data: for every (r, b) with created[r][b] = 1 and a block-table
 * entry >= 0, copy the (layer, K|V) slabs of layers l0 .. l1-1 of
 * cache[..][block_table[r][b]] into pool[ids[r][b]].
 */
int orc_scatter_layers(ostore_t *s, const int32_t *ids, const uint8_t *created,
                       const int32_t *block_table, int32_t R, int32_t max_blocks, int32_t l0,
                       int32_t l1, const uint8_t *cache, int64_t cache_blocks)
{
    if (!s->pool || R < 0 || max_blocks < 1 || cache_blocks < 0 || l0 < 0 || l1 > s->layers ||
        l0 >= l1)
        return ORC_ERR_INVALID;
    for (int32_t r = 0; r < R; r++) {
        for (int32_t b = 0; b < max_blocks; b++) {
            int64_t k = (int64_t)r * max_blocks + b;
            if (!created[k]) continue;
            int64_t id = ids[k];
            int64_t cb = block_table[k];
            if (cb < 0) continue;
            if (cb >= cache_blocks || id < 0 || id >= s->count || !s->by_id[id]) {
                s->bad_entries++;
                continue;
            }
            for (int32_t l = l0; l < l1; l++)
                for (int32_t kv = 0; kv < 2; kv++)
                    memcpy(s->pool + pool_off(s, id, l, kv),
                           cache + cache_off(s, cache_blocks, l, kv, cb), (size_t)s->chunk[l]);
        }
    }
    return ORC_OK;
}

int orc_scatter(ostore_t *s, const int32_t *ids, const uint8_t *created,
                const int32_t *block_table, int32_t R, int32_t max_blocks,
                const uint8_t *cache, int64_t cache_blocks)
{
    return orc_scatter_layers(s, ids, created, block_table, R, max_blocks, 0, s->layers, cache,
                              cache_blocks);
}

/* ---- inspection helpers for the tests ---- */

int64_t orc_count(const ostore_t *s) { return s->count; }
void orc_set_evict(ostore_t *s, int32_t on) { s->evict = on ? 1 : 0; }
int64_t orc_clock(const ostore_t *s) { return s->clock; }
int64_t orc_evictions(const ostore_t *s) { return s->evictions; }

/*
 * Hot set (Section 4.1, replication of popular prefixes): of the nodes with
 * ids in [lo, hi), the `k` with the highest priority H, ties going to the
 * smaller id; written to out[] in ascending id order. Returns how many were
 * written (fewer than k if the range holds fewer nodes).
 */
typedef struct { int64_t prio; int32_t id; } hot_key_t;

/* Highest priority first, then the smaller id. */
static int cmp_hot(const void *a, const void *b)
{
    const hot_key_t *x = (const hot_key_t *)a, *y = (const hot_key_t *)b;
    if (x->prio != y->prio) return x->prio > y->prio ? -1 : 1;
    return (x->id > y->id) - (x->id < y->id);
}

int64_t orc_hot_set(const ostore_t *s, int64_t lo, int64_t hi, int64_t k, int32_t *out)
{
    if (lo < 0) lo = 0;
    if (hi > s->count) hi = s->count;
    if (hi <= lo || k <= 0) return 0;
    hot_key_t *all = (hot_key_t *)malloc((size_t)(hi - lo) * sizeof(hot_key_t));
    if (!all) abort();  /* test infrastructure: no recovery */
    int64_t n = 0;
    for (int64_t i = lo; i < hi; i++) {
        if (!s->by_id[i]) continue;
        all[n].prio = s->by_id[i]->prio;
        all[n].id = (int32_t)i;
        n++;
    }
    qsort(all, (size_t)n, sizeof(hot_key_t), cmp_hot);
    if (n > k) n = k;
    for (int64_t j = 0; j < n; j++) out[j] = all[j].id;
    free(all);
    qsort(out, (size_t)n, sizeof(int32_t), cmp_i32);
    return n;
}

/* Eviction bookkeeping of node `id`; ORC_ERR_INVALID if it holds no node. */
int orc_node_stats(const ostore_t *s, int64_t id, int64_t *freq, int64_t *prio,
                   int32_t *live_children, int32_t *depth)
{
    if (id < 0 || id >= s->count || !s->by_id[id]) return ORC_ERR_INVALID;
    *freq = s->by_id[id]->freq;
    *prio = s->by_id[id]->prio;
    *live_children = s->by_id[id]->live_children;
    *depth = s->by_id[id]->depth;
    return ORC_OK;
}
int64_t orc_bad_entries(const ostore_t *s) { return s->bad_entries; }
int64_t orc_block_bytes(const ostore_t *s) { return s->block_bytes; }
uint8_t *orc_pool(ostore_t *s) { return s->pool; }

/* parent id (-1 = root) and tokens of node `id`; returns ORC_ERR_INVALID if absent. */
int orc_node(const ostore_t *s, int64_t id, int32_t *parent, int32_t *tokens_out)
{
    if (id < 0 || id >= s->count || !s->by_id[id]) return ORC_ERR_INVALID;
    const onode_t *n = s->by_id[id];
    *parent = n->parent ? n->parent->id : -1;
    if (tokens_out)
        memcpy(tokens_out, n->tokens, (size_t)s->block_tokens * sizeof(int32_t));
    return ORC_OK;
}
