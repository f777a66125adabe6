// Host runtime of the prefix store: the C ABI declared in include/ptstore.h.
//
// The store owns, on one device:
//   pool    [dev rows][layer][K|V][head][slot][dim]  KV payload, per-block contiguous:
//           the home of ids below `owned`, then the replica slots
//   host    [host rows][...] pinned host tier, the home of ids owned..
//   parent  [capacity] int32, tokens [capacity][block_tokens] int32   block metadata
//   slots   [index_slots] {key, id, parent}          open-addressing block index
//   ht      key-chain constants, state: counters and the block count
//   evs     with eviction on: per-block access counts, priorities, child
//           counts, depths, index keys and slots, and the victim-selection
//           scratch (all sized by the capacity, allocated here once)
//   insert_scratch insert work space; copy_scratch gather/scatter descriptor lists,
//           one per stream the store's calls are enqueued on (both grown on
//           demand, so the hot path allocates only when a batch is larger
//           than every earlier one on that stream)
// Calls check their arguments, enqueue kernels on the caller's stream and
// return; nothing on the lookup / gather path allocates or synchronises.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "ptstore.h"
#include "kernels.hpp"

using namespace ptsd;

// Descriptor-list scratch of ptstore_lookup_gather_noalloc, for callers that
// cannot allocate: one copy per device, held until the process ends, shared
// by every such call on that device (calls that overlap on one device race).
// Its size is the gather's list for PTSTORE_NOALLOC_MAX_ENTRIES (request,
// block) entries: a row table of twice as many slots (12 bytes each), then
// 36 bytes per entry (pair, slice, cache block, table slot and rank), 2 x
// (4 + 8) per request (at most one request per entry) and the counters,
// each part a multiple of 256 bytes. Static storage starts zeroed, so the
// row table starts empty, as every call leaves it.
constexpr uint64_t kNoAllocTableSlots = 2ull * PTSTORE_NOALLOC_MAX_ENTRIES;
constexpr size_t kNoAllocScratchBytes = kNoAllocTableSlots * 12 +
                                        (size_t)PTSTORE_NOALLOC_MAX_ENTRIES * (36 + 2 * (4 + 8)) + 256;
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

struct ptstore {
    ptstore_config_t cfg;
    int device;
    int64_t chunk_bytes, block_bytes, capacity;
    uint64_t slots_n;
    uint8_t* pool;
    int32_t* parent;
    int32_t* tokens;
    Slot* slots;
    HashTables* ht;
    DevState* state;
    void* insert_scratch;
    size_t insert_scratch_size;
    // descriptor-list scratch per stream, so that lookups and gathers on
    // different streams may run at the same time
    struct StreamScratch {
        hipStream_t stream;
        void* p;
        size_t bytes;
        uint64_t table_cap;  // row-table slots at the start of p, kept empty between calls
        bool dirty;          // a call failed between filling and emptying the row table
    };
    std::vector<StreamScratch> copy_scratch;
    int32_t chunks_per_group, threads, grid;
    bool chunks_set;  // chunks_per_group set by ptstore_set_copy_shape
    int32_t cus;  // compute units of the device
    EvictView evs;  // evs.on = 0 without PTSTORE_FLAG_EVICT
    void* ev_mem;  // one allocation holding every ev array
    TierView tier;  // owned = capacity and no host rows for a device-only store
    void* tier_mem; // replica map and replicate scratch
    void* host_mem; // the host tier as allocated (tier.host is its device address)
    void* layer_tab; // per-layer slab bases [L + 1], int64 (layer l's slabs are half of
                     // base[l+1] - base[l] each); null if every layer has chunk_bytes
    std::vector<int64_t> lbase_host;  // the bases, for launch shapes
    // the block list of ptstore_gather_prepare, while it is valid
    bool prep_valid;
    void* prep_list;  // the copy scratch holding it
    uint64_t prep_table_cap;
    int32_t prep_R, prep_max_blocks;
    int64_t prep_cache_blocks;
    // HIP events around kernels, per kind; bit k of timing_kinds records kind k
    uint32_t timing_kinds;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> ev[7];
    std::vector<hipEvent_t> free_ev;
};

namespace {

// A fixed buffer, so that no error path allocates host memory either.
thread_local char g_last_error[512];

int fail(int code, const char* what, hipError_t e = hipSuccess) {
    if (e != hipSuccess)
        snprintf(g_last_error, sizeof g_last_error, "%s: %s", what, hipGetErrorString(e));
    else
        snprintf(g_last_error, sizeof g_last_error, "%s", what);
    return code;
}

// Shape limits that keep every size and offset well inside 64 bits.
constexpr int32_t kMaxLayers = 1 << 20;
constexpr uint64_t kMaxChunkBytes = 1ull << 30;
constexpr uint64_t kMaxTierBytes = 1ull << 56;

uint64_t next_pow2(uint64_t x) {
    uint64_t p = 1;
    while (p < x) p <<= 1;
    return p;
}

// (a * b) mod 2^61-1 on the host
uint64_t host_mulmod61(uint64_t a, uint64_t b) {
    unsigned __int128 p = (unsigned __int128)a * b;
    uint64_t lo = (uint64_t)p & kM61;
    uint64_t hi = (uint64_t)(p >> 61);
    return mod61(lo + hi);
}

void make_hash_tables(uint64_t seed, bool weak, bool weak_tag, HashTables* h) {
    memset(h, 0, sizeof *h);
    const uint64_t P = mod61(mix64(seed ^ 0x2545F4914F6CDD1Dull)) % (kM61 - 2) + 2;
    uint64_t x = P;
    for (int j = 0; j < kWave; ++j) {
        h->pow_lane[j] = x;  // P^(j+1)
        x = host_mulmod61(x, P);
    }
    // P^-1 = P^(p-2) (Fermat; p = 2^61-1 is prime)
    uint64_t pinv = 1, base = P;
    for (uint64_t e = kM61 - 2; e; e >>= 1) {
        if (e & 1) pinv = host_mulmod61(pinv, base);
        base = host_mulmod61(base, base);
    }
    uint64_t a = 1, b = 1;
    for (int j = 0; j < kWave; ++j) {
        h->pow0[j] = a;     // P^j
        h->inv_pow[j] = b;  // P^-j
        a = host_mulmod61(a, P);
        b = host_mulmod61(b, pinv);
    }
    h->p = P;
    h->root_key = mod61(mix64(seed ^ 0x9E3779B97F4A7C15ull));
    h->content_seed = mix64(seed ^ 0xD6E8FEB86659FD93ull);
    h->slot_seed = mix64(seed ^ 0xA0761D6478BD642Full);
    h->weak = weak ? 1u : 0u;
    h->weak_tag = weak_tag ? 1u : 0u;
}

// Device address of `scratch` per device, taken once with the device
// current (each device holds its own copy of the array at its own address).
// Host code uses only these addresses, never the array's name.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

int bind_static_scratch(int device) {
    if (device < 0 || device >= kMaxDevices) return PTSTORE_OK;  // the no-alloc call refuses
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[device]) return PTSTORE_OK;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return fail(PTSTORE_ERR_HIP, "ptstore_create: static scratch address", e);
    g_scratch_ptr[device] = p;
    return PTSTORE_OK;
}

void* static_scratch(int device) {
    if (device < 0 || device >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    return g_scratch_ptr[device];
}

// Whether a no-alloc call on `device` failed between filling and emptying
// the static scratch's row table; with set, records `value` instead.
bool g_scratch_dirty[kMaxDevices];
bool static_dirty(int device, bool set, bool value = false) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (set) g_scratch_dirty[device] = value;
    return g_scratch_dirty[device];
}

IndexView index_view(ptstore_t* s) {
    IndexView ix;
    ix.slots = s->slots;
    ix.slot_mask = s->slots_n - 1;
    ix.parent = s->parent;
    ix.tokens = s->tokens;
    ix.ht = s->ht;
    ix.state = s->state;
    ix.freq = s->evs.on ? s->evs.freq : nullptr;
    ix.prio = s->evs.on ? s->evs.prio : nullptr;
    ix.block_tokens = s->cfg.block_tokens;
    ix.counters = (s->cfg.flags & PTSTORE_FLAG_COUNTERS) ? 1 : 0;
    return ix;
}

CopyPlan copy_plan(ptstore_t* s) {
    CopyPlan p;
    p.pool = s->pool;
    p.block_bytes = s->block_bytes;
    p.chunk_bytes = s->chunk_bytes;
    p.chunks_per_block = 2 * s->cfg.num_layers;
    p.chunks_per_group = s->chunks_per_group;
    p.threads = s->threads;
    p.grid = s->grid;
    // in rounds of the workgroups the device holds at once (2048 threads per
    // compute unit): a gather launches one workgroup per possible unit, up to
    // 512 rounds, past which a workgroup takes further units a grid apart.
    // The host cannot know how many units a call has: entries that miss, and
    // entries that share a row with others, leave possible units empty, and
    // each empty workgroup still costs its launch (about 0.8 ns). On the
    // trie's 8,192 walks, whose 517,672 entries read 70,570 rows (184,474
    // units of 1,048,576 possible), 512 rounds copy in 7.46 ms against 8.11
    // at 2,048 rounds and 7.42 with exactly one workgroup per unit; on the 8B
    // shape (759,808 units) 12.38 against 12.47 and 12.21. A scatter, whose units are
    // sparse, launches 16 rounds that loop (4 rounds: 7 % slower on a large
    // scatter; 128 rounds: 45 % slower on a small one).
    const int resident = s->cus * (2048 / s->threads);
    p.gather_grid = resident * 512;
    p.loop_grid = resident * 16;
    // host-tier rows move over the host link whatever the grid: a quarter of
    // the compute units carry one workgroup each, the rest stay free
    p.host_grid = s->cus / 4 > 0 ? s->cus / 4 : 1;
    p.state = s->state;
    p.tier = s->tier;
    p.lbase = s->layer_tab ? static_cast<const int64_t*>(s->layer_tab) : nullptr;
    p.lbase_host = s->layer_tab ? s->lbase_host.data() : nullptr;
    return p;
}

// The plan of a gather of layers layer_begin .. layer_end-1. A layer range
// of at most 4 chunks per block (one or two layers of K and V slabs) moves
// as one unit per descriptor: the host sizes the grid by the possible
// units, the empty ones still cost their launch, and a per-layer load of
// the 8B shape (32 layers, one prepared list) took 16.0 ms this way against
// 16.7 with one unit per chunk. A whole-block gather keeps the store's
// shape (on the trie's one-layer blocks, two chunks per unit lost 1.4 %).
CopyPlan range_plan(ptstore_t* s, int32_t layer_begin, int32_t layer_end) {
    CopyPlan p = copy_plan(s);
    const int32_t chunks = 2 * (layer_end - layer_begin);
    if (!s->chunks_set && !s->layer_tab && chunks < p.chunks_per_block && chunks <= 4 &&
        chunks > p.chunks_per_group)
        p.chunks_per_group = chunks;
    return p;
}

hipEvent_t take_event(ptstore_t* s) {
    if (!s->free_ev.empty()) {
        hipEvent_t e = s->free_ev.back();
        s->free_ev.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Every kind of kernel ptstore_kernel_times() reports (0..6).
constexpr uint32_t kAllKinds = 0x7Fu;

// Most event pairs kept per kind between two ptstore_kernel_times() calls;
// beyond that, launches are no longer recorded (the sum stays consistent).
constexpr size_t kMaxTimed = 1 << 16;

// Brackets the kernels enqueued during its lifetime with two events.
struct Timed {
    ptstore_t* s;
    int kind;
    hipStream_t st;
    hipEvent_t a = nullptr;
    Timed(ptstore_t* s_, int k, hipStream_t st_) : s(s_), kind(k), st(st_) {
        if (((s->timing_kinds >> kind) & 1u) && s->ev[kind].size() < kMaxTimed) {
            a = take_event(s);
            if (a) (void)hipEventRecord(a, st);
        }
    }
    ~Timed() {
        if (!a) return;
        hipEvent_t b = take_event(s);
        if (!b) {  // not recorded after all: the first event goes back to the pool
            s->free_ev.push_back(a);
            return;
        }
        (void)hipEventRecord(b, st);
        s->ev[kind].push_back({a, b});
    }
};

// Most (request, block) entries one call takes.
constexpr int64_t kMaxEntries = 1ll << 29;

bool check_batch(ptstore_t* s, const int32_t* tokens, const int64_t* offsets, int64_t n_tokens,
                 int32_t R, int32_t max_blocks) {
    (void)s;
    if (R < 0 || max_blocks < 1) return false;
    if (n_tokens < 0 || n_tokens >= (int64_t)0xFFFFFFFFll) return false;
    if ((int64_t)R * max_blocks > kMaxEntries) return false;
    if (R > 0 && (!offsets || (!tokens && n_tokens > 0))) return false;
    return true;
}

// Makes the store's device current for the rest of a call and gives the
// caller's current device back when the call returns.
struct DeviceScope {
    int prev = -1;
    int rc = PTSTORE_OK;
    explicit DeviceScope(ptstore_t* s) {
        hipError_t e = hipGetDevice(&prev);
        if (e == hipSuccess && prev != s->device) e = hipSetDevice(s->device);
        if (e != hipSuccess) {
            prev = -1;
            rc = fail(PTSTORE_ERR_HIP, "hipSetDevice", e);
        }
    }
    ~DeviceScope() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

// Make *buf hold at least `need` bytes. Growing waits for `st` first, since
// work already enqueued on it may still read the old buffer.
int ensure_scratch(void** buf, size_t* have, size_t need, hipStream_t st, const char* who) {
    if (need <= *have) return PTSTORE_OK;
    hipError_t e = hipStreamSynchronize(st);
    if (e != hipSuccess) return fail(PTSTORE_ERR_HIP, who, e);
    (void)hipFree(*buf);
    *buf = nullptr;
    *have = 0;
    const size_t grow = need + need / 4;
    if ((e = hipMalloc(buf, grow)) != hipSuccess) {
        (void)hipGetLastError();
        return fail(PTSTORE_ERR_NOMEM, who, e);
    }
    *have = grow;
    return PTSTORE_OK;
}

// Most streams a store keeps a descriptor scratch for.
constexpr size_t kMaxStreams = 16;

// Is work on `st` being captured into a graph? No allocation or wait may
// happen then.
bool capturing(hipStream_t st) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    return hipStreamIsCapturing(st, &cs) == hipSuccess && cs != hipStreamCaptureStatusNone;
}

// The descriptor scratch of `st` for a call of R x max_blocks entries; made
// on the first call on a stream and grown when a call needs more (waiting
// for `st` first, since work enqueued on it may still read the old buffer).
// A new buffer's row table is emptied by a kernel on `st`, and so is the
// table of a scratch whose last call failed half-way. Under graph capture
// nothing is allocated or emptied: a stream that has a scratch must already
// have one of this size, and a stream that has made no call yet (such as a
// capture stream of its own) uses the scratch of the store's first stream.
int copy_scratch_for(ptstore_t* s, hipStream_t st, int32_t R, int32_t max_blocks, void** out,
                     uint64_t* table_cap, ptstore::StreamScratch** entry, const char* who) {
    const bool cap = capturing(st);
    const uint64_t slots = copy_table_slots(R, max_blocks);
    auto fits = [&](const ptstore::StreamScratch& e) {
        return e.table_cap >= slots && e.bytes >= copy_scratch_bytes(R, max_blocks, e.table_cap);
    };
    ptstore::StreamScratch* e = nullptr;
    for (auto& x : s->copy_scratch)
        if (x.stream == st) e = &x;
    if (cap) {
        ptstore::StreamScratch* use = e ? e : (s->copy_scratch.empty() ? nullptr : &s->copy_scratch[0]);
        if (!use || !fits(*use) || use->dirty)
            return fail(PTSTORE_ERR_INVALID, "a captured call needs a larger scratch than its stream "
                        "has: run a call of that size on the stream (or, for a new stream, on the "
                        "store's first stream) before capturing");
        *out = use->p;
        *table_cap = use->table_cap;
        *entry = use;
        return PTSTORE_OK;
    }
    if (!e) {
        if (s->copy_scratch.size() >= kMaxStreams)
            return fail(PTSTORE_ERR_INVALID, "calls on more than 16 streams of one store");
        s->copy_scratch.push_back({st, nullptr, 0, 0, false});
        e = &s->copy_scratch.back();
    }
    if (!fits(*e)) {
        const uint64_t new_cap = slots > e->table_cap ? slots : e->table_cap;
        size_t have = e->bytes;
        const int rc = ensure_scratch(&e->p, &have, copy_scratch_bytes(R, max_blocks, new_cap), st, who);
        e->bytes = have;
        e->table_cap = e->p ? new_cap : 0;
        if (rc) return rc;
        e->dirty = true;  // a new buffer: its table is emptied below
    }
    if (e->dirty) {
        const hipError_t z = launch_zero(e->p, copy_scratch_bytes(0, 0, e->table_cap) - 256, st);
        if (z != hipSuccess) return fail(PTSTORE_ERR_HIP, who, z);
        e->dirty = false;
    }
    *out = e->p;
    *table_cap = e->table_cap;
    *entry = e;
    return PTSTORE_OK;
}

// Carves the eviction arrays out of one block of device memory; returns the
// bytes needed (base may be null to only size them).
size_t carve_evict(void* base, int64_t capacity, EvictView* ev) {
    const int64_t cap = capacity > 0 ? capacity : 1;
    const int64_t words = (cap + kWave - 1) / kWave;
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    uint8_t* p = static_cast<uint8_t*>(base);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        void* q = p ? p + off : nullptr;
        off += up(bytes);
        return q;
    };
    ev->freq = static_cast<uint64_t*>(take(cap * 8));
    ev->prio = static_cast<uint64_t*>(take(cap * 8));
    ev->live = static_cast<int32_t*>(take(cap * 4));
    ev->prot = static_cast<int32_t*>(take(cap * 4));
    ev->depth = static_cast<int32_t*>(take(cap * 4));
    ev->nkey = static_cast<uint64_t*>(take(cap * 8));
    ev->spos = static_cast<uint32_t*>(take(cap * 4));
    ev->victims = static_cast<int32_t*>(take(cap * 4));
    ev->wmask = static_cast<uint64_t*>(take(words * 8));
    ev->wcnt = static_cast<uint32_t*>(take(words * 4));
    ev->wbase = static_cast<uint32_t*>(take(words * 4));
    ev->hist = static_cast<uint32_t*>(take((size_t)kSelPasses * kSelBins * 4));
    ev->part = static_cast<uint64_t*>(take((size_t)kSelGroups * 8 * 8));
    ev->words = words;
    return off;
}

}  // namespace

namespace ptsd {
int set_last_error(int code, const char* what) { return fail(code, what); }

__global__ void k_fill_slots(Slot* slots, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        Slot z;
        z.key = kEmptyKey;
        z.id = -1;
        z.parent = -1;
        slots[i] = z;
    }
}

hipError_t launch_fill_slots(Slot* slots, int64_t n, hipStream_t s) {
    int64_t g = (n + 255) / 256;
    if (g > 65536) g = 65536;
    if (g < 1) g = 1;
    hipLaunchKernelGGL(k_fill_slots, dim3((unsigned)g), dim3(256), 0, s, slots, n);
    return hipGetLastError();
}
}  // namespace ptsd

#pragma GCC visibility push(default)
extern "C" {

const char* ptstore_strerror(int code) {
    switch (code) {
        case PTSTORE_OK: return "ok";
        case PTSTORE_ERR_INVALID: return "invalid argument";
        case PTSTORE_ERR_FULL: return "store full";
        case PTSTORE_ERR_HIP: return "HIP runtime error";
        case PTSTORE_ERR_NOMEM: return "out of memory";
        default: return "unknown error";
    }
}

const char* ptstore_last_error(void) { return g_last_error; }

int ptstore_create(const ptstore_config_t* cfg, ptstore_t** out) {
    if (!cfg || !out) return fail(PTSTORE_ERR_INVALID, "ptstore_create: null argument");
    *out = nullptr;
    const ptstore_config_t c = *cfg;
    if (c.num_layers < 1 || c.num_layers > kMaxLayers || c.num_kv_heads < 1 || c.head_dim < 1 ||
        c.block_tokens < 1 || c.block_tokens > 64 || c.elem_bytes < 1)
        return fail(PTSTORE_ERR_INVALID, "ptstore_create: bad shape");
    if (c.pool_blocks < 0 || c.host_blocks < 0 || c.pool_blocks + c.host_blocks > (int64_t)0x7FFFFFFC)
        return fail(PTSTORE_ERR_INVALID, "ptstore_create: pool_blocks / host_blocks out of range");
    if (c.replica_blocks < 0 || c.replica_blocks > c.pool_blocks / 2 ||
        (c.replica_blocks > 0 && (c.host_blocks == 0 || !(c.flags & PTSTORE_FLAG_EVICT))))
        return fail(PTSTORE_ERR_INVALID,
                    "ptstore_create: replica_blocks must be <= pool_blocks/2 and needs host_blocks "
                    "and PTSTORE_FLAG_EVICT");
    const int64_t want_ids = c.pool_blocks - c.replica_blocks + c.host_blocks;
    // the slab size in 128 bits: four int32 factors can overflow 64
    const unsigned __int128 chunk_wide = (unsigned __int128)c.num_kv_heads * (uint32_t)c.block_tokens *
                                         (uint32_t)c.head_dim * (uint32_t)c.elem_bytes;
    if (!c.layer_chunk_bytes && chunk_wide > kMaxChunkBytes)
        return fail(PTSTORE_ERR_INVALID, "ptstore_create: a (layer, K|V) slab exceeds 1 GiB");
    int64_t chunk = (int64_t)chunk_wide;
    int64_t block = chunk * 2 * c.num_layers;
    std::vector<int64_t> lchunk, lbase;
    if (c.layer_chunk_bytes) {  // per-layer slab sizes
        if (c.num_layers > kMaxVarLayers)
            return fail(PTSTORE_ERR_INVALID, "ptstore_create: too many layers for per-layer sizes");
        lchunk.assign(c.layer_chunk_bytes, c.layer_chunk_bytes + c.num_layers);
        lbase.resize(c.num_layers + 1);
        block = 0;
        for (int l = 0; l < c.num_layers; ++l) {
            if (lchunk[l] < 16 || lchunk[l] % 16 != 0 || lchunk[l] > (int64_t)kMaxChunkBytes)
                return fail(PTSTORE_ERR_INVALID,
                            "ptstore_create: layer_chunk_bytes must be positive multiples of 16");
            lbase[l] = block;
            block += 2 * lchunk[l];
        }
        lbase[c.num_layers] = block;
        chunk = lchunk[0];
    } else if (chunk % 16 != 0) {
        return fail(PTSTORE_ERR_INVALID, "ptstore_create: chunk bytes must be a multiple of 16");
    }
    uint64_t slots_n;
    if (c.index_slots == 0) {
        slots_n = next_pow2((uint64_t)(2 * (want_ids > 1 ? want_ids : 1)));
        if (slots_n < 64) slots_n = 64;
    } else {
        if (c.index_slots < 2 || (c.index_slots & (c.index_slots - 1)) != 0 ||
            c.index_slots > (1ll << 32))
            return fail(PTSTORE_ERR_INVALID, "ptstore_create: index_slots must be a power of two >= 2");
        slots_n = (uint64_t)c.index_slots;
    }
    ptstore_t* s = new (std::nothrow) ptstore();
    if (!s) return fail(PTSTORE_ERR_NOMEM, "ptstore_create: host allocation");
    s->cfg = c;
    s->chunk_bytes = chunk;
    s->block_bytes = block;
    s->cfg.layer_chunk_bytes = nullptr;  // the caller's array is not kept
    s->slots_n = slots_n;
    s->capacity = want_ids < (int64_t)(slots_n / 2) ? want_ids : (int64_t)(slots_n / 2);
    {
        const int64_t owned = c.pool_blocks - c.replica_blocks;
        s->tier.owned = owned < s->capacity ? owned : s->capacity;
        s->tier.replicas = c.replica_blocks;
        s->tier.dev_rows = s->tier.owned + c.replica_blocks;
        s->tier.host_blocks = s->capacity - s->tier.owned;
    }
    // rows < 2^31 and block bytes <= 2^51: the byte sizes are formed in 128
    // bits, and one beyond any memory is refused here, not left to wrap
    if ((unsigned __int128)s->tier.dev_rows * (uint64_t)block > kMaxTierBytes ||
        (unsigned __int128)s->tier.host_blocks * (uint64_t)block > kMaxTierBytes) {
        delete s;
        return fail(PTSTORE_ERR_INVALID, "ptstore_create: pool larger than 2^56 bytes");
    }
    // 1024-thread workgroups, each moving the smallest whole number of
    // 32 KiB-class chunks that leaves at most 64 units per block: one chunk up
    // to 64 chunks per block (the 8B shape, where that shape held up best
    // whatever the placement), 4 at the 70B shape's 160. A gather's grid
    // covers every possible unit, hit or miss; at the 70B shape a larger share
    // of entries miss, and groups of 4 (4x fewer workgroups) measured 4.6-7 %
    // faster than single chunks there, while groups of 2 lost 1.3 % at 64.
    {
        const int cpb = 2 * c.num_layers;
        int cpg = 1;
        while (cpb / cpg > 64 || cpb % cpg != 0) ++cpg;
        s->chunks_per_group = cpg;
    }
    s->threads = 1024;
    s->grid = 0;
    s->chunks_set = false;
    s->timing_kinds = (c.flags & PTSTORE_FLAG_TIMING) ? kAllKinds : 0u;
    hipError_t e = hipGetDevice(&s->device);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&s->cus, hipDeviceAttributeMultiprocessorCount, s->device);
    if (e != hipSuccess) {
        delete s;
        return fail(PTSTORE_ERR_HIP, "ptstore_create: device query", e);
    }
    {  // the device's copy of the no-alloc call's scratch, with the device current
        const int rc = bind_static_scratch(s->device);
        if (rc) {
            delete s;
            return rc;
        }
    }
    const size_t pool_bytes = (size_t)(s->tier.dev_rows > 0 ? s->tier.dev_rows : 1) * (size_t)s->block_bytes;
    const size_t cap1 = (size_t)(s->capacity > 0 ? s->capacity : 1);
    if ((e = hipMalloc(&s->pool, pool_bytes)) != hipSuccess ||
        (e = hipMalloc(&s->parent, cap1 * 4)) != hipSuccess ||
        (e = hipMalloc(&s->tokens, cap1 * 4 * c.block_tokens)) != hipSuccess ||
        (e = hipMalloc(&s->slots, slots_n * sizeof(Slot))) != hipSuccess ||
        (e = hipMalloc(&s->ht, sizeof(HashTables))) != hipSuccess ||
        (e = hipMalloc(&s->state, sizeof(DevState))) != hipSuccess) {
        ptstore_destroy(s);
        (void)hipGetLastError();
        return fail(PTSTORE_ERR_NOMEM, "ptstore_create: hipMalloc", e);
    }
    if (!lchunk.empty()) {
        const size_t n = ((size_t)c.num_layers + 1) * sizeof(int64_t);
        s->lbase_host = lbase;
        if ((e = hipMalloc(&s->layer_tab, n)) != hipSuccess ||
            (e = hipMemcpy(s->layer_tab, lbase.data(), n, hipMemcpyHostToDevice)) != hipSuccess) {
            ptstore_destroy(s);
            (void)hipGetLastError();
            return fail(PTSTORE_ERR_NOMEM, "ptstore_create: layer tables", e);
        }
    }
    if (s->tier.host_blocks > 0) {
        void* h = nullptr;
        if ((e = hipHostMalloc(&h, (size_t)s->tier.host_blocks * (size_t)s->block_bytes,
                               hipHostMallocDefault)) != hipSuccess ||
            (e = hipHostGetDevicePointer((void**)&s->tier.host, h, 0)) != hipSuccess) {
            if (h) (void)hipHostFree(h);
            s->tier.host = nullptr;
            ptstore_destroy(s);
            (void)hipGetLastError();
            return fail(PTSTORE_ERR_NOMEM, "ptstore_create: host tier", e);
        }
        s->host_mem = h;
    }
    if (s->tier.replicas > 0) {
        const int64_t R = s->tier.replicas, H = s->tier.host_blocks;
        const int64_t words = (H + kWave - 1) / kWave;
        auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
        const size_t bytes = up(H * 4) + up(R * 4) * 3 + up(words * 8) + up(R * sizeof(Pair));
        if ((e = hipMalloc(&s->tier_mem, bytes)) != hipSuccess ||
            (e = hipMemset(s->tier_mem, 0xFF, bytes)) != hipSuccess) {  // every map entry -1
            ptstore_destroy(s);
            (void)hipGetLastError();
            return fail(PTSTORE_ERR_NOMEM, "ptstore_create: replica map", e);
        }
        uint8_t* q = static_cast<uint8_t*>(s->tier_mem);
        s->tier.rep_of = reinterpret_cast<int32_t*>(q);
        q += up(H * 4);
        s->tier.rep_id = reinterpret_cast<int32_t*>(q);
        q += up(R * 4);
        s->tier.free_list = reinterpret_cast<int32_t*>(q);
        q += up(R * 4);
        s->tier.enter_list = reinterpret_cast<int32_t*>(q);
        q += up(R * 4);
        s->tier.enter_mask = reinterpret_cast<uint64_t*>(q);
        q += up(words * 8);
        s->tier.copies = reinterpret_cast<Pair*>(q);
    }
    if (c.flags & PTSTORE_FLAG_EVICT) {
        const size_t evb = carve_evict(nullptr, s->capacity, &s->evs);
        if ((e = hipMalloc(&s->ev_mem, evb)) != hipSuccess ||
            (e = hipMemset(s->ev_mem, 0, evb)) != hipSuccess) {
            ptstore_destroy(s);
            (void)hipGetLastError();
            return fail(PTSTORE_ERR_NOMEM, "ptstore_create: eviction arrays", e);
        }
        carve_evict(s->ev_mem, s->capacity, &s->evs);
        s->evs.on = 1;
    }
    s->evs.tier = s->tier;
    HashTables h;
    make_hash_tables(c.hash_seed, (c.flags & PTSTORE_FLAG_WEAK_HASH) != 0,
                     (c.flags & PTSTORE_FLAG_WEAK_TAGS) != 0, &h);
    DevState st;
    memset(&st, 0, sizeof st);
    if ((e = hipMemcpy(s->ht, &h, sizeof h, hipMemcpyHostToDevice)) != hipSuccess ||
        (e = hipMemcpy(s->state, &st, sizeof st, hipMemcpyHostToDevice)) != hipSuccess ||
        (e = launch_fill_slots(s->slots, (int64_t)slots_n, nullptr)) != hipSuccess ||
        (e = hipDeviceSynchronize()) != hipSuccess) {
        ptstore_destroy(s);
        return fail(PTSTORE_ERR_HIP, "ptstore_create: initialisation", e);
    }
    *out = s;
    return PTSTORE_OK;
}

int ptstore_destroy(ptstore_t* s) {
    if (!s) return PTSTORE_OK;
    DeviceScope dev(s);
    (void)hipDeviceSynchronize();
    for (auto& v : s->ev)
        for (auto& p : v) {
            (void)hipEventDestroy(p.first);
            (void)hipEventDestroy(p.second);
        }
    for (auto e : s->free_ev) (void)hipEventDestroy(e);
    (void)hipFree(s->pool);
    (void)hipFree(s->parent);
    (void)hipFree(s->tokens);
    (void)hipFree(s->slots);
    (void)hipFree(s->ht);
    (void)hipFree(s->state);
    (void)hipFree(s->insert_scratch);
    for (auto& e : s->copy_scratch) (void)hipFree(e.p);
    (void)hipFree(s->ev_mem);
    (void)hipFree(s->tier_mem);
    (void)hipFree(s->layer_tab);
    if (s->host_mem) (void)hipHostFree(s->host_mem);
    delete s;
    return PTSTORE_OK;
}

int ptstore_lookup(ptstore_t* s, const int32_t* tokens, const int64_t* offsets, int64_t n_tokens,
                   int32_t R, int32_t max_blocks, int32_t* m, int32_t* ids, void* stream) {
    if (!s || !check_batch(s, tokens, offsets, n_tokens, R, max_blocks) || (R > 0 && (!m || !ids)))
        return fail(PTSTORE_ERR_INVALID, "ptstore_lookup: bad argument");
    if (R == 0) return PTSTORE_OK;
    DeviceScope dev(s);
    if (dev.rc) return dev.rc;
    hipStream_t st = (hipStream_t)stream;
    Batch b{tokens, offsets, n_tokens, R, max_blocks};
    hipError_t e;
    {
        Timed t(s, 1, st);
        e = launch_lookup(index_view(s), b, m, ids, st);
    }
    return e == hipSuccess ? PTSTORE_OK : fail(PTSTORE_ERR_HIP, "ptstore_lookup: launch", e);
}

int ptstore_gather_layers(ptstore_t* s, const int32_t* ids, const int32_t* m,
                          const int32_t* block_table, int32_t R, int32_t max_blocks,
                          int32_t layer_begin, int32_t layer_end, void* cache, int64_t cache_blocks,
                          void* stream) {
    if (!s || R < 0 || max_blocks < 1 || (int64_t)R * max_blocks > kMaxEntries || cache_blocks < 0 ||
        (R > 0 && (!ids || !m || !block_table || !cache)) ||
        (reinterpret_cast<uintptr_t>(cache) & 15) != 0 || layer_begin < 0 ||
        layer_end > s->cfg.num_layers || layer_begin >= layer_end)
        return fail(PTSTORE_ERR_INVALID, "ptstore_gather: bad argument");
    s->prep_valid = false;
    if (R == 0) return PTSTORE_OK;
    DeviceScope dev(s);
    if (dev.rc) return dev.rc;
    int rc = PTSTORE_OK;
    hipStream_t st = (hipStream_t)stream;
    void* scr = nullptr;
    uint64_t tcap = 0;
    ptstore::StreamScratch* ent = nullptr;
    rc = copy_scratch_for(s, st, R, max_blocks, &scr, &tcap, &ent, "ptstore_gather: scratch");
    if (rc) return rc;
    CopyScratch sc;
    copy_scratch_carve(scr, R, max_blocks, tcap, &sc);
    const CopyPlan plan = range_plan(s, layer_begin, layer_end);
    hipError_t e;
    {
        Timed t(s, 4, st);
        e = launch_gather_select(plan, sc, ids, m, block_table, R, max_blocks, cache_blocks, st);
    }
    if (e != hipSuccess) ent->dirty = true;
    if (e == hipSuccess) {
        Timed t(s, 0, st);
        e = launch_gather_copy(plan, sc, static_cast<uint8_t*>(cache), cache_blocks, R, max_blocks,
                               layer_begin, layer_end, st);
    }
    return e == hipSuccess ? PTSTORE_OK : fail(PTSTORE_ERR_HIP, "ptstore_gather: launch", e);
}

int ptstore_gather_prepare(ptstore_t* s, const int32_t* ids, const int32_t* m,
                           const int32_t* block_table, int32_t R, int32_t max_blocks,
                           int64_t cache_blocks, void* stream) {
    if (!s || R < 0 || max_blocks < 1 || (int64_t)R * max_blocks > kMaxEntries || cache_blocks < 0 ||
        (R > 0 && (!ids || !m || !block_table)))
        return fail(PTSTORE_ERR_INVALID, "ptstore_gather_prepare: bad argument");
    s->prep_valid = false;
    DeviceScope dev(s);
    if (dev.rc) return dev.rc;
    int rc = PTSTORE_OK;
    hipStream_t st = (hipStream_t)stream;
    if (R > 0) {
        void* scr = nullptr;
        uint64_t tcap = 0;
        ptstore::StreamScratch* ent = nullptr;
        rc = copy_scratch_for(s, st, R, max_blocks, &scr, &tcap, &ent, "ptstore_gather_prepare: scratch");
        if (rc) return rc;
        s->prep_list = scr;
        s->prep_table_cap = tcap;
        CopyScratch sc;
        copy_scratch_carve(scr, R, max_blocks, tcap, &sc);
        hipError_t e;
        {
            Timed t(s, 4, st);
            e = launch_gather_select(copy_plan(s), sc, ids, m, block_table, R, max_blocks,
                                     cache_blocks, st);
        }
        if (e != hipSuccess) {
            ent->dirty = true;
            return fail(PTSTORE_ERR_HIP, "ptstore_gather_prepare: launch", e);
        }
    }
    s->prep_valid = true;
    s->prep_R = R;
    s->prep_max_blocks = max_blocks;
    s->prep_cache_blocks = cache_blocks;
    return PTSTORE_OK;
}

int ptstore_gather_prepared(ptstore_t* s, int32_t layer_begin, int32_t layer_end, void* cache,
                            int64_t cache_blocks, void* stream) {
    if (!s || !s->prep_valid || cache_blocks != s->prep_cache_blocks || layer_begin < 0 ||
        layer_end > s->cfg.num_layers || layer_begin >= layer_end ||
        (s->prep_R > 0 && !cache) || (reinterpret_cast<uintptr_t>(cache) & 15) != 0)
        return fail(PTSTORE_ERR_INVALID, "ptstore_gather_prepared: no prepared list or bad argument");
    if (s->prep_R == 0) return PTSTORE_OK;
    DeviceScope dev(s);
    if (dev.rc) return dev.rc;
    hipStream_t st = (hipStream_t)stream;
    CopyScratch sc;
    copy_scratch_carve(s->prep_list, s->prep_R, s->prep_max_blocks, s->prep_table_cap, &sc);
    hipError_t e;
    {
        Timed t(s, 0, st);
        e = launch_gather_copy(range_plan(s, layer_begin, layer_end), sc, static_cast<uint8_t*>(cache),
                               cache_blocks, s->prep_R, s->prep_max_blocks, layer_begin, layer_end, st);
    }
    return e == hipSuccess ? PTSTORE_OK : fail(PTSTORE_ERR_HIP, "ptstore_gather_prepared: launch", e);
}

int ptstore_gather(ptstore_t* s, const int32_t* ids, const int32_t* m, const int32_t* block_table,
                   int32_t R, int32_t max_blocks, void* cache, int64_t cache_blocks, void* stream) {
    if (!s) return fail(PTSTORE_ERR_INVALID, "ptstore_gather: bad argument");
    return ptstore_gather_layers(s, ids, m, block_table, R, max_blocks, 0, s->cfg.num_layers, cache,
                                 cache_blocks, stream);
}

int ptstore_lookup_gather(ptstore_t* s, const int32_t* tokens, const int64_t* offsets,
                          int64_t n_tokens, int32_t R, int32_t max_blocks, int32_t* m, int32_t* ids,
                          const int32_t* block_table, void* cache, int64_t cache_blocks,
                          void* stream) {
    if (!s || (R > 0 && (!block_table || !cache)) || cache_blocks < 0 ||
        (reinterpret_cast<uintptr_t>(cache) & 15) != 0)
        return fail(PTSTORE_ERR_INVALID, "ptstore_lookup_gather: bad argument");
    int rc = ptstore_lookup(s, tokens, offsets, n_tokens, R, max_blocks, m, ids, stream);
    if (rc) return rc;
    return ptstore_gather(s, ids, m, block_table, R, max_blocks, cache, cache_blocks, stream);
}

int ptstore_lookup_gather_noalloc(ptstore_t* s, const int32_t* tokens, const int64_t* offsets,
                                  int64_t n_tokens, int32_t R, int32_t max_blocks, int32_t* m,
                                  int32_t* ids, const int32_t* block_table, void* cache,
                                  int64_t cache_blocks, void* stream) {
    if (!s || !check_batch(s, tokens, offsets, n_tokens, R, max_blocks) ||
        (R > 0 && (!m || !ids || !block_table || !cache)) || cache_blocks < 0 ||
        (reinterpret_cast<uintptr_t>(cache) & 15) != 0)
        return fail(PTSTORE_ERR_INVALID, "ptstore_lookup_gather_noalloc: bad argument");
    if ((int64_t)R * max_blocks > PTSTORE_NOALLOC_MAX_ENTRIES ||
        copy_table_slots(R, max_blocks) > kNoAllocTableSlots ||
        copy_scratch_bytes(R, max_blocks, kNoAllocTableSlots) > kNoAllocScratchBytes)
        return fail(PTSTORE_ERR_INVALID,
                    "ptstore_lookup_gather_noalloc: R * max_blocks exceeds PTSTORE_NOALLOC_MAX_ENTRIES");
    if (R == 0) return PTSTORE_OK;
    DeviceScope dev(s);
    if (dev.rc) return dev.rc;
    void* sp = static_scratch(s->device);
    if (!sp)
        return fail(PTSTORE_ERR_INVALID, "ptstore_lookup_gather_noalloc: no static scratch on this device");
    hipStream_t st = (hipStream_t)stream;
    Batch b{tokens, offsets, n_tokens, R, max_blocks};
    // the same kernels as ptstore_lookup_gather; no events are recorded, so
    // nothing is created on the way either
    hipError_t e = hipSuccess;
    if (static_dirty(s->device, false))  // a call failed half-way: empty the row table first
        e = launch_zero(sp, copy_scratch_bytes(0, 0, kNoAllocTableSlots) - 256, st);
    if (e == hipSuccess) static_dirty(s->device, true, false);
    if (e == hipSuccess) e = launch_lookup(index_view(s), b, m, ids, st);
    CopyScratch sc;
    copy_scratch_carve(sp, R, max_blocks, kNoAllocTableSlots, &sc);
    const CopyPlan plan = copy_plan(s);
    if (e == hipSuccess) {
        e = launch_gather_select(plan, sc, ids, m, block_table, R, max_blocks, cache_blocks, st);
        if (e != hipSuccess) static_dirty(s->device, true, true);
    }
    if (e == hipSuccess)
        e = launch_gather_copy(plan, sc, static_cast<uint8_t*>(cache), cache_blocks, R, max_blocks, 0,
                               s->cfg.num_layers, st);
    return e == hipSuccess ? PTSTORE_OK
                           : fail(PTSTORE_ERR_HIP, "ptstore_lookup_gather_noalloc: launch", e);
}

int ptstore_insert(ptstore_t* s, const int32_t* tokens, const int64_t* offsets, int64_t n_tokens,
                   int32_t R, int32_t max_blocks, int32_t* m_out, int32_t* ids, uint8_t* created,
                   void* stream) {
    if (!s || !check_batch(s, tokens, offsets, n_tokens, R, max_blocks) ||
        (R > 0 && (!m_out || !ids || !created)))
        return fail(PTSTORE_ERR_INVALID, "ptstore_insert: bad argument");
    s->prep_valid = false;
    if (R == 0) return PTSTORE_OK;
    DeviceScope dev(s);
    if (dev.rc) return dev.rc;
    hipStream_t st = (hipStream_t)stream;
    uint64_t tn;
    const size_t need = insert_scratch_bytes(R, max_blocks, &tn);
    hipError_t e;
    if (need > s->insert_scratch_size && capturing(st))
        return fail(PTSTORE_ERR_INVALID, "a captured insert needs a larger scratch than the store "
                    "has: run an insert of that size before capturing");
    int rc2 = ensure_scratch(&s->insert_scratch, &s->insert_scratch_size, need, st, "ptstore_insert: scratch");
    if (rc2) return rc2;
    InsertScratch sc;
    insert_scratch_carve(s->insert_scratch, R, max_blocks, &sc);
    InsertTarget tgt{s->slots, s->parent, s->tokens, s->capacity};
    Batch b{tokens, offsets, n_tokens, R, max_blocks};
    {
        Timed t(s, 3, st);
        const IndexView ix = index_view(s);
        e = launch_insert_match(ix, tgt, s->evs, b, sc, m_out, ids, created, st);
        if (e == hipSuccess && s->evs.on) {
            Timed te(s, 5, st);
            e = launch_evict(ix, tgt, s->evs, st);
        }
        if (e == hipSuccess) e = launch_insert_commit(ix, tgt, s->evs, b, sc, m_out, ids, created, st);
    }
    return e == hipSuccess ? PTSTORE_OK : fail(PTSTORE_ERR_HIP, "ptstore_insert: launch", e);
}

int ptstore_insert_sync(ptstore_t* s, const int32_t* tokens, const int64_t* offsets,
                        int64_t n_tokens, int32_t R, int32_t max_blocks, int32_t* m_out,
                        int32_t* ids, uint8_t* created, void* stream) {
    if (s && capturing((hipStream_t)stream))
        return fail(PTSTORE_ERR_INVALID, "ptstore_insert_sync waits for its stream: it cannot be "
                    "captured (capture ptstore_insert)");
    const int rc = ptstore_insert(s, tokens, offsets, n_tokens, R, max_blocks, m_out, ids, created,
                                  stream);
    if (rc || R == 0) return rc;
    DeviceScope dev(s);
    if (dev.rc) return dev.rc;
    hipStream_t st = (hipStream_t)stream;
    unsigned long long full = 0;
    hipError_t e = hipMemcpyAsync(&full, &s->state->insert_full, sizeof full, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return fail(PTSTORE_ERR_HIP, "ptstore_insert_sync: status", e);
    return full ? fail(PTSTORE_ERR_FULL, "ptstore_insert_sync: blocks refused for lack of room")
                : PTSTORE_OK;
}

int ptstore_scatter_layers(ptstore_t* s, const int32_t* ids, const uint8_t* created,
                           const int32_t* block_table, int32_t R, int32_t max_blocks,
                           int32_t layer_begin, int32_t layer_end, const void* cache,
                           int64_t cache_blocks, void* stream) {
    if (!s || R < 0 || max_blocks < 1 || (int64_t)R * max_blocks > kMaxEntries || cache_blocks < 0 ||
        (R > 0 && (!ids || !created || !block_table || !cache)) ||
        (reinterpret_cast<uintptr_t>(cache) & 15) != 0 || layer_begin < 0 ||
        layer_end > s->cfg.num_layers || layer_begin >= layer_end)
        return fail(PTSTORE_ERR_INVALID, "ptstore_scatter: bad argument");
    s->prep_valid = false;
    if (R == 0) return PTSTORE_OK;
    DeviceScope dev(s);
    if (dev.rc) return dev.rc;
    int rc = PTSTORE_OK;
    hipStream_t st = (hipStream_t)stream;
    void* scr = nullptr;
    uint64_t tcap = 0;
    ptstore::StreamScratch* ent = nullptr;
    rc = copy_scratch_for(s, st, R, max_blocks, &scr, &tcap, &ent, "ptstore_scatter: scratch");
    if (rc) return rc;
    CopyScratch sc;
    copy_scratch_carve(scr, R, max_blocks, tcap, &sc);
    const CopyPlan plan = copy_plan(s);
    hipError_t e;
    {
        Timed t(s, 4, st);
        e = launch_scatter_select(plan, sc, ids, created, block_table, R, max_blocks, cache_blocks, st);
    }
    if (e == hipSuccess) {
        Timed t(s, 2, st);
        e = launch_scatter_copy(plan, sc, static_cast<const uint8_t*>(cache), cache_blocks, R,
                                max_blocks, layer_begin, layer_end, st);
    }
    return e == hipSuccess ? PTSTORE_OK : fail(PTSTORE_ERR_HIP, "ptstore_scatter: launch", e);
}

int ptstore_scatter(ptstore_t* s, const int32_t* ids, const uint8_t* created,
                    const int32_t* block_table, int32_t R, int32_t max_blocks, const void* cache,
                    int64_t cache_blocks, void* stream) {
    if (!s) return fail(PTSTORE_ERR_INVALID, "ptstore_scatter: bad argument");
    return ptstore_scatter_layers(s, ids, created, block_table, R, max_blocks, 0, s->cfg.num_layers,
                                  cache, cache_blocks, stream);
}

int ptstore_replicate(ptstore_t* s, void* stream) {
    if (!s) return fail(PTSTORE_ERR_INVALID, "ptstore_replicate: null store");
    if (s->tier.replicas == 0)
        return fail(PTSTORE_ERR_INVALID, "ptstore_replicate: store has no replica slots");
    s->prep_valid = false;
    DeviceScope dev(s);
    if (dev.rc) return dev.rc;
    hipStream_t st = (hipStream_t)stream;
    hipError_t e;
    {
        Timed t(s, 6, st);
        e = launch_replicate(index_view(s), s->evs, copy_plan(s), st);
    }
    return e == hipSuccess ? PTSTORE_OK : fail(PTSTORE_ERR_HIP, "ptstore_replicate: launch", e);
}

int ptstore_stats(ptstore_t* s, ptstore_stats_t* out) {
    if (!s || !out) return fail(PTSTORE_ERR_INVALID, "ptstore_stats: null argument");
    DeviceScope dev(s);
    if (dev.rc) return dev.rc;
    DevState st;
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipMemcpy(&st, s->state, sizeof st, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail(PTSTORE_ERR_HIP, "ptstore_stats", e);
    out->blocks_stored = (int64_t)st.count;
    out->capacity = s->capacity;
    out->index_slots = (int64_t)s->slots_n;
    out->block_bytes = s->block_bytes;
    out->chunk_bytes = s->chunk_bytes;
    out->full_events = (int64_t)st.full_events;
    out->bad_entries = (int64_t)st.bad_entries;
    unsigned long long probes = 0, compares = 0, cas = 0, cas_fail = 0;
    for (int i = 0; i < kCounterSlots; ++i) {
        probes += st.slot[i].probes;
        compares += st.slot[i].token_compares;
        cas += st.slot[i].cas_attempts;
        cas_fail += st.slot[i].cas_failures;
    }
    out->probes = (int64_t)probes;
    out->token_compares = (int64_t)compares;
    out->cas_attempts = (int64_t)cas;
    out->cas_failures = (int64_t)cas_fail;
    out->insert_fallbacks = (int64_t)st.insert_fallbacks;
    out->evictions = (int64_t)st.evictions;
    out->clock = (int64_t)st.clock;
    out->index_rebuilds = (int64_t)st.rebuilds;
    out->device_blocks = s->tier.owned;
    out->replicas = (int64_t)st.rep_count;
    out->replica_copies = (int64_t)st.rep_copies;
    return PTSTORE_OK;
}

int ptstore_set_counters(ptstore_t* s, int on) {
    if (!s) return fail(PTSTORE_ERR_INVALID, "ptstore_set_counters: null store");
    if (on)
        s->cfg.flags |= PTSTORE_FLAG_COUNTERS;
    else
        s->cfg.flags &= ~(uint32_t)PTSTORE_FLAG_COUNTERS;
    return PTSTORE_OK;
}

int ptstore_set_timing_kinds(ptstore_t* s, uint32_t kinds) {
    if (!s || (kinds & ~kAllKinds)) return fail(PTSTORE_ERR_INVALID, "ptstore_set_timing_kinds: bad argument");
    s->timing_kinds = kinds;
    if (kinds)
        s->cfg.flags |= PTSTORE_FLAG_TIMING;
    else
        s->cfg.flags &= ~(uint32_t)PTSTORE_FLAG_TIMING;
    return PTSTORE_OK;
}

int ptstore_set_timing(ptstore_t* s, int on) {
    if (!s) return fail(PTSTORE_ERR_INVALID, "ptstore_set_timing: null store");
    return ptstore_set_timing_kinds(s, on ? kAllKinds : 0u);
}

int ptstore_reset_counters(ptstore_t* s) {
    if (!s) return fail(PTSTORE_ERR_INVALID, "ptstore_reset_counters: null store");
    DeviceScope dev(s);
    if (dev.rc) return dev.rc;
    DevState st;
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipMemcpy(&st, s->state, sizeof st, hipMemcpyDeviceToHost);
    if (e == hipSuccess) {
        DevState keep;
        memset(&keep, 0, sizeof keep);
        keep.count = st.count;
        keep.clock = st.clock;
        keep.evictions = st.evictions;
        keep.tombstones = st.tombstones;
        keep.rep_count = st.rep_count;
        keep.rep_copies = st.rep_copies;
        keep.ev_epoch = st.ev_epoch;  // protection marks are compared with it
        keep.insert_full = st.insert_full;
        e = hipMemcpy(s->state, &keep, sizeof keep, hipMemcpyHostToDevice);
    }
    return e == hipSuccess ? PTSTORE_OK : fail(PTSTORE_ERR_HIP, "ptstore_reset_counters", e);
}

int ptstore_get_buffers(ptstore_t* s, ptstore_buffers_t* out) {
    if (!s || !out) return fail(PTSTORE_ERR_INVALID, "ptstore_get_buffers: null argument");
    out->pool = s->pool;
    out->parent = s->parent;
    out->tokens = s->tokens;
    out->slots = s->slots;
    out->capacity = s->capacity;
    out->index_slots = (int64_t)s->slots_n;
    out->freq = s->evs.on ? s->evs.freq : nullptr;
    out->prio = s->evs.on ? s->evs.prio : nullptr;
    out->host_pool = s->host_mem;
    out->host_blocks = s->tier.host_blocks;
    out->device_blocks = s->tier.owned;
    out->replica_of = s->tier.rep_of;
    return PTSTORE_OK;
}

int ptstore_kernel_times(ptstore_t* s, int32_t kind, double* total_ms, int64_t* launches) {
    if (!s || kind < 0 || kind > 6 || !total_ms || !launches)
        return fail(PTSTORE_ERR_INVALID, "ptstore_kernel_times: bad argument");
    DeviceScope dev(s);
    if (dev.rc) return dev.rc;
    double sum = 0;
    int64_t n = 0;
    auto& v = s->ev[kind];
    for (auto& p : v) {
        hipError_t e = hipEventSynchronize(p.second);
        float ms = 0;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.first, p.second);
        if (e != hipSuccess) {  // the pairs read so far are back in the pool: not kept twice
            v.erase(v.begin(), v.begin() + n);
            return fail(PTSTORE_ERR_HIP, "ptstore_kernel_times", e);
        }
        sum += ms;
        ++n;
        s->free_ev.push_back(p.first);
        s->free_ev.push_back(p.second);
    }
    v.clear();
    *total_ms = sum;
    *launches = n;
    return PTSTORE_OK;
}

int ptstore_set_copy_shape(ptstore_t* s, int32_t chunks_per_group, int32_t threads, int32_t grid) {
    if (!s || chunks_per_group < 0 || threads < 0 || grid < 0 ||
        (threads && (threads < 64 || threads > 1024 || threads % 64)))
        return fail(PTSTORE_ERR_INVALID, "ptstore_set_copy_shape: bad argument");
    if (chunks_per_group) {
        s->chunks_per_group = chunks_per_group;
        s->chunks_set = true;
    }
    if (threads) s->threads = threads;
    if (grid) s->grid = grid;
    return PTSTORE_OK;
}

}  // extern "C"
#pragma GCC visibility pop
