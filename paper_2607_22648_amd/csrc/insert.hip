// Deduplicating insert (PTStore Sections 1 and 4: a store keeps only the
// increment beyond the longest common prefix, so stored prefixes grow
// without redundancy like a trie; the new object appends ids for its
// increment, Section 4.1).
//
// The result equals inserting the requests one after another: a missing
// block becomes a new node whose id is the next free one in (request, block)
// order, and a block already created by an earlier request of the batch is
// reused. The GPU gets there without serialising requests:
//
//   lookup     match every request against the store as it was (m0, ids)
//   hash_all   chained keys of every block
//   claim      one thread per request walks its missing blocks b >= m0.
//              Each new block is named by (parent label, its tokens), where
//              the parent label is the stored id of block m0-1 (or the root)
//              for b = m0 and the batch-table slot of block b-1 otherwise.
//              The walk claims or finds that name in a batch hash table by
//              compare-and-swap, so every distinct new block gets exactly
//              one slot, and records the smallest request that needs it.
//   count      per request, the blocks it is the first (smallest r) to need
//   scan       exclusive scan of the counts -> rank base per request; the
//              store count advances, clipped at capacity
//   assign     new id = old count + base[r] + rank within r; ids at or
//              beyond capacity are refused (children rank after parents, so
//              what is refused is always a suffix of a path)
//   publish    ids / created / m_out, block metadata, index slots
//
// Ids come from a scan, never from an atomic counter, so they are
// deterministic and equal the sequential ones.
#include "kernels.hpp"

namespace ptsd {

struct alignas(16) BatchEntry {
    unsigned long long word;  // (parent label << 32) | token position; kEmptyKey if free
    int32_t owner;            // smallest request that needs this block
    int32_t node_id;          // id assigned, -1 if refused
};

namespace {

constexpr int kThreads = 256;
constexpr uint32_t kStoreLabel = 0x80000000u;  // parent label of a stored block: bit 31 | (id + 1)

__global__ void k_table_clear(BatchEntry* __restrict__ t, uint64_t n) {
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x) {
        BatchEntry e;
        e.word = kEmptyKey;
        e.owner = 0x7FFFFFFF;
        e.node_id = -1;
        t[i] = e;
    }
}

__device__ inline bool same_tokens(const int32_t* __restrict__ a, const int32_t* __restrict__ b, int bt) {
    for (int i = 0; i < bt; ++i)
        if (a[i] != b[i]) return false;
    return true;
}

// Blocks of request r considered by this batch (0 for a malformed request).
__device__ inline int32_t n_blocks(const Batch& bat, int64_t r, int bt, int64_t* o0) {
    int64_t a = bat.offsets[r], e = bat.offsets[r + 1];
    if (a < 0 || e < a || e > bat.n_tokens) {
        *o0 = 0;
        return 0;
    }
    *o0 = a;
    int64_t n = (e - a) / bt;
    return (int32_t)(n < bat.max_blocks ? n : bat.max_blocks);
}

struct InsertArgs {
    IndexView ix;
    InsertTarget tgt;
    Batch bat;
    InsertScratch sc;
    int32_t* m_out;
    int32_t* ids;
    uint8_t* created;
};

__global__ __launch_bounds__(kThreads) void k_claim(InsertArgs a) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= a.bat.R) return;
    const int bt = a.ix.block_tokens;
    const int64_t maxb = a.bat.max_blocks;
    int64_t o0;
    const int32_t n = n_blocks(a.bat, r, bt, &o0);
    const int32_t m0 = a.sc.m0[r];
    BatchEntry* __restrict__ tab = reinterpret_cast<BatchEntry*>(a.sc.table);
    const HashTables* __restrict__ ht = a.ix.ht;
    uint32_t plabel = m0 == 0 ? kStoreLabel : (kStoreLabel | (uint32_t)(a.ids[r * maxb + m0 - 1] + 1));
    unsigned long long cas = 0, fails = 0;
    for (int32_t b = m0; b < n; ++b) {
        const uint64_t ik = index_key(a.sc.keys[r * maxb + b], *ht);
        const uint32_t tpos = (uint32_t)(o0 + (int64_t)b * bt);
        const unsigned long long word = ((unsigned long long)plabel << 32) | tpos;
        uint64_t pos = slot_of(ik, ~ht->slot_seed, a.sc.table_mask);
        while (true) {
            const unsigned long long prev = atomicCAS(&tab[pos].word, kEmptyKey, word);
            ++cas;
            if (prev == kEmptyKey) break;
            if ((uint32_t)(prev >> 32) == plabel &&
                same_tokens(a.bat.tokens + (uint32_t)prev, a.bat.tokens + tpos, bt))
                break;
            ++fails;
            pos = (pos + 1) & a.sc.table_mask;
        }
        atomicMin(&tab[pos].owner, (int32_t)r);
        a.sc.label[r * maxb + b] = (int32_t)pos;
        plabel = (uint32_t)pos;
    }
    if (a.ix.counters) {
        if (cas) atomicAdd(&a.ix.state->cas_attempts, cas);
        if (fails) atomicAdd(&a.ix.state->cas_failures, fails);
    }
}

__global__ __launch_bounds__(kThreads) void k_count(InsertArgs a) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= a.bat.R) return;
    const int64_t maxb = a.bat.max_blocks;
    int64_t o0;
    const int32_t n = n_blocks(a.bat, r, a.ix.block_tokens, &o0);
    const BatchEntry* __restrict__ tab = reinterpret_cast<const BatchEntry*>(a.sc.table);
    int32_t c = 0;
    for (int32_t b = a.sc.m0[r]; b < n; ++b) c += tab[a.sc.label[r * maxb + b]].owner == (int32_t)r;
    a.sc.cnt[r] = c;
}

// One workgroup: exclusive scan of cnt into base, then advance the count.
__global__ __launch_bounds__(1024) void k_scan(InsertArgs a) {
    __shared__ long long part[1024];
    const int R = a.bat.R;
    const int t = threadIdx.x, nt = blockDim.x;
    const int per = (R + nt - 1) / nt;
    const int lo = min(R, t * per), hi = min(R, lo + per);
    long long s = 0;
    for (int i = lo; i < hi; ++i) s += a.sc.cnt[i];
    part[t] = s;
    __syncthreads();
    // Hillis-Steele inclusive scan over the per-thread sums
    for (int d = 1; d < nt; d <<= 1) {
        long long v = t >= d ? part[t - d] : 0;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    long long run = part[t] - s;
    for (int i = lo; i < hi; ++i) {
        a.sc.base[i] = (int32_t)run;
        run += a.sc.cnt[i];
    }
    if (t == nt - 1) {
        const long long total = part[nt - 1];
        DevState* st = a.ix.state;
        const long long old = (long long)st->count;
        const long long cap = a.tgt.capacity;
        st->insert_old_count = (unsigned long long)old;
        if (old + total > cap) {
            st->full_events += 1;
            st->count = (unsigned long long)cap;
        } else {
            st->count = (unsigned long long)(old + total);
        }
    }
}

__global__ __launch_bounds__(kThreads) void k_assign(InsertArgs a) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= a.bat.R) return;
    const int64_t maxb = a.bat.max_blocks;
    int64_t o0;
    const int32_t n = n_blocks(a.bat, r, a.ix.block_tokens, &o0);
    BatchEntry* __restrict__ tab = reinterpret_cast<BatchEntry*>(a.sc.table);
    const long long old = (long long)a.ix.state->insert_old_count;
    long long id = old + a.sc.base[r];
    for (int32_t b = a.sc.m0[r]; b < n; ++b) {
        BatchEntry* e = &tab[a.sc.label[r * maxb + b]];
        if (e->owner == (int32_t)r) {
            e->node_id = id < a.tgt.capacity ? (int32_t)id : -1;
            ++id;
        }
    }
}

__global__ __launch_bounds__(kThreads) void k_publish(InsertArgs a) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= a.bat.R) return;
    const int bt = a.ix.block_tokens;
    const int64_t maxb = a.bat.max_blocks;
    int64_t o0;
    const int32_t n = n_blocks(a.bat, r, bt, &o0);
    const int32_t m0 = a.sc.m0[r];
    const BatchEntry* __restrict__ tab = reinterpret_cast<const BatchEntry*>(a.sc.table);
    const HashTables* __restrict__ ht = a.ix.ht;
    int32_t* __restrict__ row = a.ids + r * maxb;
    uint8_t* __restrict__ crow = a.created + r * maxb;
    int32_t parent = m0 == 0 ? -1 : row[m0 - 1];
    int32_t m = m0;
    unsigned long long cas = 0, fails = 0;
    for (int32_t b = 0; b < m0; ++b) crow[b] = 0;
    for (int32_t b = m0; b < n; ++b) {
        const BatchEntry e = tab[a.sc.label[r * maxb + b]];
        if (e.node_id < 0) break;
        const int32_t id = e.node_id;
        row[b] = id;
        const bool mine = e.owner == (int32_t)r;
        crow[b] = mine ? 1 : 0;
        if (mine) {
            a.tgt.parent[id] = parent;
            const int32_t* src = a.bat.tokens + o0 + (int64_t)b * bt;
            int32_t* dst = a.tgt.tokens + (int64_t)id * bt;
            for (int i = 0; i < bt; ++i) dst[i] = src[i];
            const uint64_t ik = index_key(a.sc.keys[r * maxb + b], *ht);
            uint64_t pos = slot_of(ik, ht->slot_seed, a.ix.slot_mask);
            Slot* slots = a.tgt.slots;
            while (true) {
                const unsigned long long prev =
                    atomicCAS(reinterpret_cast<unsigned long long*>(&slots[pos].key), kEmptyKey,
                              (unsigned long long)ik);
                ++cas;
                if (prev == kEmptyKey) {
                    slots[pos].id = id;
                    slots[pos].parent = parent;
                    break;
                }
                ++fails;
                pos = (pos + 1) & a.ix.slot_mask;
            }
        }
        parent = id;
        m = b + 1;
    }
    for (int32_t b = m; b < maxb; ++b) crow[b] = 0;
    for (int32_t b = m; b < n; ++b) row[b] = -1;
    a.m_out[r] = m;
    if (a.ix.counters) {
        if (cas) atomicAdd(&a.ix.state->cas_attempts, cas);
        if (fails) atomicAdd(&a.ix.state->cas_failures, fails);
    }
}

}  // namespace

size_t insert_scratch_bytes(int32_t R, int32_t max_blocks, uint64_t* table_entries) {
    const uint64_t rb = (uint64_t)R * (uint64_t)max_blocks;
    uint64_t t = 64;
    while (t < 2 * rb) t <<= 1;
    *table_entries = t;
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    return up(rb * 8) + up((size_t)R * 4) + up(rb * 4) + up((size_t)R * 4) * 2 + up(t * sizeof(BatchEntry));
}

void insert_scratch_carve(void* base, int32_t R, int32_t max_blocks, InsertScratch* out) {
    uint64_t t;
    insert_scratch_bytes(R, max_blocks, &t);
    const uint64_t rb = (uint64_t)R * (uint64_t)max_blocks;
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    uint8_t* p = static_cast<uint8_t*>(base);
    out->keys = reinterpret_cast<uint64_t*>(p);
    p += up(rb * 8);
    out->m0 = reinterpret_cast<int32_t*>(p);
    p += up((size_t)R * 4);
    out->label = reinterpret_cast<int32_t*>(p);
    p += up(rb * 4);
    out->cnt = reinterpret_cast<int32_t*>(p);
    p += up((size_t)R * 4);
    out->base = reinterpret_cast<int32_t*>(p);
    p += up((size_t)R * 4);
    out->table = p;
    out->table_mask = t - 1;
}

hipError_t launch_insert(const IndexView& ix, const InsertTarget& tgt, const Batch& b,
                         const InsertScratch& sc, int32_t* m_out, int32_t* ids, uint8_t* created,
                         hipStream_t s) {
    hipError_t e;
    if ((e = launch_lookup(ix, b, sc.m0, ids, s)) != hipSuccess) return e;
    if ((e = launch_hash_all(ix, b, sc.keys, s)) != hipSuccess) return e;
    const uint64_t tn = sc.table_mask + 1;
    const unsigned cgrid = (unsigned)((tn + kThreads - 1) / kThreads < 65536 ? (tn + kThreads - 1) / kThreads : 65536);
    hipLaunchKernelGGL(k_table_clear, dim3(cgrid), dim3(kThreads), 0, s,
                       reinterpret_cast<BatchEntry*>(sc.table), tn);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    InsertArgs a{ix, tgt, b, sc, m_out, ids, created};
    const unsigned grid = (unsigned)((b.R + kThreads - 1) / kThreads);
    hipLaunchKernelGGL(k_claim, dim3(grid), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_count, dim3(grid), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_assign, dim3(grid), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_publish, dim3(grid), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace ptsd
