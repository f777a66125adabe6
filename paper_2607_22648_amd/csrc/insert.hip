// Deduplicating insert (PTStore Sections 1 and 4: a store keeps only the
// increment beyond the longest common prefix, so stored prefixes grow
// without redundancy like a trie; the new object appends ids for its
// increment, Section 4.1).
//
// The result equals inserting the requests one after another: a missing
// block becomes a new node whose id is the next free one in (request, block)
// order, and a block already created by an earlier request of the batch is
// reused. The GPU gets there without serialising requests or blocks:
//
//   lookup     match every request against the store as it was (m0, ids)
//   hash_all   chained keys of every block (the key of block b is a function
//              of the whole prefix up to b)
//   claim      wave per request, lane per missing block b >= m0: the block
//              claims or joins the batch-table entry named by (key, depth)
//              and records in it the smallest request that needs it; the
//              block that claims an entry also records its depth there
//   verify     wave per request, lane per block: the entry must hold the
//              block's depth (else blocks of two depths, possibly of one
//              request, share it), and the entry's smallest request o must
//              hold the same prefix. It does if block b's tokens are
//              equal and either b is both requests' first missing block under
//              the same stored parent, or both requests' blocks b-1 sit in
//              the same entry (by induction, equal prefixes). Any failure --
//              a collision of names between different prefixes -- raises a
//              flag.
//   exact      only when the flag is up: the table is cleared and rebuilt one
//              block after another per request, each block named exactly by
//              (entry of its parent, its tokens); slower, same result
//   count      per request, the blocks it is the first (smallest r) to need
//   scan       exclusive scan of the counts -> rank base per request; the
//              store count advances, clipped at capacity
//   assign     new id = old count + base[r] + rank within r (wave ballot);
//              ids at or beyond capacity are refused (children rank after
//              parents, so what is refused is always a suffix of a path)
//   publish    ids / created / m_out, block metadata, index slots
//
// Ids come from a scan, never from an atomic counter, so they are
// deterministic and equal the sequential ones.
//
// With eviction on, count also marks the blocks the batch matched
// (protected), scan computes how many blocks must be evicted, evict.hip
// frees them between scan and assign, assign hands out never-used ids and
// then the freed ones, publish may take a deleted index slot, and the
// resident paths are accessed last.
#include "kernels.hpp"

namespace ptsd {

struct alignas(16) BatchEntry {
    unsigned long long word;  // claim: tag of (key, depth); exact: (parent label << 32) | token position
    int32_t owner;            // smallest request that needs this block
    int32_t node_id;          // claim to verify: depth of the claiming block (exact path: -1);
                              // from assign on: id assigned, -1 if refused
};

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr uint32_t kStoreLabel = 0x80000000u;  // parent label of a stored block: bit 31 | (id + 1)

__device__ inline unsigned long long lanes_below(int lane) {
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Clears the batch table. The first clear of an insert (only_if_collision =
// 0) also lowers the collision flag; the second runs only if it was raised.
// The insert's first kernel (only_if_collision = 0) also advances the
// eviction epoch, so that a replayed capture marks its own matches.
__global__ void k_table_clear(BatchEntry* __restrict__ t, uint64_t n, unsigned int* collision,
                              int only_if_collision, DevState* st, int ev_on) {
    if (only_if_collision && *collision == 0) return;
    if (!only_if_collision && blockIdx.x == 0 && threadIdx.x == 0) {
        *collision = 0;
        if (ev_on) {  // protection marks are compared with it; 0 marks nothing
            const unsigned long long e = st->ev_epoch + 1;
            st->ev_epoch = e >= 0x7FFFFFFFull ? 1ull : e;
        }
    }
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

// Name of a new block in the batch table: its chained key and its depth
// (only the depth's parity with the weak test tags). The top bit is clear,
// so a tag never equals the empty marker.
__device__ inline unsigned long long tag_of(uint64_t key, int32_t b, const HashTables& ht) {
    const uint64_t d = ht.weak_tag ? (uint64_t)(b & 1) : (uint64_t)b;
    return mix64(index_key(key, ht) ^ (0x9E3779B97F4A7C15ull * (d + 1)) ^ ~ht.slot_seed) &
           0x7FFFFFFFFFFFFFFFull;
}

struct InsertArgs {
    IndexView ix;
    InsertTarget tgt;
    EvictView ev;
    Batch bat;
    InsertScratch sc;
    int32_t* m_out;
    int32_t* ids;
    uint8_t* created;
};

__device__ inline void count_cas(const InsertArgs& a, unsigned long long cas,
                                 unsigned long long fails, int lane) {
    if (!a.ix.counters) return;
    CounterSlot* cs = counter_slot(a.ix.state);
    wave_count(&cs->cas_attempts, cas, lane);
    wave_count(&cs->cas_failures, fails, lane);
}

__global__ __launch_bounds__(kThreads) void k_claim(InsertArgs a) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r = (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave;
    if (r >= a.bat.R) return;
    const int64_t maxb = a.bat.max_blocks;
    int64_t o0;
    const int32_t n = n_blocks(a.bat, r, a.ix.block_tokens, &o0);
    const int32_t m0 = a.sc.m0[r];
    BatchEntry* __restrict__ tab = reinterpret_cast<BatchEntry*>(a.sc.table);
    unsigned long long cas = 0, fails = 0;
    for (int32_t w0 = m0; w0 < n; w0 += kWave) {
        const int32_t b = w0 + lane;
        if (b >= n) continue;
        const unsigned long long tag = tag_of(a.sc.keys[r * maxb + b], b, *a.ix.ht);
        uint64_t pos = tag & a.sc.table_mask;
        while (true) {
            const unsigned long long prev = atomicCAS(&tab[pos].word, kEmptyKey, tag);
            ++cas;
            if (prev == kEmptyKey) {
                tab[pos].node_id = b;  // read by verify, kernels later
                break;
            }
            if (prev == tag) break;
            ++fails;
            pos = (pos + 1) & a.sc.table_mask;
        }
        atomicMin(&tab[pos].owner, (int32_t)r);
        a.sc.label[r * maxb + b] = (int32_t)pos;
    }
    count_cas(a, cas, fails, lane);
}

__global__ __launch_bounds__(kThreads) void k_verify(InsertArgs a) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r = (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave;
    if (r >= a.bat.R) return;
    const int bt = a.ix.block_tokens;
    const int64_t maxb = a.bat.max_blocks;
    int64_t o0;
    const int32_t n = n_blocks(a.bat, r, bt, &o0);
    const int32_t m0 = a.sc.m0[r];
    const BatchEntry* __restrict__ tab = reinterpret_cast<const BatchEntry*>(a.sc.table);
    bool ok = true;
    for (int32_t w0 = m0; w0 < n; w0 += kWave) {
        const int32_t b = w0 + lane;
        if (b >= n) continue;
        const BatchEntry te = tab[a.sc.label[r * maxb + b]];
        if (te.node_id != b) {  // the entry was claimed at another depth
            ok = false;
            continue;
        }
        const int64_t o = te.owner;
        if (o == r) continue;
        int64_t oo0;
        const int32_t on = n_blocks(a.bat, o, bt, &oo0);
        const int32_t om0 = a.sc.m0[o];
        bool good = b < on && b >= om0 &&
                    same_tokens(a.bat.tokens + oo0 + (int64_t)b * bt, a.bat.tokens + o0 + (int64_t)b * bt, bt);
        if (good) {
            if (b == m0)
                good = om0 == b && (b == 0 || a.ids[o * maxb + b - 1] == a.ids[r * maxb + b - 1]);
            else
                good = om0 <= b - 1 && a.sc.label[o * maxb + b - 1] == a.sc.label[r * maxb + b - 1];
        }
        ok &= good;
    }
    if (!ok) *a.sc.collision = 1;
}

// Exact claim, one block after another per request (runs only on a collision).
__global__ __launch_bounds__(kThreads) void k_claim_exact(InsertArgs a) {
    if (*a.sc.collision == 0) return;
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r == 0) atomicAdd(&a.ix.state->insert_fallbacks, 1ull);
    if (r >= a.bat.R) return;
    const int bt = a.ix.block_tokens;
    const int64_t maxb = a.bat.max_blocks;
    int64_t o0;
    const int32_t n = n_blocks(a.bat, r, bt, &o0);
    const int32_t m0 = a.sc.m0[r];
    BatchEntry* __restrict__ tab = reinterpret_cast<BatchEntry*>(a.sc.table);
    const HashTables* __restrict__ ht = a.ix.ht;
    uint32_t plabel = m0 == 0 ? kStoreLabel : (kStoreLabel | (uint32_t)(a.ids[r * maxb + m0 - 1] + 1));
    for (int32_t b = m0; b < n; ++b) {
        const uint64_t ik = index_key(a.sc.keys[r * maxb + b], *ht);
        const uint32_t tpos = (uint32_t)(o0 + (int64_t)b * bt);
        const unsigned long long word = ((unsigned long long)plabel << 32) | tpos;
        uint64_t pos = slot_of(ik, ~ht->slot_seed, a.sc.table_mask);
        while (true) {
            const unsigned long long prev = atomicCAS(&tab[pos].word, kEmptyKey, word);
            if (prev == kEmptyKey) break;
            if ((uint32_t)(prev >> 32) == plabel &&
                same_tokens(a.bat.tokens + (uint32_t)prev, a.bat.tokens + tpos, bt))
                break;
            pos = (pos + 1) & a.sc.table_mask;
        }
        atomicMin(&tab[pos].owner, (int32_t)r);
        a.sc.label[r * maxb + b] = (int32_t)pos;
        plabel = (uint32_t)pos;
    }
}

__global__ __launch_bounds__(kThreads) void k_count(InsertArgs a) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r = (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave;
    if (r >= a.bat.R) return;
    const int64_t maxb = a.bat.max_blocks;
    int64_t o0;
    const int32_t n = n_blocks(a.bat, r, a.ix.block_tokens, &o0);
    const BatchEntry* __restrict__ tab = reinterpret_cast<const BatchEntry*>(a.sc.table);
    if (a.ev.on) {  // the blocks this request matched cannot be evicted by this insert
        const int32_t epoch = (int32_t)a.ix.state->ev_epoch;
        for (int32_t b = lane; b < a.sc.m0[r]; b += kWave) a.ev.prot[a.ids[r * maxb + b]] = epoch;
    }
    int32_t c = 0;
    for (int32_t w0 = a.sc.m0[r]; w0 < n; w0 += kWave) {
        const int32_t b = w0 + lane;
        const bool mine = b < n && tab[a.sc.label[r * maxb + b]].owner == (int32_t)r;
        c += __popcll(ballot64(mine));
    }
    if (lane == 0) a.sc.cnt[r] = c;
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
    DevState* st = a.ix.state;
    if (a.ev.on && t < kSelPasses) st->sel_done[t] = 0;  // fresh selection state for evict.hip
    if (t == nt - 1) {
        const long long total = part[nt - 1];
        const long long old = (long long)st->count;
        const long long cap = a.tgt.capacity;
        st->insert_old_count = (unsigned long long)old;
        st->insert_full = 0;
        if (old + total > cap) {
            if (!a.ev.on) {  // with eviction: decided once victims are known
                st->full_events += 1;
                st->insert_full = 1;
            }
            st->count = (unsigned long long)cap;
        } else {
            st->count = (unsigned long long)(old + total);
        }
        if (a.ev.on) {
            const long long want = total - (cap - old);
            st->ev_new = (unsigned long long)total;
            st->ev_want = want > 0 ? (unsigned long long)want : 0ull;
            st->ev_all = 0;
            st->ev_nv = 0;
            st->sel_range_done = 0;
            st->sel_npass = 0;
            st->sel_hot = 0;
            st->sel_lo_id = 0;
            st->sel_hi_id = (unsigned long long)old;
            st->sel_hi = 0;
            st->sel_lo = 0;
            st->sel_need = st->ev_want;
        }
    }
}

__global__ __launch_bounds__(kThreads) void k_assign(InsertArgs a) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r = (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave;
    if (r >= a.bat.R) return;
    const int64_t maxb = a.bat.max_blocks;
    int64_t o0;
    const int32_t n = n_blocks(a.bat, r, a.ix.block_tokens, &o0);
    BatchEntry* __restrict__ tab = reinterpret_cast<BatchEntry*>(a.sc.table);
    const long long old = (long long)a.ix.state->insert_old_count;
    const long long fresh = a.tgt.capacity - old;                        // never-used ids
    const long long nv = a.ev.on ? (long long)a.ix.state->ev_nv : 0;    // freed ids
    long long run = a.sc.base[r];  // rank among the batch's new blocks
    for (int32_t w0 = a.sc.m0[r]; w0 < n; w0 += kWave) {
        const int32_t b = w0 + lane;
        BatchEntry* e = b < n ? &tab[a.sc.label[r * maxb + b]] : nullptr;
        const bool mine = e && e->owner == (int32_t)r;
        const unsigned long long mask = ballot64(mine);
        if (mine) {
            const long long k = run + __popcll(mask & lanes_below(lane));
            int32_t id = -1;
            if (k < fresh)
                id = (int32_t)(old + k);
            else if (k - fresh < nv)
                id = a.ev.victims[k - fresh];
            e->node_id = id;
            if (a.ev.on && id >= 0) {  // a new block starts unaccessed, with no resident child
                a.ev.freq[id] = 0;
                a.ev.prio[id] = 0;
                a.ev.live[id] = 0;
                a.ev.prot[id] = 0;
                a.ev.depth[id] = b;
            }
        }
        run += __popcll(mask);
    }
}

__global__ __launch_bounds__(kThreads) void k_publish(InsertArgs a) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r = (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave;
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
    for (int32_t b = lane; b < maxb; b += kWave)
        if (b < m0 || b >= n) crow[b] = 0;
    int32_t carry = m0 == 0 ? -1 : row[m0 - 1];  // id of the block before the window
    int32_t m = n;                               // resident blocks after the call
    unsigned long long cas = 0, fails = 0, tombs_taken = 0;
    for (int32_t w0 = m0; w0 < n; w0 += kWave) {
        const int32_t b = w0 + lane;
        const bool valid = b < n;
        BatchEntry e;
        e.node_id = -1;
        e.owner = -1;
        if (valid) e = tab[a.sc.label[r * maxb + b]];
        const unsigned long long refused = ballot64(valid && e.node_id < 0);
        if (refused) {
            const int32_t cut = w0 + __ffsll((long long)refused) - 1;
            m = cut < m ? cut : m;
        }
        int32_t parent = __shfl_up(e.node_id, 1, kWave);
        if (lane == 0) parent = carry;
        carry = __shfl(e.node_id, kWave - 1, kWave);
        if (!valid) continue;
        if (b >= m) {
            row[b] = -1;
            crow[b] = 0;
            continue;
        }
        const int32_t id = e.node_id;
        row[b] = id;
        const bool mine = e.owner == (int32_t)r;
        crow[b] = mine ? 1 : 0;
        if (!mine) continue;
        a.tgt.parent[id] = parent;
        const int32_t* src = a.bat.tokens + o0 + (int64_t)b * bt;
        int32_t* dst = a.tgt.tokens + (int64_t)id * bt;
        for (int i = 0; i < bt; ++i) dst[i] = src[i];
        const uint64_t ik = index_key(a.sc.keys[r * maxb + b], *ht);
        uint64_t pos = slot_of(ik, ht->slot_seed, a.ix.slot_mask);
        Slot* slots = a.tgt.slots;
        // at most half the slots hold blocks and at most a quarter are
        // deleted, so a free slot is always found
        for (uint64_t step = 0; step <= a.ix.slot_mask; ++step) {
            unsigned long long* kp = reinterpret_cast<unsigned long long*>(&slots[pos].key);
            unsigned long long prev = atomicCAS(kp, kEmptyKey, (unsigned long long)ik);
            ++cas;
            bool got = prev == kEmptyKey;
            if (!got && a.ev.on && prev == kTombKey) {
                prev = atomicCAS(kp, kTombKey, (unsigned long long)ik);
                ++cas;
                got = prev == kTombKey;
                tombs_taken += got ? 1 : 0;
            }
            if (got) {
                slots[pos].id = id;
                slots[pos].parent = parent;
                break;
            }
            ++fails;
            pos = (pos + 1) & a.ix.slot_mask;
        }
        if (a.ev.on) {  // (the rest was reset by assign, before any child counts itself here)
            a.ev.nkey[id] = ik;
            a.ev.spos[id] = (uint32_t)pos;
            if (parent >= 0) atomicAdd(&a.ev.live[parent], 1);
        }
    }
    if (lane == 0) a.m_out[r] = m;
    count_cas(a, cas, fails, lane);
    if (a.ev.on) wave_sub(&a.ix.state->tombstones, tombs_taken, lane);
}

}  // namespace

size_t insert_scratch_bytes(int32_t R, int32_t max_blocks, uint64_t* table_entries) {
    const uint64_t rb = (uint64_t)R * (uint64_t)max_blocks;
    uint64_t t = 64;
    while (t < 2 * rb) t <<= 1;
    *table_entries = t;
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    return up(rb * 8) + up((size_t)R * 4) + up(rb * 4) + up((size_t)R * 4) * 2 +
           up(t * sizeof(BatchEntry)) + 256;
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
    p += up(t * sizeof(BatchEntry));
    out->collision = reinterpret_cast<unsigned int*>(p);
}

hipError_t launch_insert_match(const IndexView& ix, const InsertTarget& tgt, const EvictView& ev,
                               const Batch& b, const InsertScratch& sc, int32_t* m_out, int32_t* ids,
                               uint8_t* created, hipStream_t s) {
    hipError_t e;
    IndexView quiet = ix;  // the insert's own match is not an access
    quiet.freq = nullptr;
    quiet.prio = nullptr;
    if ((e = launch_lookup(quiet, b, sc.m0, ids, s)) != hipSuccess) return e;
    if ((e = launch_hash_all(ix, b, sc.keys, s)) != hipSuccess) return e;
    const uint64_t tn = sc.table_mask + 1;
    const uint64_t cg = (tn + kThreads - 1) / kThreads;
    const unsigned cgrid = (unsigned)(cg < 65536 ? cg : 65536);
    BatchEntry* table = reinterpret_cast<BatchEntry*>(sc.table);
    InsertArgs a{quiet, tgt, ev, b, sc, m_out, ids, created};
    const unsigned wgrid = (unsigned)((b.R + kWaves - 1) / kWaves);      // wave per request
    const unsigned tgrid = (unsigned)((b.R + kThreads - 1) / kThreads);  // thread per request
    hipLaunchKernelGGL(k_table_clear, dim3(cgrid), dim3(kThreads), 0, s, table, tn, sc.collision, 0,
                       ix.state, ev.on);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_claim, dim3(wgrid), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_verify, dim3(wgrid), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_table_clear, dim3(cgrid), dim3(kThreads), 0, s, table, tn, sc.collision, 1,
                       ix.state, 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_claim_exact, dim3(tgrid), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_count, dim3(wgrid), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_insert_commit(const IndexView& ix, const InsertTarget& tgt, const EvictView& ev,
                                const Batch& b, const InsertScratch& sc, int32_t* m_out, int32_t* ids,
                                uint8_t* created, hipStream_t s) {
    hipError_t e;
    IndexView quiet = ix;
    quiet.freq = nullptr;
    quiet.prio = nullptr;
    InsertArgs a{quiet, tgt, ev, b, sc, m_out, ids, created};
    const unsigned wgrid = (unsigned)((b.R + kWaves - 1) / kWaves);
    hipLaunchKernelGGL(k_assign, dim3(wgrid), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_publish, dim3(wgrid), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev.on) return launch_touch_paths(quiet, ev, m_out, ids, b.R, b.max_blocks, s);
    return hipSuccess;
}

}  // namespace ptsd
