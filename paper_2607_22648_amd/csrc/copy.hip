// KV block movement between the store's pool and a caller's paged cache.
//
// Gather is the load of Section 4.1 (iterate over an object's ids and copy
// their tensors into application-supplied GPU memory); scatter stores the
// tensors of blocks an insert created. Both move whole (layer, K|V) chunks
// of heads x slots x dim elements, which are contiguous on both sides:
//   pool  [row][layer][K|V][head][slot][dim]       chunk c at row*block + c*chunk
//   cache [layer][K|V][cache block][head][slot][dim] chunk c at (c*NB + cb)*chunk
// (chunk c = layer c/2, K or V by c%2). With per-layer slab sizes, layer l's
// slabs are lchunk[l] bytes: at row*block + lbase[l] + kv*lchunk[l] in the
// pool, at NB*lbase[l] + (kv*NB + cb)*lchunk[l] in the cache. A call may
// move a range of layers only.
// A block's row is where its bytes are read from: its home in device memory,
// a device replica of a host-tier block, or its home in the pinned host tier
// (rows past the device pool), which the same kernel reads over the host
// link.
//
// A call runs in two parts, like the paper's bulk transfer of a list of
// (offset, size) segments in one request (Section 4.1, RDMA-aware
// consolidation):
//   select  count the blocks each request must move (wave per request), scan
//           the counts, then write a dense list of (row, cache block)
//           entries, compacted with a wave ballot (three kernels; one
//           workgroup does all three for a small batch). Entries with an id
//           or cache block out of range are dropped here and counted.
//   group   (a gather of several requests) the entries are grouped by the
//           row they read: a row table in the scratch (in LDS for a small
//           batch) counts each row's entries, and each row gets slices of
//           up to kSliceDests of its cache blocks. A row that many requests
//           share is then read from memory once per slice, not once per
//           request. A scatter, and a gather of one request (whose blocks
//           are distinct), keep one slice per entry.
//   copy    workgroups walk (descriptor, group of chunks) units; the number
//           of units is read on the device, so no host round trip separates
//           the parts. Threads move 16-byte vectors with non-temporal loads
//           and stores (the stream is touched once); a gather writes each
//           vector it reads to every cache block of its slice.
// Only blocks that are really copied cost work, however sparse they are in
// the [request][block] arrays (a few created blocks per insert, half the
// requests missing the store). The default copy shape gives each
// 1024-thread workgroup one chunk per unit (two vectors per thread for a
// 32 KiB chunk). The copies are pure HBM streaming: no MFMA. LDS holds the
// row tables of the grouping step and the per-layer kernel's table of layer
// bases.
#include "kernels.hpp"

namespace ptsd {
namespace {

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

constexpr int kUnroll = 8;
constexpr int kSelThreads = 256;
constexpr int kSelWaves = kSelThreads / kWave;

__device__ inline v4u ld_nt(const v4u* p) { return __builtin_nontemporal_load(p); }
__device__ inline void st_nt(v4u* p, v4u v) { __builtin_nontemporal_store(v, p); }

// Copy n16 16-byte vectors with blockDim.x threads.
__device__ inline void copy_span(const v4u* __restrict__ src, v4u* __restrict__ dst, int n16) {
    const int nt = blockDim.x;
    int i = threadIdx.x;
    for (; i + (kUnroll - 1) * nt < n16; i += kUnroll * nt) {
        v4u v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) v[u] = ld_nt(src + i + u * nt);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) st_nt(dst + i + u * nt, v[u]);
    }
    for (; i < n16; i += nt) st_nt(dst + i, ld_nt(src + i));
}

struct SelectArgs {
    const int32_t* ids;
    const int32_t* m;          // gather: blocks b < m[r] are moved
    const uint8_t* created;    // scatter: blocks with created != 0 are moved
    const int32_t* block_table;
    int32_t R;
    int32_t max_blocks;
    int64_t cache_blocks;
    DevState* state;
    CopyScratch sc;
    TierView tier;
    int32_t group;             // gather: 1 = group the entries by row (R >= 2)
};

// The row a gather reads block `id` from: its device home, its replica, or
// its host-tier home.
__device__ inline int32_t gather_row(const TierView& t, int32_t id) {
    if (id < t.owned) return id;
    const int64_t h = id - t.owned;
    if (t.rep_of) {
        const int32_t slot = t.rep_of[h];
        if (slot >= 0) return (int32_t)(t.owned + slot);
    }
    return (int32_t)(t.dev_rows + h);
}

// The row a scatter writes block `id` to: always its home.
__device__ inline int32_t home_row(const TierView& t, int32_t id) {
    return id < t.owned ? id : (int32_t)(t.dev_rows + (id - t.owned));
}

// Should (r, b) be moved? Sets *bad for an entry out of range.
template <bool GATHER>
__device__ inline bool selected(const SelectArgs& a, int64_t rb, unsigned long long count,
                                Pair* out, bool* bad) {
    // every load before any test (the three arrays are [R][max_blocks], so
    // the loads are in bounds): with no branch between them and their use
    // they are issued together and cost one trip instead of two or three
    const bool made = GATHER || a.created[rb] != 0;
    const int32_t cb = a.block_table[rb];
    const int32_t id = a.ids[rb];
    const bool skip = !made | (cb < 0);
    const bool out_of_range = ((int64_t)cb >= a.cache_blocks) | (id < 0) |
                              ((unsigned long long)id >= count);
    *bad = !skip & out_of_range;
    if (skip | out_of_range) return false;
    out->row = GATHER ? gather_row(a.tier, id) : home_row(a.tier, id);
    out->cb = cb;
    return true;
}

template <bool GATHER>
__device__ inline int32_t row_len(const SelectArgs& a, int64_t r) {
    if (!GATHER) return a.max_blocks;
    const int32_t mr = a.m[r];
    return mr < 0 ? 0 : (mr < a.max_blocks ? mr : a.max_blocks);
}

__device__ inline unsigned long long lanes_below(int lane) {
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Request r's blocks to move, counted by the whole wave: in device rows, in
// host-tier rows, and entries out of range (added to *bad).
template <bool GATHER>
__device__ inline void count_row(const SelectArgs& a, int64_t r, int lane, unsigned long long count,
                                 int32_t* cnt, int32_t* cnt_h, int32_t* bad) {
    const int32_t n = row_len<GATHER>(a, r);
    int32_t c = 0, ch = 0;
    for (int32_t b0 = 0; b0 < n; b0 += kWave) {
        const int32_t b = b0 + lane;
        Pair p;
        bool isbad = false;
        const bool sel = b < n && selected<GATHER>(a, r * a.max_blocks + b, count, &p, &isbad);
        c += __popcll(ballot64(sel && p.row < a.tier.dev_rows));
        ch += __popcll(ballot64(sel && p.row >= a.tier.dev_rows));
        *bad += __popcll(ballot64(isbad));
    }
    *cnt = c;
    *cnt_h = ch;
}

__device__ inline int32_t ld_agent(const int32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline unsigned long long ld_agent(const unsigned long long* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

constexpr uint32_t kNoSlot = 0xFFFFFFFFu;  // an entry the row table had no slot for

// List entry i: a scatter's (home row, cache block) pair, also a grouping
// gather's (its row table comes next); a gather's slice of its own when it
// does not group.
template <bool GATHER>
__device__ inline void place(const SelectArgs& a, const Pair& p, int64_t i) {
    if (!GATHER || a.group) {
        a.sc.pairs[i] = p;
    } else {
        Slice q;
        q.row = p.row;
        q.base = (int32_t)i;
        q.n = 1;
        q.pad = 0;
        a.sc.slices[i] = q;
        a.sc.dests[i] = p.cb;
    }
}

// Request r's descriptors, written by the whole wave from list position pos
// (device rows) and pos_h (host-tier rows), in block order.
template <bool GATHER>
__device__ inline void fill_row(const SelectArgs& a, int64_t r, int lane, unsigned long long count,
                                int64_t pos, int64_t pos_h) {
    const int32_t n = row_len<GATHER>(a, r);
    for (int32_t b0 = 0; b0 < n; b0 += kWave) {
        const int32_t b = b0 + lane;
        Pair p;
        bool isbad = false;
        const bool sel = b < n && selected<GATHER>(a, r * a.max_blocks + b, count, &p, &isbad);
        const bool dev = sel && p.row < a.tier.dev_rows;
        const unsigned long long mask = ballot64(dev);
        const unsigned long long mask_h = ballot64(sel && !dev);
        if (dev) place<GATHER>(a, p, pos + __popcll(mask & lanes_below(lane)));
        if (sel && !dev) place<GATHER>(a, p, pos_h + __popcll(mask_h & lanes_below(lane)));
        pos += __popcll(mask);
        pos_h += __popcll(mask_h);
        // new bytes for a host-tier block: its device replica is stale, drop it
        if (!GATHER && sel && a.tier.rep_of && p.row >= a.tier.dev_rows) {
            const int64_t h = p.row - a.tier.dev_rows;
            const int32_t slot = atomicExch(&a.tier.rep_of[h], -1);
            if (slot >= 0) {
                a.tier.rep_id[slot] = -1;
                atomicSub(&a.state->rep_count, 1ull);
            }
        }
    }
}

template <bool GATHER>
__global__ __launch_bounds__(kSelThreads) void k_select_count(SelectArgs a) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r = (int64_t)blockIdx.x * kSelWaves + threadIdx.x / kWave;
    if (r >= a.R) return;
    int32_t cnt, cnt_h, bad = 0;
    count_row<GATHER>(a, r, lane, a.state->count, &cnt, &cnt_h, &bad);
    if (lane == 0) {
        a.sc.row_cnt[r] = cnt;
        a.sc.row_cnt_h[r] = cnt_h;
        if (bad) atomicAdd(&a.state->bad_entries, (unsigned long long)bad);
    }
}

// The slice and cache-block counters of a call: a gather that groups hands
// them out from zero; one that does not has one slice per list entry.
__device__ inline void set_counters(const SelectArgs& a, unsigned long long total,
                                    unsigned long long total_h) {
    *a.sc.total = total;
    *a.sc.total_h = total_h;
    *a.sc.nslices = a.group ? 0ull : total;
    *a.sc.nslices_h = a.group ? 0ull : total_h;
    *a.sc.ndests = 0;
    *a.sc.ndests_h = 0;
}

// One workgroup: exclusive scans of row_cnt and row_cnt_h into row_base and
// row_base_h, their totals into *total and *total_h. The requests go in
// tiles of 1024 x 4, each thread holding 4 neighbouring counts, so every
// load instruction reads whole lines and a tile costs one wave scan and two
// barriers. A call has at most 2^29 entries, so every sum fits in 32 bits.
constexpr int kScanPer = 4;

__global__ __launch_bounds__(1024) void k_select_scan(SelectArgs a) {
    __shared__ int32_t wsum[1024 / kWave], wsum_h[1024 / kWave];
    const int R = a.R;
    const int t = threadIdx.x, lane = t & (kWave - 1), wv = t / kWave;
    const int nw = blockDim.x / kWave;
    int32_t carry = 0, carry_h = 0;
    for (int base = 0; base < R; base += blockDim.x * kScanPer) {
        const int i0 = base + t * kScanPer;
        int32_t v[kScanPer], vh[kScanPer];
        int32_t s = 0, sh = 0;
#pragma unroll
        for (int k = 0; k < kScanPer; ++k) {
            v[k] = i0 + k < R ? a.sc.row_cnt[i0 + k] : 0;
            vh[k] = i0 + k < R ? a.sc.row_cnt_h[i0 + k] : 0;
            s += v[k];
            sh += vh[k];
        }
        int32_t x = s, xh = sh;  // inclusive scan over the wave
        for (int d = 1; d < kWave; d <<= 1) {
            const int32_t y = __shfl_up(x, d, kWave), yh = __shfl_up(xh, d, kWave);
            if (lane >= d) {
                x += y;
                xh += yh;
            }
        }
        if (lane == kWave - 1) {
            wsum[wv] = x;
            wsum_h[wv] = xh;
        }
        __syncthreads();
        int32_t run = carry + x - s, run_h = carry_h + xh - sh;
        for (int w = 0; w < nw; ++w) {
            const int32_t ws = wsum[w], wsh = wsum_h[w];
            if (w < wv) {
                run += ws;
                run_h += wsh;
            }
            carry += ws;
            carry_h += wsh;
        }
#pragma unroll
        for (int k = 0; k < kScanPer; ++k) {
            if (i0 + k < R) {
                a.sc.row_base[i0 + k] = run;
                a.sc.row_base_h[i0 + k] = run_h;
            }
            run += v[k];
            run_h += vh[k];
        }
        __syncthreads();  // wsum is written again by the next tile
    }
    if (t == 0) set_counters(a, (unsigned long long)carry, (unsigned long long)carry_h);
}

template <bool GATHER>
__global__ __launch_bounds__(kSelThreads) void k_select_fill(SelectArgs a) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r = (int64_t)blockIdx.x * kSelWaves + threadIdx.x / kWave;
    if (r >= a.R) return;
    // host rows after all device rows
    fill_row<GATHER>(a, r, lane, a.state->count, a.sc.row_base[r],
                     (int64_t)*a.sc.total + a.sc.row_base_h[r]);
}

// List entry i's cache block into its row's cache-block list; the row's
// rank-0 entry then empties the row's table slot, so the table is empty
// again when the call ends (this step reads only the slot's base, which
// stays).
__device__ inline void place_dest(const CopyScratch& sc, int64_t i) {
    const int32_t h = ld_agent(&sc.pslot[i]);
    if (h < 0) return;  // an entry the table had no slot for
    const int32_t rank = ld_agent(&sc.prank[i]);
    const int32_t cb = ld_agent(&sc.pairs[i].cb);
    sc.dests[ld_agent(&sc.tbase[h]) + rank] = cb;
    if (rank == 0) __hip_atomic_store(&sc.tkey[h], 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(kSelThreads) void k_group_dests(SelectArgs a) {
    const int64_t all = (int64_t)*a.sc.total + (int64_t)*a.sc.total_h;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < all;
         i += (int64_t)gridDim.x * blockDim.x)
        place_dest(a.sc, i);
}

// Small batches (at most kSmallMaxEntries (request, block) slots): the whole
// list in one workgroup, thread t holding slots s = k * 1024 + t. Every
// slot's loads are issued together (one trip to memory for the batch, where
// a walk over each request's windows costs a trip per window); list
// positions come from ballots and one exclusive scan of the per-wave counts
// in LDS. The list is the selected slots in slot order, device rows first,
// as the three-kernel path builds it. A gather of several requests groups
// its entries by row in an LDS table, each thread keeping its entries' table
// slots, ranks and cache blocks in registers.
constexpr int kSmallThreads = 1024;
constexpr int kSmallWaves = kSmallThreads / kWave;
constexpr int64_t kSmallMaxEntries = 8192;
constexpr int kSmallPer = (int)(kSmallMaxEntries / kSmallThreads);  // slots per thread
constexpr int kSmallCounts = kSmallPer * kSmallWaves;               // (k, wave) counts
constexpr uint32_t kSmallSlots = 2 * kSmallMaxEntries;               // LDS row table

// Enter an entry that reads `row` into the LDS row table (words (row + 1)
// << 32 | entries so far, 0 empty); returns slot | rank << 16, or kNoSlot if
// one pass over the table found no slot (it holds at least twice as many
// slots as entries, so one is always found).
__device__ inline uint32_t lds_enter(unsigned long long* tw, uint32_t slots, int32_t row) {
    const unsigned long long want = (unsigned long long)(uint32_t)(row + 1) << 32;
    uint32_t h = (uint32_t)(((uint64_t)(uint32_t)mix64((uint64_t)(uint32_t)row) * slots) >> 32);
    for (uint32_t probe = 0; probe < slots; ++probe) {
        const unsigned long long k = atomicCAS(&tw[h], 0ull, want | 1ull);
        if (k == 0) return h;
        if ((k & 0xFFFFFFFF00000000ull) == want)
            return h | (uint32_t)(atomicAdd(&tw[h], 1ull) & 0xFFFFFFFFull) << 16;
        h = h + 1 == slots ? 0 : h + 1;
    }
    return kNoSlot;
}

template <bool GATHER, bool GROUP>
__global__ __launch_bounds__(kSmallThreads) void k_select_small(SelectArgs a) {
    __shared__ int32_t wc[kSmallCounts], wch[kSmallCounts];  // per (k, wave); then their bases
    __shared__ int32_t total_dev, total_host;
    __shared__ unsigned long long alloc[2];  // per part: slices << 32 | cache blocks
    __shared__ unsigned long long tw[GROUP ? kSmallSlots : 1];  // only a grouping call holds it
    const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
    const int t = threadIdx.x;
    const unsigned long long count = a.state->count;
    constexpr bool group = GATHER && GROUP;
    const int32_t E = a.R * a.max_blocks;  // the host's condition: E <= kSmallMaxEntries
    uint32_t slots = 2u * (uint32_t)E;
    if (slots < 64) slots = 64;
    if (slots > kSmallSlots) slots = kSmallSlots;
    if (group) {
        for (uint32_t h = t; h < slots; h += blockDim.x) tw[h] = 0ull;
        if (t == 0) alloc[0] = alloc[1] = 0ull;
    }
    // every load first, from in-bounds (clamped) slots, with no branch between
    // them, so that they are all in flight together
    int32_t id[kSmallPer], cb[kSmallPer], mr[kSmallPer], made[kSmallPer];
    const int32_t last = E > 0 ? E - 1 : 0;
#pragma unroll
    for (int k = 0; k < kSmallPer; ++k) {
        const int32_t s = E > 0 ? min(k * kSmallThreads + t, last) : 0;
        id[k] = E > 0 ? a.ids[s] : -1;
        cb[k] = E > 0 ? a.block_table[s] : -1;
        mr[k] = GATHER && E > 0 ? a.m[s / a.max_blocks] : 0;
        made[k] = GATHER || (E > 0 && a.created[s] != 0);
    }
    Pair p[kSmallPer];
    unsigned long long dm[kSmallPer], hm[kSmallPer];  // the wave's selected slots: device, host rows
    int32_t bad = 0;
#pragma unroll
    for (int k = 0; k < kSmallPer; ++k) {
        const int32_t s = k * kSmallThreads + t;
        const int32_t r = s / (a.max_blocks > 0 ? a.max_blocks : 1), b = s - r * a.max_blocks;
        const int32_t n = GATHER ? (mr[k] < 0 ? 0 : (mr[k] < a.max_blocks ? mr[k] : a.max_blocks))
                                 : a.max_blocks;
        const bool use = (s < E) & (b < n);
        const bool skip = !made[k] | (cb[k] < 0);
        const bool out_of_range = ((int64_t)cb[k] >= a.cache_blocks) | (id[k] < 0) |
                                  ((unsigned long long)(int64_t)id[k] >= count);
        const bool sel = use & !skip & !out_of_range;
        p[k].row = 0;
        p[k].cb = cb[k];
        if (sel) p[k].row = GATHER ? gather_row(a.tier, id[k]) : home_row(a.tier, id[k]);
        const bool dev = sel && p[k].row < a.tier.dev_rows;
        dm[k] = ballot64(dev);
        hm[k] = ballot64(sel && !dev);
        bad += __popcll(ballot64(use & !skip & out_of_range));
        if (lane == 0) {
            wc[k * kSmallWaves + wv] = __popcll(dm[k]);
            wch[k * kSmallWaves + wv] = __popcll(hm[k]);
        }
    }
    if (lane == 0 && bad) atomicAdd(&a.state->bad_entries, (unsigned long long)bad);
    __syncthreads();
    // exclusive scans of the counts in (k, wave) order by the first wave, two
    // counts a lane (kSmallCounts = 128); totals of at most kSmallMaxEntries
    // fit in 32 bits
    if (wv == 0) {
        const int32_t c0 = wc[2 * lane], c1 = wc[2 * lane + 1];
        const int32_t h0 = wch[2 * lane], h1 = wch[2 * lane + 1];
        int32_t x = c0 + c1, xh = h0 + h1;
        for (int d = 1; d < kWave; d <<= 1) {
            const int32_t y = __shfl_up(x, d, kWave), yh = __shfl_up(xh, d, kWave);
            if (lane >= d) {
                x += y;
                xh += yh;
            }
        }
        const int32_t ex = x - c0 - c1, exh = xh - h0 - h1;
        wc[2 * lane] = ex;
        wc[2 * lane + 1] = ex + c0;
        wch[2 * lane] = exh;
        wch[2 * lane + 1] = exh + h0;
        if (lane == kWave - 1) {
            total_dev = x;
            total_host = xh;
            set_counters(a, (unsigned long long)x, (unsigned long long)xh);
        }
    }
    __syncthreads();
    const int32_t total = total_dev;  // host rows after all device rows
    uint32_t e[kSmallPer];
    int32_t pos[kSmallPer];
#pragma unroll
    for (int k = 0; k < kSmallPer; ++k) {
        e[k] = kNoSlot;
        pos[k] = -1;
        const bool dev = (dm[k] >> lane) & 1ull, host = (hm[k] >> lane) & 1ull;
        if (!dev && !host) continue;
        const int32_t i = dev ? wc[k * kSmallWaves + wv] + __popcll(dm[k] & lanes_below(lane))
                              : total + wch[k * kSmallWaves + wv] + __popcll(hm[k] & lanes_below(lane));
        pos[k] = i;
        const Pair& q = p[k];
        if (!GATHER) {
            a.sc.pairs[i] = q;
            // new bytes for a host-tier block: its device replica is stale, drop it
            if (host && a.tier.rep_of) {
                const int32_t slot = atomicExch(&a.tier.rep_of[q.row - a.tier.dev_rows], -1);
                if (slot >= 0) {
                    a.tier.rep_id[slot] = -1;
                    atomicSub(&a.state->rep_count, 1ull);
                }
            }
        } else if (group) {
            e[k] = lds_enter(tw, slots, q.row);
            if (e[k] == kNoSlot) atomicAdd(&a.state->bad_entries, 1ull);
        } else {
            Slice sl;
            sl.row = q.row;
            sl.base = i;
            sl.n = 1;
            sl.pad = 0;
            a.sc.slices[i] = sl;
            a.sc.dests[i] = q.cb;
        }
    }
    if (!group) return;  // uniform over the workgroup
    // every entry is in the table. Each row's rank-0 entry takes the slices
    // and cache blocks of all of the row's entries from its part's counters
    // (one 64-bit LDS atomic) and replaces the row's table word by where its
    // cache blocks start; then each entry's cache block goes to its row's list
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kSmallPer; ++k) {
        if (e[k] == kNoSlot || (e[k] >> 16) != 0) continue;
        const int part = pos[k] >= total ? 1 : 0;
        const int32_t off = part ? total : 0;
        const uint32_t h = e[k] & 0xFFFFu;
        const int32_t n = (int32_t)(tw[h] & 0xFFFFFFFFull);
        const int32_t nsl = (n + kSliceDests - 1) / kSliceDests;
        const unsigned long long got = atomicAdd(&alloc[part], (unsigned long long)nsl << 32 | (uint32_t)n);
        const int32_t sb = off + (int32_t)(got >> 32), db = off + (int32_t)(got & 0xFFFFFFFFull);
        tw[h] = (unsigned long long)(uint32_t)db;
        for (int j = 0; j < nsl; ++j) {
            const int32_t left = n - j * kSliceDests;
            Slice sl;
            sl.row = p[k].row;
            sl.base = db + j * kSliceDests;
            sl.n = left < kSliceDests ? left : kSliceDests;
            sl.pad = 0;
            a.sc.slices[sb + j] = sl;
        }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kSmallPer; ++k)
        if (e[k] != kNoSlot) a.sc.dests[(int32_t)tw[e[k] & 0xFFFFu] + (int32_t)(e[k] >> 16)] = p[k].cb;
    if (t == 0) {
        *a.sc.nslices = alloc[0] >> 32;
        *a.sc.nslices_h = alloc[1] >> 32;
        *a.sc.ndests = alloc[0] & 0xFFFFFFFFull;
        *a.sc.ndests_h = alloc[1] & 0xFFFFFFFFull;
    }
}

// A gather of several requests with more slots than one workgroup takes:
// the list's entries grouped by row in chunks of kGroupChunk entries, one
// workgroup each. The entries of one row in a chunk are first combined in
// an LDS table, so that the row takes one device-scope add per chunk, not
// one per entry: adds on one word are serialised across the device, and
// rows that thousands of requests share made them the longest step.
constexpr int kGroupThreads = 1024;
constexpr int kGroupPer = 2;                             // entries per thread
constexpr int kGroupChunk = kGroupThreads * kGroupPer;  // entries per workgroup
constexpr uint32_t kGroupSlots = 2 * kGroupChunk;       // LDS table of a chunk

// Reserve n ranks of `row` in the call's row table ((row + 1) << 32 |
// entries so far, 0 empty): its slot and the first of the n ranks. The
// table holds at least twice as many slots as entries and every call leaves
// it empty, so a slot is always found; the probe still stops after one pass.
__device__ inline bool table_add(const CopyScratch& sc, int32_t row, uint32_t n, int32_t* slot,
                                 int32_t* first) {
    const unsigned long long want = (unsigned long long)(uint32_t)(row + 1) << 32;
    uint64_t h = mix64((uint64_t)(uint32_t)row) & sc.table_mask;
    for (uint64_t probe = 0; probe <= sc.table_mask; ++probe, h = (h + 1) & sc.table_mask) {
        unsigned long long k = ld_agent(&sc.tkey[h]);
        if (k == 0) {
            k = atomicCAS(&sc.tkey[h], 0ull, want | n);
            if (k == 0) {
                *slot = (int32_t)h;
                *first = 0;
                return true;
            }
        }
        if ((k & 0xFFFFFFFF00000000ull) == want) {
            *slot = (int32_t)h;
            *first = (int32_t)(atomicAdd(&sc.tkey[h], (unsigned long long)n) & 0xFFFFFFFFull);
            return true;
        }
    }
    return false;
}

// Each list entry's row-table slot and rank (slot -1: none found, counted
// as bad). Ranks of one row are unique over the call: a chunk reserves a
// run of them and hands them out in LDS order.
__global__ __launch_bounds__(kGroupThreads) void k_group_enter(SelectArgs a) {
    __shared__ unsigned long long tw[kGroupSlots];  // (row + 1) << 32 | the chunk's entries
    __shared__ int32_t gslot[kGroupSlots], gfirst[kGroupSlots];
    const int64_t all = (int64_t)*a.sc.total + (int64_t)*a.sc.total_h;
    const int64_t c0 = (int64_t)blockIdx.x * kGroupChunk;
    if (c0 >= all) return;  // the whole workgroup
    const int t = threadIdx.x;
    for (uint32_t h = t; h < kGroupSlots; h += kGroupThreads) tw[h] = 0ull;
    __syncthreads();
    uint32_t e[kGroupPer];
#pragma unroll
    for (int k = 0; k < kGroupPer; ++k) {
        const int64_t i = c0 + t + k * kGroupThreads;
        e[k] = kNoSlot;
        if (i < all) {
            e[k] = lds_enter(tw, kGroupSlots, a.sc.pairs[i].row);
            if (e[k] == kNoSlot) atomicAdd(&a.state->bad_entries, 1ull);
        }
    }
    __syncthreads();
    for (uint32_t h = t; h < kGroupSlots; h += kGroupThreads) {
        const unsigned long long w = tw[h];
        if (w == 0) continue;
        int32_t slot = -1, first = 0;
        if (!table_add(a.sc, (int32_t)(w >> 32) - 1, (uint32_t)(w & 0xFFFFFFFFull), &slot, &first))
            atomicAdd(&a.state->bad_entries, w & 0xFFFFFFFFull);
        gslot[h] = slot;
        gfirst[h] = first;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kGroupPer; ++k) {
        const int64_t i = c0 + t + k * kGroupThreads;
        if (i >= all) continue;
        const int32_t slot = e[k] == kNoSlot ? -1 : gslot[e[k] & 0xFFFFu];
        a.sc.pslot[i] = slot;
        if (slot >= 0) a.sc.prank[i] = gfirst[e[k] & 0xFFFFu] + (int32_t)(e[k] >> 16);
    }
}

// Descriptors of the chunk's rows: each row's rank-0 entry takes slices for
// all of the row's entries (kSliceDests cache blocks each) and records where
// the row's cache blocks start; the chunk takes its slices and cache blocks
// from its part's counters with one device-scope add each.
__global__ __launch_bounds__(kGroupThreads) void k_group_slices(SelectArgs a) {
    __shared__ unsigned long long alloc[2], gs[2], gd[2];  // per part: slices << 32 | cache blocks
    const int64_t total = (int64_t)*a.sc.total;
    const int64_t all = total + (int64_t)*a.sc.total_h;
    const int64_t c0 = (int64_t)blockIdx.x * kGroupChunk;
    if (c0 >= all) return;  // the whole workgroup
    const int t = threadIdx.x;
    if (t < 2) alloc[t] = 0ull;
    __syncthreads();
    int32_t h[kGroupPer], n[kGroupPer], row[kGroupPer];
    unsigned long long got[kGroupPer];
#pragma unroll
    for (int k = 0; k < kGroupPer; ++k) {
        const int64_t i = c0 + t + k * kGroupThreads;
        n[k] = 0;
        if (i >= all) continue;
        h[k] = a.sc.pslot[i];
        if (h[k] < 0 || a.sc.prank[i] != 0) continue;
        const unsigned long long w = a.sc.tkey[h[k]];
        n[k] = (int32_t)(w & 0xFFFFFFFFull);
        row[k] = (int32_t)(w >> 32) - 1;
        const int32_t nsl = (n[k] + kSliceDests - 1) / kSliceDests;
        got[k] = atomicAdd(&alloc[i >= total ? 1 : 0], (unsigned long long)nsl << 32 | (uint32_t)n[k]);
    }
    __syncthreads();
    if (t < 2 && alloc[t]) {
        gs[t] = atomicAdd(t ? a.sc.nslices_h : a.sc.nslices, alloc[t] >> 32);
        gd[t] = atomicAdd(t ? a.sc.ndests_h : a.sc.ndests, alloc[t] & 0xFFFFFFFFull);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kGroupPer; ++k) {
        if (!n[k]) continue;
        const int64_t i = c0 + t + k * kGroupThreads;
        const int part = i >= total ? 1 : 0;
        const int64_t off = part ? total : 0;
        const int64_t sb = off + (int64_t)(gs[part] + (got[k] >> 32));
        const int64_t db = off + (int64_t)(gd[part] + (got[k] & 0xFFFFFFFFull));
        a.sc.tbase[h[k]] = (int32_t)db;
        const int32_t nsl = (n[k] + kSliceDests - 1) / kSliceDests;
        for (int j = 0; j < nsl; ++j) {
            const int32_t left = n[k] - j * kSliceDests;
            Slice q;
            q.row = row[k];
            q.base = (int32_t)(db + j * kSliceDests);
            q.n = left < kSliceDests ? left : kSliceDests;
            q.pad = 0;
            a.sc.slices[sb + j] = q;
        }
    }
}

struct CopyArgs {
    uint8_t* pool;
    uint8_t* host;      // host tier: rows dev_rows.. of the pool's row space
    int64_t dev_rows;
    uint8_t* cache;
    const Pair* pairs;       // scatter, row copies: the descriptors
    const Slice* slices;     // gather: the descriptors
    const int32_t* dests;    // gather: the slices' cache blocks
    const unsigned long long* first;  // the first descriptor (null: 0)
    const unsigned long long* total;  // descriptors from there
    int64_t block_bytes;
    int64_t chunk_bytes;
    int64_t cache_blocks;
    int32_t chunks_per_block;
    int32_t chunks_per_group;
    int32_t groups;            // ceil((c_hi - c_lo) / chunks_per_group)
    int32_t c_lo, c_hi;        // chunks moved: 2*l0 .. 2*l1-1
    const int64_t* lbase;      // per-layer slab bases (null when uniform)
};

// The (descriptor, chunk group) units are visited grid-stride. The host
// picks the grid: a gather launches one workgroup per possible unit, up to
// 512 times what the device holds at once, so the dense front of the list
// runs in hardware dispatch order (neighbouring workgroups copy neighbouring
// chunks; past the cap a workgroup also takes the unit one grid further on,
// and workgroups past the end exit at once); a scatter, whose created blocks
// are sparse, launches 16 times what the device holds, looping.
// Scatter, uniform slabs: a unit is (pair, group of chunks_per_group slabs).
__global__ __launch_bounds__(1024) void k_copy_pairs(CopyArgs a) {
    const unsigned long long units = *a.total * (unsigned long long)a.groups;
    const Pair* pairs = a.pairs + (a.first ? *a.first : 0ull);
    const int n16 = (int)(a.chunk_bytes >> 4);
    for (unsigned long long unit = blockIdx.x; unit < units; unit += gridDim.x) {
        const unsigned long long d = unit / (unsigned)a.groups;
        const int g = (int)(unit - d * (unsigned)a.groups);
        const Pair p = pairs[d];
        const int c0 = a.c_lo + g * a.chunks_per_group;
        const int c1 = min(c0 + a.chunks_per_group, a.c_hi);
        uint8_t* blk = p.row < a.dev_rows ? a.pool + (int64_t)p.row * a.block_bytes
                                          : a.host + (int64_t)(p.row - a.dev_rows) * a.block_bytes;
        for (int c = c0; c < c1; ++c) {
            uint8_t* row_chunk = blk + (int64_t)c * a.chunk_bytes;
            const uint8_t* cache_chunk = a.cache + ((int64_t)c * a.cache_blocks + p.cb) * a.chunk_bytes;
            copy_span(reinterpret_cast<const v4u*>(cache_chunk), reinterpret_cast<v4u*>(row_chunk), n16);
        }
    }
}

// A slice's cache blocks, one per lane (lane k holds the k-th; a slice has
// at most kSliceDests <= kWave of them), loaded once per unit. The copy
// loops take them with readlane: read from memory inside the store loop,
// each would be a vector load (the stores might alias the list, as far as
// the compiler knows) waiting for every store issued before it.
static_assert(kSliceDests <= kWave, "a slice's cache blocks must fit one per lane");
__device__ inline int32_t slice_dests(const CopyArgs& a, const Slice& q) {
    const int lane = threadIdx.x & (kWave - 1);
    // lanes past the last cache block read it again: no branch, so the load
    // is issued together with the row's first vectors
    return a.dests[q.base + min(lane, max(q.n - 1, 0))];
}

// Gather, uniform slabs: a unit is (slice, group of chunks). Each chunk of
// the slice's row is read once, two vectors per thread in flight, and
// written to each of the slice's cache blocks: a row that several requests
// need crosses the memory bus once per kSliceDests of them.
__global__ __launch_bounds__(1024) void k_copy_slices(CopyArgs a) {
    const unsigned long long units = *a.total * (unsigned long long)a.groups;
    const Slice* slices = a.slices + (a.first ? *a.first : 0ull);
    const int n16 = (int)(a.chunk_bytes >> 4);
    const int nt = blockDim.x;
    for (unsigned long long unit = blockIdx.x; unit < units; unit += gridDim.x) {
        const unsigned long long d = unit / (unsigned)a.groups;
        const int g = (int)(unit - d * (unsigned)a.groups);
        const Slice q = slices[d];
        const int32_t lane_cb = slice_dests(a, q);
        const int c0 = a.c_lo + g * a.chunks_per_group;
        const int c1 = min(c0 + a.chunks_per_group, a.c_hi);
        const uint8_t* blk = q.row < a.dev_rows ? a.pool + (int64_t)q.row * a.block_bytes
                                                : a.host + (int64_t)(q.row - a.dev_rows) * a.block_bytes;
        for (int c = c0; c < c1; ++c) {
            const v4u* src = reinterpret_cast<const v4u*>(blk + (int64_t)c * a.chunk_bytes);
            uint8_t* plane = a.cache + (int64_t)c * a.cache_blocks * a.chunk_bytes;
            // loops over uniform bounds, so that every lane is active at the
            // readlane (it reads a lane's register whatever the exec mask)
            for (int i0 = 0; i0 < n16; i0 += 2 * nt) {
                const int i = i0 + (int)threadIdx.x;
                const bool one = i < n16, two = i + nt < n16;
                // both loads unconditional (a thread past the chunk's end
                // re-reads its last vector): with no branch between them
                // they are issued together with the cache-block load
                const v4u x = ld_nt(src + min(i, n16 - 1));
                const v4u y = ld_nt(src + min(i + nt, n16 - 1));
                for (int k = 0; k < q.n; ++k) {
                    const int32_t cb = __builtin_amdgcn_readlane(lane_cb, k);
                    v4u* dst = reinterpret_cast<v4u*>(plane + (int64_t)cb * a.chunk_bytes);
                    if (one) st_nt(dst + i, x);
                    if (two) st_nt(dst + i + nt, y);
                }
            }
        }
    }
}

// Per-layer slab sizes. Layers l0 .. l1-1 of a pool row are one contiguous
// byte range [lbase[l0], lbase[l1]); a unit is (descriptor, kSpanBytes of
// that range), so every workgroup moves the same amount however small the
// slabs. Each 16-byte vector finds its slab (layer, K|V) from the layer
// bases, kept in LDS: a thread's offsets only grow, so it resumes the search
// from its previous layer. The per-workgroup set-up (the table load and a
// barrier) is paid once per 256 KiB: with 32 KiB units, one vector in
// flight, it cost a third of the bandwidth in some placements of pool and
// cache (4.1 against 6.3 TB/s on a 32-layer model with 32 and 8 KiB slabs).
constexpr int kSpanBytes = 256 << 10;

// Largest layer l in [li, n) with lb[l] <= o, given lb[li] <= o < lb[n].
__device__ inline int slab_from(const int64_t* lb, int li, int n, int64_t o) {
    if (lb[li + 1] > o) return li;
    int lo = li + 1, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (lb[mid] <= o) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// Cache address of the 16 bytes at range offset o of layer li for cache
// block cb (lb relative to the first layer of the call, l0); the pool row's
// bytes are at the same offset o of the row.
__device__ inline v4u* span_cache(const CopyArgs& a, const int64_t* lb, int li, int64_t o, int32_t cb) {
    const int64_t ch = (lb[li + 1] - lb[li]) >> 1;  // the layer's K (or V) slab
    const int64_t in = o - lb[li];
    const int kv = in >= ch ? 1 : 0;
    return reinterpret_cast<v4u*>(a.cache + a.cache_blocks * lb[li] +
                                  ((int64_t)kv * a.cache_blocks + cb) * ch + (in - kv * ch));
}

// A gather's unit is (slice, span): each vector of the row is read once
// and written to each of the slice's cache blocks; a scatter's is (pair,
// span).
template <bool GATHER>
__global__ __launch_bounds__(1024) void k_copy_spans(CopyArgs a) {
    __shared__ int64_t lb[kMaxVarLayers + 1];
    const unsigned long long spans = (unsigned)a.groups;  // kSpanBytes units per descriptor
    const unsigned long long units = *a.total * spans;
    const unsigned long long first = a.first ? *a.first : 0ull;
    if (blockIdx.x >= units) return;  // the whole workgroup: nothing to move
    const int l0 = a.c_lo >> 1, l1 = a.c_hi >> 1, nl = l1 - l0;
    for (int l = l0 + (int)threadIdx.x; l <= l1; l += blockDim.x) lb[l - l0] = a.lbase[l];
    __syncthreads();
    const int64_t b0 = lb[0], b1 = lb[nl];
    const int64_t step = 16 * (int64_t)blockDim.x;
    for (unsigned long long unit = blockIdx.x; unit < units; unit += gridDim.x) {
        const unsigned long long d = unit / spans;
        const int64_t s0 = b0 + (int64_t)(unit - d * spans) * kSpanBytes;
        const int64_t s1 = min(s0 + (int64_t)kSpanBytes, b1);
        int32_t row, n = 1, cb0 = 0, lane_cb = 0;
        if (GATHER) {
            const Slice q = a.slices[first + d];
            row = q.row;
            n = q.n;
            lane_cb = slice_dests(a, q);
        } else {
            const Pair p = a.pairs[first + d];
            row = p.row;
            cb0 = p.cb;
        }
        uint8_t* blk = row < a.dev_rows ? a.pool + (int64_t)row * a.block_bytes
                                        : a.host + (int64_t)(row - a.dev_rows) * a.block_bytes;
        // two vectors per thread in flight: both loaded before either is
        // stored. The loop runs over uniform bounds, so that every lane is
        // active at the readlane (it reads a lane's register whatever the
        // exec mask).
        int li = 0;
        for (int64_t o0 = s0; o0 < s1; o0 += 2 * step) {
            const int64_t o = o0 + 16 * (int64_t)threadIdx.x;
            const bool one = o < s1, two = o + step < s1;
            if (one) li = slab_from(lb, li, nl, o);
            const int li1 = two ? slab_from(lb, li, nl, o + step) : li;
            v4u* pv0 = reinterpret_cast<v4u*>(blk + o);
            v4u* pv1 = reinterpret_cast<v4u*>(blk + o + step);
            if (GATHER) {
                // unconditional loads (past the span's end a thread re-reads
                // its last vector), issued together
                const v4u x0 = ld_nt(reinterpret_cast<const v4u*>(blk + min(o, s1 - 16)));
                const v4u x1 = ld_nt(reinterpret_cast<const v4u*>(blk + min(o + step, s1 - 16)));
                for (int k = 0; k < n; ++k) {
                    const int32_t cb = __builtin_amdgcn_readlane(lane_cb, k);
                    if (one) st_nt(span_cache(a, lb, li, o, cb), x0);
                    if (two) st_nt(span_cache(a, lb, li1, o + step, cb), x1);
                }
            } else if (one) {
                const v4u x0 = ld_nt(span_cache(a, lb, li, o, cb0));
                v4u x1;
                if (two) x1 = ld_nt(span_cache(a, lb, li1, o + step, cb0));
                st_nt(pv0, x0);
                if (two) st_nt(pv1, x1);
            }
            li = li1;
        }
    }
}

// Whole blocks from one row to another (replication): pairs[k].row is the
// source row, pairs[k].cb the destination row; *total pairs. A block is
// moved in pieces of kRowPiece bytes whatever its layers.
constexpr int64_t kRowPiece = 32 << 10;

__global__ __launch_bounds__(1024) void k_copy_rows(CopyArgs a) {
    const int64_t pieces = (a.block_bytes + kRowPiece - 1) / kRowPiece;
    const unsigned long long units = *a.total * (unsigned long long)pieces;
    for (unsigned long long unit = blockIdx.x; unit < units; unit += gridDim.x) {
        const unsigned long long d = unit / (unsigned long long)pieces;
        const int64_t off = (int64_t)(unit - d * (unsigned long long)pieces) * kRowPiece;
        const int n16 = (int)(min(kRowPiece, a.block_bytes - off) >> 4);
        const Pair p = a.pairs[d];
        const int64_t rows[2] = {p.row, p.cb};
        uint8_t* blk[2];
        for (int k = 0; k < 2; ++k)
            blk[k] = rows[k] < a.dev_rows ? a.pool + rows[k] * a.block_bytes
                                          : a.host + (rows[k] - a.dev_rows) * a.block_bytes;
        copy_span(reinterpret_cast<const v4u*>(blk[0] + off), reinterpret_cast<v4u*>(blk[1] + off), n16);
    }
}

template <bool GATHER>
hipError_t select(const CopyPlan& p, const CopyScratch& sc, const int32_t* ids, const int32_t* m,
                  const uint8_t* created, const int32_t* bt, int32_t R, int32_t max_blocks,
                  int64_t cache_blocks, hipStream_t s) {
    // a gather of one request lists each row once (its ids are a path), so
    // only a gather of several requests groups its entries by row
    SelectArgs a{ids, m, created, bt, R, max_blocks, cache_blocks, p.state, sc, p.tier,
                 GATHER && R >= 2 ? 1 : 0};
    if ((int64_t)R * max_blocks <= kSmallMaxEntries) {
        if (a.group)
            hipLaunchKernelGGL((k_select_small<GATHER, true>), dim3(1), dim3(kSmallThreads), 0, s, a);
        else
            hipLaunchKernelGGL((k_select_small<GATHER, false>), dim3(1), dim3(kSmallThreads), 0, s, a);
        return hipGetLastError();
    }
    const unsigned grid = (unsigned)((R + kSelWaves - 1) / kSelWaves);
    hipLaunchKernelGGL(k_select_count<GATHER>, dim3(grid), dim3(kSelThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_select_scan, dim3(1), dim3(1024), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_select_fill<GATHER>, dim3(grid), dim3(kSelThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess || !a.group) return e;
    const int64_t entries = (int64_t)R * max_blocks;
    const unsigned chunks = (unsigned)((entries + kGroupChunk - 1) / kGroupChunk);
    hipLaunchKernelGGL(k_group_enter, dim3(chunks), dim3(kGroupThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_group_slices, dim3(chunks), dim3(kGroupThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    int64_t dgrid = (entries + kSelThreads - 1) / kSelThreads;
    if (dgrid > 4096) dgrid = 4096;
    hipLaunchKernelGGL(k_group_dests, dim3((unsigned)dgrid), dim3(kSelThreads), 0, s, a);
    return hipGetLastError();
}

template <bool GATHER>
hipError_t copy(const CopyPlan& p, const CopyScratch& sc, uint8_t* cache, int64_t cache_blocks,
                int32_t R, int32_t max_blocks, int32_t l0, int32_t l1, hipStream_t s) {
    CopyArgs a{};
    a.pool = p.pool;
    a.host = p.tier.host;
    a.dev_rows = p.tier.dev_rows;
    a.cache = cache;
    a.pairs = sc.pairs;
    a.slices = sc.slices;
    a.dests = sc.dests;
    a.total = GATHER ? sc.nslices : sc.total;  // a gather has at most one slice per entry
    a.block_bytes = p.block_bytes;
    a.chunk_bytes = p.chunk_bytes;
    a.cache_blocks = cache_blocks;
    a.chunks_per_block = p.chunks_per_block;
    a.chunks_per_group = p.chunks_per_group;
    a.c_lo = 2 * l0;
    a.c_hi = 2 * l1;
    a.lbase = p.lbase;
    if (p.lbase) {  // units are kSpanBytes spans of the layer range
        const int64_t lo = p.lbase_host[l0], hi = p.lbase_host[l1];
        a.groups = (int32_t)((hi - lo + kSpanBytes - 1) / kSpanBytes);
    } else {
        a.groups = (a.c_hi - a.c_lo + p.chunks_per_group - 1) / p.chunks_per_group;
    }
    const int64_t bound = (int64_t)R * max_blocks * a.groups;  // units if every entry moves
    const int64_t cap = (1ll << 31) / p.threads;                 // launch limit on work-items
    int64_t grid = p.grid ? p.grid : (GATHER ? (int64_t)p.gather_grid : (int64_t)p.loop_grid);
    if (grid > bound) grid = bound;
    if (grid > cap) grid = cap;
    if (grid < 1) return hipSuccess;
    if (p.lbase)
        hipLaunchKernelGGL(k_copy_spans<GATHER>, dim3((unsigned)grid), dim3(p.threads), 0, s, a);
    else if (GATHER)
        hipLaunchKernelGGL(k_copy_slices, dim3((unsigned)grid), dim3(p.threads), 0, s, a);
    else
        hipLaunchKernelGGL(k_copy_pairs, dim3((unsigned)grid), dim3(p.threads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.tier.host_blocks == 0) return e;
    // host-tier rows: bound by the host link, so a small looping grid moves
    // them and the device's other compute units stay free for device rows
    // (of this call or of calls on other streams)
    CopyArgs h = a;
    h.first = sc.total;
    h.total = GATHER ? sc.nslices_h : sc.total_h;
    int64_t hg = p.host_grid;
    if (hg > bound) hg = bound;
    if (hg > cap) hg = cap;
    if (p.lbase)
        hipLaunchKernelGGL(k_copy_spans<GATHER>, dim3((unsigned)hg), dim3(p.threads), 0, s, h);
    else if (GATHER)
        hipLaunchKernelGGL(k_copy_slices, dim3((unsigned)hg), dim3(p.threads), 0, s, h);
    else
        hipLaunchKernelGGL(k_copy_pairs, dim3((unsigned)hg), dim3(p.threads), 0, s, h);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_copy_rows(const CopyPlan& p, const Pair* pairs, const unsigned long long* total,
                            int64_t max_pairs, hipStream_t s) {
    CopyArgs a{};
    a.pool = p.pool;
    a.host = p.tier.host;
    a.dev_rows = p.tier.dev_rows;
    a.pairs = pairs;
    a.total = total;
    a.block_bytes = p.block_bytes;
    a.chunk_bytes = p.chunk_bytes;
    a.chunks_per_block = p.chunks_per_block;
    int64_t grid = (int64_t)p.loop_grid;
    const int64_t bound = max_pairs * ((p.block_bytes + kRowPiece - 1) / kRowPiece);
    if (grid > bound) grid = bound;
    if (grid < 1) return hipSuccess;
    hipLaunchKernelGGL(k_copy_rows, dim3((unsigned)grid), dim3(p.threads), 0, s, a);
    return hipGetLastError();
}

uint64_t copy_table_slots(int32_t R, int32_t max_blocks) {
    const uint64_t need = 2ull * (uint64_t)R * (uint64_t)max_blocks;
    uint64_t h = 64;
    while (h < need) h <<= 1;
    return h;
}

namespace {
size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }
}  // namespace

size_t copy_scratch_bytes(int32_t R, int32_t max_blocks, uint64_t table_cap) {
    const size_t E = (size_t)R * max_blocks, Rs = (size_t)R;
    return up256(table_cap * 8) + up256(table_cap * 4) + up256(E * sizeof(Pair)) +
           up256(E * sizeof(Slice)) + 3 * up256(E * 4) + 2 * up256(Rs * 4) + 2 * up256(Rs * 8) + 256;
}

void copy_scratch_carve(void* base, int32_t R, int32_t max_blocks, uint64_t table_cap,
                        CopyScratch* out) {
    const size_t E = (size_t)R * max_blocks, Rs = (size_t)R;
    uint8_t* q = static_cast<uint8_t*>(base);
    auto take = [&](size_t bytes) {
        uint8_t* r = q;
        q += up256(bytes);
        return r;
    };
    out->tkey = reinterpret_cast<unsigned long long*>(take(table_cap * 8));
    out->tbase = reinterpret_cast<int32_t*>(take(table_cap * 4));
    out->table_mask = copy_table_slots(R, max_blocks) - 1;
    out->pairs = reinterpret_cast<Pair*>(take(E * sizeof(Pair)));
    out->slices = reinterpret_cast<Slice*>(take(E * sizeof(Slice)));
    out->dests = reinterpret_cast<int32_t*>(take(E * 4));
    out->pslot = reinterpret_cast<int32_t*>(take(E * 4));
    out->prank = reinterpret_cast<int32_t*>(take(E * 4));
    out->row_cnt = reinterpret_cast<int32_t*>(take(Rs * 4));
    out->row_cnt_h = reinterpret_cast<int32_t*>(take(Rs * 4));
    out->row_base = reinterpret_cast<int64_t*>(take(Rs * 8));
    out->row_base_h = reinterpret_cast<int64_t*>(take(Rs * 8));
    out->total = reinterpret_cast<unsigned long long*>(q);
    out->total_h = out->total + 1;
    out->nslices = out->total + 2;
    out->nslices_h = out->total + 3;
    out->ndests = out->total + 4;
    out->ndests_h = out->total + 5;
}

namespace {
__global__ void k_zero(uint32_t* p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0u;
}
}  // namespace

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s) {
    const size_t n = bytes / 4;
    if (n == 0) return hipSuccess;
    size_t g = (n + 255) / 256;
    if (g > 65536) g = 65536;
    hipLaunchKernelGGL(k_zero, dim3((unsigned)g), dim3(256), 0, s, static_cast<uint32_t*>(p), n);
    return hipGetLastError();
}

hipError_t launch_gather_select(const CopyPlan& p, const CopyScratch& sc, const int32_t* ids,
                                const int32_t* m, const int32_t* block_table, int32_t R,
                                int32_t max_blocks, int64_t cache_blocks, hipStream_t s) {
    return select<true>(p, sc, ids, m, nullptr, block_table, R, max_blocks, cache_blocks, s);
}

hipError_t launch_scatter_select(const CopyPlan& p, const CopyScratch& sc, const int32_t* ids,
                                 const uint8_t* created, const int32_t* block_table, int32_t R,
                                 int32_t max_blocks, int64_t cache_blocks, hipStream_t s) {
    return select<false>(p, sc, ids, nullptr, created, block_table, R, max_blocks, cache_blocks, s);
}

hipError_t launch_gather_copy(const CopyPlan& p, const CopyScratch& sc, uint8_t* cache,
                              int64_t cache_blocks, int32_t R, int32_t max_blocks, int32_t l0,
                              int32_t l1, hipStream_t s) {
    return copy<true>(p, sc, cache, cache_blocks, R, max_blocks, l0, l1, s);
}

hipError_t launch_scatter_copy(const CopyPlan& p, const CopyScratch& sc, const uint8_t* cache,
                               int64_t cache_blocks, int32_t R, int32_t max_blocks, int32_t l0,
                               int32_t l1, hipStream_t s) {
    return copy<false>(p, sc, const_cast<uint8_t*>(cache), cache_blocks, R, max_blocks, l0, l1, s);
}

}  // namespace ptsd
