// Frequency-based leaf eviction (PTStore Section 4.1, "Access
// pattern-aware eviction policy": frequency over recency, GDSF adapted to
// shared prefixes).
//
// Every access of a block adds 1 to its frequency F and sets its priority
// H = L + F, L being the store's clock. An insert that needs more new blocks
// than the never-used ids left evicts the difference, each time taking a
// block with no resident child that the batch did not match, the one with
// the lowest H, then the deepest, then the smallest id, and raising L to its
// H. Taken one at a time that is a sequential walk; it has a parallel form:
//
//   a child is never accessed without its parent and the clock only grows,
//   so H(child) <= H(parent), and with depth as the second key the child
//   ranks strictly before its parent in the order (H, deeper first, id).
//   The blocks the batch did not match include every descendant of each of
//   them. Hence the lowest-ranked of them always has no resident child, and
//   the one-at-a-time walk takes exactly the first `want` of them in that
//   order.
//
// So the victims are the `want` smallest keys (H, depth descending, id)
// among the unmatched blocks, found by a radix select. A range pass first
// takes the minimum and maximum of each field over the candidates; the key
// then keeps only the bits in which candidates can differ,
//   (H - Hmin) | (depth_max - depth) | (id - id_min),
// left-aligned in 128 bits (typically some 40 bits wide). Each digit pass
// is a 2048-bin histogram of the next 11 bits among the keys that agree with
// the threshold found so far; the last workgroup of a pass to finish picks
// the digit. Then the victims are marked in a bit mask, their index slots
// become tombstones, their parents lose a child, L takes their largest H,
// and a scan lists them by ascending id, the order in which their ids are
// reused. When deleted slots have piled up, the index is rebuilt from the
// surviving blocks.
#include "kernels.hpp"

namespace ptsd {
namespace {

constexpr int kThreads = 256;

typedef unsigned __int128 u128;

__device__ inline unsigned bit_width(uint64_t x) { return x ? 64u - (unsigned)__clzll((long long)x) : 0u; }

// Is `id` ranked by the running search? (sel_lo_id <= id < sel_hi_id holds.)
__device__ inline bool sel_candidate(const EvictView& ev, const DevState* st, int64_t id) {
    return st->sel_hot || ev.prot[id] != (int32_t)st->ev_epoch;
}

// The candidate's compressed key, left-aligned in 128 bits (state written by
// the range pass). Eviction: (H - Hmin, depth_max - depth, id - id_min), the
// smallest go. Hot set: (Hmax - H, id - id_min), the smallest stay.
__device__ inline u128 sel_key(const EvictView& ev, const DevState* st, int64_t id) {
    const bool hot = st->sel_hot != 0;
    const u128 p = (u128)(hot ? st->sel_pbase - ev.prio[id] : ev.prio[id] - st->sel_pbase);
    const u128 d = hot ? (u128)0 : (u128)(st->sel_dmax - (uint64_t)ev.depth[id]);
    const u128 i = (u128)((uint64_t)id - st->sel_imin);
    const unsigned wd = st->sel_wd, wi = st->sel_wi, w = st->sel_w;
    const u128 c = (p << (wd + wi)) | (d << wi) | i;
    return w == 0 ? (u128)0 : c << (128u - w);
}

__device__ inline unsigned long long lanes_below(int lane) {
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

template <typename T, typename Op>
__device__ inline T wave_reduce(T v, Op op, int lane) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) v = op(v, (T)shfl_u64((uint64_t)v, lane ^ d));
    return v;
}

// Ranges of H, depth and id over the candidates, their number, and from them
// the key layout. Also clears the digit histograms. Each workgroup writes its
// own partial (no shared-address atomics); the last one to finish combines
// them. Serves both searches (eviction and hot set, see sel_key).
__global__ __launch_bounds__(kThreads) void k_sel_range(EvictView ev, DevState* st) {
    if (st->ev_want == 0) return;  // uniform over the grid
    const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < (int64_t)kSelPasses * kSelBins;
         i += (int64_t)gridDim.x * kThreads)
        ev.hist[i] = 0;
    const int64_t lo_id = (int64_t)st->sel_lo_id, hi_id = (int64_t)st->sel_hi_id;
    // [0] min H, [1] -max H, [2] min depth, [3] -max depth, [4] min id, [5] -max id: all minima
    uint64_t v[6] = {~0ull, ~0ull, ~0ull, ~0ull, ~0ull, ~0ull};
    uint64_t n = 0;
    for (int64_t id = lo_id + (int64_t)blockIdx.x * kThreads + threadIdx.x; id < hi_id;
         id += (int64_t)gridDim.x * kThreads) {
        if (!sel_candidate(ev, st, id)) continue;
        const uint64_t x[6] = {ev.prio[id], ~ev.prio[id], (uint64_t)ev.depth[id], ~(uint64_t)ev.depth[id],
                               (uint64_t)id, ~(uint64_t)id};
#pragma unroll
        for (int k = 0; k < 6; ++k) v[k] = x[k] < v[k] ? x[k] : v[k];
        ++n;
    }
    auto mn = [](uint64_t a, uint64_t b) { return a < b ? a : b; };
    auto sum = [](uint64_t a, uint64_t b) { return a + b; };
    __shared__ uint64_t red[kThreads / kWave][8];
#pragma unroll
    for (int k = 0; k < 6; ++k) v[k] = wave_reduce(v[k], mn, lane);
    n = wave_reduce(n, sum, lane);
    if (lane == 0) {
        for (int k = 0; k < 6; ++k) red[wv][k] = v[k];
        red[wv][6] = n;
    }
    __syncthreads();
    if (threadIdx.x < 7) {
        const int k = threadIdx.x;
        uint64_t a = red[0][k];
        for (int w = 1; w < kThreads / kWave; ++w) a = k < 6 ? mn(a, red[w][k]) : a + red[w][k];
        ev.part[(int64_t)blockIdx.x * 8 + k] = a;
    }
    __shared__ int last;
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) last = atomicAdd(&st->sel_range_done, 1u) == gridDim.x - 1;
    __syncthreads();
    if (!last) return;
    __threadfence();
    // last workgroup: combine the partials (one wave per field)
    __shared__ uint64_t tot[8];
    for (int k = wv; k < 7; k += kThreads / kWave) {
        uint64_t a = k < 6 ? ~0ull : 0ull;
        for (int64_t g = lane; g < gridDim.x; g += kWave) {
            const uint64_t x = __hip_atomic_load(&ev.part[g * 8 + k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            a = k < 6 ? mn(a, x) : a + x;
        }
        a = k < 6 ? wave_reduce(a, mn, lane) : wave_reduce(a, sum, lane);
        if (lane == 0) tot[k] = a;
    }
    __syncthreads();
    if (threadIdx.x != 0) return;
    if (tot[6] <= st->ev_want) {  // every candidate goes
        st->ev_all = 1;
        return;
    }
    const uint64_t pmin = tot[0], pmax = ~tot[1], dmin = tot[2], dmax = ~tot[3], imin = tot[4],
                   imax = ~tot[5];
    const bool hot = st->sel_hot != 0;
    const unsigned wp = bit_width(pmax - pmin), wd = hot ? 0u : bit_width(dmax - dmin),
                   wi = bit_width(imax - imin);
    st->sel_pbase = hot ? pmax : pmin;
    st->sel_dmax = dmax;
    st->sel_imin = imin;
    st->sel_wd = wd;
    st->sel_wi = wi;
    st->sel_w = wp + wd + wi;  // <= 64 + 31 + 31
    st->sel_npass = (wp + wd + wi + kSelBits - 1) / kSelBits;
}

// One digit pass of the threshold search.
__global__ __launch_bounds__(kThreads) void k_sel_pass(EvictView ev, DevState* st, int pass) {
    if (st->ev_want == 0 || st->ev_all || (unsigned)pass >= st->sel_npass) return;  // uniform
    __shared__ unsigned int h[kSelBins];
    __shared__ unsigned int part[kThreads];
    __shared__ int last;
    const int t = threadIdx.x;
    for (int b = t; b < kSelBins; b += kThreads) h[b] = 0;
    __syncthreads();
    const int64_t lo_id = (int64_t)st->sel_lo_id, hi_id = (int64_t)st->sel_hi_id;
    const u128 thr = ((u128)st->sel_hi << 64) | (u128)st->sel_lo;
    const int hi_bit = 128 - kSelBits * pass;          // digit = key bits [lo_bit, hi_bit)
    const int lo_bit = hi_bit - kSelBits > 0 ? hi_bit - kSelBits : 0;
    const unsigned dmask = (1u << (hi_bit - lo_bit)) - 1u;
    for (int64_t id = lo_id + (int64_t)blockIdx.x * kThreads + t; id < hi_id;
         id += (int64_t)gridDim.x * kThreads) {
        if (!sel_candidate(ev, st, id)) continue;
        const u128 k = sel_key(ev, st, id);
        if (pass > 0 && (k >> hi_bit) != (thr >> hi_bit)) continue;
        atomicAdd(&h[(unsigned)(k >> lo_bit) & dmask], 1u);
    }
    __syncthreads();
    uint32_t* gh = ev.hist + pass * kSelBins;
    for (int b = t; b < kSelBins; b += kThreads)
        if (h[b]) atomicAdd(&gh[b], h[b]);
    __threadfence();
    __syncthreads();
    if (t == 0) last = atomicAdd(&st->sel_done[pass], 1u) == gridDim.x - 1;
    __syncthreads();
    if (!last) return;
    __threadfence();
    // last workgroup: the digit whose bin holds the need-th smallest key
    constexpr int kPer = kSelBins / kThreads;
    unsigned own = 0;
    for (int j = 0; j < kPer; ++j) {
        h[t * kPer + j] = __hip_atomic_load(&gh[t * kPer + j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        own += h[t * kPer + j];
    }
    part[t] = own;
    __syncthreads();
    for (int d = 1; d < kThreads; d <<= 1) {  // inclusive scan of the per-thread sums
        const unsigned v = t >= d ? part[t - d] : 0u;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    const uint64_t need = st->sel_need;
    const uint64_t before = part[t] - own;
    if (before < need && need <= part[t]) {  // exactly one thread
        uint64_t cum = before;
        int j = 0;
        for (; j < kPer - 1; ++j) {
            if (cum + h[t * kPer + j] >= need) break;
            cum += h[t * kPer + j];
        }
        const unsigned digit = (unsigned)(t * kPer + j);
        const u128 nt = thr | ((u128)digit << lo_bit);
        st->sel_need = need - cum;
        st->sel_hi = (uint64_t)(nt >> 64);
        st->sel_lo = (uint64_t)nt;
    }
}

// Marks the victims (one bit per id), deletes their index entries, takes a
// child from their parents and raises the clock to their largest priority.
__global__ __launch_bounds__(kThreads) void k_ev_mark(EvictView ev, DevState* st, Slot* slots,
                                                      const int32_t* parent) {
    if (st->ev_want == 0) return;
    const int lane = threadIdx.x & (kWave - 1);
    const bool all = st->ev_all != 0;
    const u128 thr = ((u128)st->sel_hi << 64) | (u128)st->sel_lo;
    const int64_t old = (int64_t)st->insert_old_count;
    const int64_t span = ev.words * kWave;
    const int32_t epoch = (int32_t)st->ev_epoch;
    uint64_t maxp = 0;
    for (int64_t base = (int64_t)blockIdx.x * kThreads; base < span; base += (int64_t)gridDim.x * kThreads) {
        const int64_t id = base + threadIdx.x;
        bool sel = false;
        if (id < old && ev.prot[id] != epoch) {
            sel = all || sel_key(ev, st, id) <= thr;
            if (sel) {
                const uint64_t hp = ev.prio[id];
                maxp = hp > maxp ? hp : maxp;
                slots[ev.spos[id]].key = kTombKey;
                const int32_t p = parent[id];
                if (p >= 0) atomicSub(&ev.live[p], 1);
                if (ev.tier.rep_of && id >= ev.tier.owned) {  // its replica goes too
                    const int64_t h = id - ev.tier.owned;
                    const int32_t slot = ev.tier.rep_of[h];
                    if (slot >= 0) {
                        ev.tier.rep_of[h] = -1;
                        ev.tier.rep_id[slot] = -1;
                        atomicSub(&st->rep_count, 1ull);
                    }
                }
            }
        }
        const unsigned long long mask = ballot64(sel);
        if (lane == 0 && id / kWave < ev.words) {
            ev.wmask[id / kWave] = mask;
            ev.wcnt[id / kWave] = (uint32_t)__popcll(mask);
        }
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const uint64_t o = shfl_u64(maxp, lane ^ d);
        maxp = o > maxp ? o : maxp;
    }
    if (lane == 0 && maxp) atomicMax(&st->clock, (unsigned long long)maxp);
}

// One workgroup: exclusive scan of the per-word victim counts; updates the
// eviction counters and decides whether the index is rebuilt.
__global__ __launch_bounds__(1024) void k_ev_scan(EvictView ev, DevState* st, int64_t capacity,
                                                  uint64_t slots_n) {
    if (st->ev_want == 0) {
        if (threadIdx.x == 0) st->ev_rebuild = 0;
        return;
    }
    __shared__ long long part[1024];
    const int64_t W = ev.words;
    const int t = threadIdx.x, nt = blockDim.x;
    const int64_t per = (W + nt - 1) / nt;
    const int64_t lo = min(W, (int64_t)t * per), hi = min(W, lo + per);
    long long s = 0;
    for (int64_t i = lo; i < hi; ++i) s += ev.wcnt[i];
    part[t] = s;
    __syncthreads();
    for (int d = 1; d < nt; d <<= 1) {
        long long v = t >= d ? part[t - d] : 0;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    long long run = part[t] - s;
    for (int64_t i = lo; i < hi; ++i) {
        ev.wbase[i] = (uint32_t)run;
        run += ev.wcnt[i];
    }
    if (t == nt - 1) {
        const unsigned long long nv = (unsigned long long)part[nt - 1];
        const unsigned long long fresh = (unsigned long long)capacity - st->insert_old_count;
        st->ev_nv = nv;
        st->evictions += nv;
        if (st->ev_new > fresh + nv) {
            st->full_events += 1;
            st->insert_full = 1;
        }
        const unsigned long long tomb = st->tombstones + nv;
        if (tomb * 4 > slots_n) {
            st->ev_rebuild = 1;
            st->rebuilds += 1;
            st->tombstones = 0;
        } else {
            st->ev_rebuild = 0;
            st->tombstones = tomb;
        }
    }
}

// Lists the victims by ascending id.
__global__ __launch_bounds__(kThreads) void k_ev_list(EvictView ev, DevState* st) {
    if (st->ev_want == 0) return;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t span = ev.words * kWave;
    for (int64_t id = (int64_t)blockIdx.x * kThreads + threadIdx.x; id < span;
         id += (int64_t)gridDim.x * kThreads) {
        const int64_t w = id / kWave;
        const uint64_t mask = ev.wmask[w];
        if ((mask >> lane) & 1ull) ev.victims[ev.wbase[w] + __popcll(mask & lanes_below(lane))] = (int32_t)id;
    }
}

__global__ __launch_bounds__(kThreads) void k_rebuild_clear(DevState* st, Slot* slots, uint64_t n) {
    if (!st->ev_rebuild) return;
    for (uint64_t i = (uint64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (uint64_t)gridDim.x * kThreads) {
        Slot z;
        z.key = kEmptyKey;
        z.id = -1;
        z.parent = -1;
        slots[i] = z;
    }
}

// Re-enters every surviving block into the cleared index.
__global__ __launch_bounds__(kThreads) void k_rebuild_insert(EvictView ev, DevState* st, Slot* slots,
                                                             uint64_t slot_mask, const int32_t* parent,
                                                             const HashTables* ht) {
    if (!st->ev_rebuild) return;
    const int64_t old = (int64_t)st->insert_old_count;
    for (int64_t id = (int64_t)blockIdx.x * kThreads + threadIdx.x; id < old;
         id += (int64_t)gridDim.x * kThreads) {
        if ((ev.wmask[id / kWave] >> (id & (kWave - 1))) & 1ull) continue;  // evicted
        const uint64_t ik = ev.nkey[id];
        uint64_t pos = slot_of(ik, ht->slot_seed, slot_mask);
        // at most half the slots hold blocks, so an empty one is always found
        for (uint64_t step = 0; step <= slot_mask; ++step) {
            const unsigned long long prev =
                atomicCAS(reinterpret_cast<unsigned long long*>(&slots[pos].key), kEmptyKey,
                          (unsigned long long)ik);
            if (prev == kEmptyKey) {
                slots[pos].id = (int32_t)id;
                slots[pos].parent = parent[id];
                ev.spos[id] = (uint32_t)pos;
                break;
            }
            pos = (pos + 1) & slot_mask;
        }
    }
}

// Accesses of the resident paths of an insert's requests (after its
// evictions, with the clock they left).
__global__ __launch_bounds__(kThreads) void k_touch(EvictView ev, DevState* st, const int32_t* m,
                                                    const int32_t* ids, int32_t R, int32_t max_blocks) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r = (int64_t)blockIdx.x * (kThreads / kWave) + threadIdx.x / kWave;
    if (r >= R) return;
    const uint64_t L = st->clock;
    const int32_t n = m[r];
    const int32_t* row = ids + r * max_blocks;
    for (int32_t b = lane; b < n; b += kWave) {
        const int32_t id = row[b];
        const uint64_t f = atomicAdd((unsigned long long*)&ev.freq[id], 1ull) + 1ull;
        atomicMax((unsigned long long*)&ev.prio[id], (unsigned long long)(L + f));
    }
}

// ---------------------------------------------------------------------------
// Replication of the hot set (Section 4.1, "Replication of popular
// prefixes"): the replica slots hold the `replicas` host-tier blocks with the
// highest H. The same threshold search ranks the host tier by (H descending,
// id); blocks that left the set free their slots, blocks that entered it are
// paired, in ascending id order, with the free slots in ascending order and
// copied in.
// ---------------------------------------------------------------------------

__global__ void k_rep_setup(DevState* st, TierView tier) {
    const int t = threadIdx.x;
    if (t < kSelPasses) st->sel_done[t] = 0;
    if (t != 0) return;
    const uint64_t count = st->count;
    st->sel_hot = 1;
    st->sel_lo_id = (uint64_t)tier.owned;
    st->sel_hi_id = count > (uint64_t)tier.owned ? count : (uint64_t)tier.owned;
    st->ev_want = (uint64_t)tier.replicas;
    st->ev_all = 0;
    st->sel_range_done = 0;
    st->sel_npass = 0;
    st->sel_hi = 0;
    st->sel_lo = 0;
    st->sel_need = (uint64_t)tier.replicas;
    st->rep_new = 0;
}

// Host-tier blocks that left the hot set give up their slot; those that
// entered it get a bit in enter_mask.
__global__ __launch_bounds__(kThreads) void k_rep_diff(EvictView ev, DevState* st) {
    const TierView& t = ev.tier;
    const int lane = threadIdx.x & (kWave - 1);
    const bool all = st->ev_all != 0;
    const u128 thr = ((u128)st->sel_hi << 64) | (u128)st->sel_lo;
    const int64_t hi_id = (int64_t)st->sel_hi_id;
    const int64_t span = ((t.host_blocks + kWave - 1) / kWave) * kWave;
    unsigned long long dropped = 0;
    for (int64_t h = (int64_t)blockIdx.x * kThreads + threadIdx.x; h - threadIdx.x < span;
         h += (int64_t)gridDim.x * kThreads) {
        const int64_t id = t.owned + h;
        bool hot = false, have = false;
        if (h < t.host_blocks) {
            hot = id < hi_id && (all || sel_key(ev, st, id) <= thr);
            const int32_t slot = t.rep_of[h];
            have = slot >= 0;
            if (have && !hot) {
                t.rep_of[h] = -1;
                t.rep_id[slot] = -1;
                ++dropped;
            }
        }
        const unsigned long long mask = ballot64(hot && !have);
        if (lane == 0 && h / kWave < span / kWave) t.enter_mask[h / kWave] = mask;
    }
    dropped = wave_reduce(dropped, [](uint64_t a, uint64_t b) { return a + b; }, lane);
    if (lane == 0 && dropped) atomicSub(&st->rep_count, dropped);
}

// Exclusive scan over the block (blockDim.x = 1024) of one value per thread;
// returns this thread's offset, *total the sum.
__device__ inline uint32_t block_scan(uint32_t v, uint32_t* part, uint32_t* total) {
    const int t = threadIdx.x, nt = blockDim.x;
    part[t] = v;
    __syncthreads();
    for (int d = 1; d < nt; d <<= 1) {
        const uint32_t x = t >= d ? part[t - d] : 0u;
        __syncthreads();
        part[t] += x;
        __syncthreads();
    }
    const uint32_t incl = part[t];
    *total = part[nt - 1];
    __syncthreads();
    return incl - v;
}

// One workgroup: lists the free slots and the entering blocks in ascending
// order, pairs them and writes the copies to make.
__global__ __launch_bounds__(1024) void k_rep_assign(EvictView ev, DevState* st) {
    const TierView& t = ev.tier;
    __shared__ uint32_t part[1024];
    const int tid = threadIdx.x, nt = blockDim.x;
    uint32_t nfree = 0;
    for (int64_t base = 0; base < t.replicas; base += nt) {
        const int64_t slot = base + tid;
        const uint32_t f = slot < t.replicas && t.rep_id[slot] < 0 ? 1u : 0u;
        uint32_t tot;
        const uint32_t off = block_scan(f, part, &tot);
        if (f) t.free_list[nfree + off] = (int32_t)slot;
        nfree += tot;
    }
    const int64_t words = (t.host_blocks + kWave - 1) / kWave;
    uint32_t nenter = 0;
    for (int64_t base = 0; base < words; base += nt) {
        const int64_t w = base + tid;
        const uint64_t mask = w < words ? t.enter_mask[w] : 0ull;
        uint32_t tot;
        uint32_t off = block_scan((uint32_t)__popcll(mask), part, &tot);
        for (uint64_t m = mask; m; m &= m - 1) {  // the hot set never exceeds the slots
            const int b = __ffsll((long long)m) - 1;
            const uint32_t k = nenter + off++;
            if (k < nfree) t.enter_list[k] = (int32_t)(w * kWave + b);
        }
        nenter += tot;
    }
    if (nenter > nfree) nenter = nfree;
    __syncthreads();
    for (uint32_t k = tid; k < nenter; k += nt) {
        const int32_t h = t.enter_list[k], slot = t.free_list[k];
        t.rep_of[h] = slot;
        t.rep_id[slot] = h;
        Pair p;
        p.row = (int32_t)(t.dev_rows + h);   // host-tier home
        p.cb = (int32_t)(t.owned + slot);    // device replica row
        t.copies[k] = p;
    }
    if (tid == 0) {
        st->rep_new = nenter;
        st->rep_count += nenter;
        st->rep_copies += nenter;
    }
}

unsigned grid_for(int64_t n, int64_t cap_groups) {
    int64_t g = (n + kThreads - 1) / kThreads;
    if (g > cap_groups) g = cap_groups;
    if (g < 1) g = 1;
    return (unsigned)g;
}

}  // namespace

hipError_t launch_evict(const IndexView& ix, const InsertTarget& tgt, const EvictView& ev,
                        hipStream_t s) {
    hipError_t e;
    // about four candidates per thread: few workgroups add to the same bins
    const unsigned g = grid_for((tgt.capacity + 3) / 4, kSelGroups);
    hipLaunchKernelGGL(k_sel_range, dim3(g), dim3(kThreads), 0, s, ev, ix.state);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    for (int p = 0; p < kSelPasses; ++p) {
        hipLaunchKernelGGL(k_sel_pass, dim3(g), dim3(kThreads), 0, s, ev, ix.state, p);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const unsigned gw = grid_for(ev.words * kWave, 2048);
    hipLaunchKernelGGL(k_ev_mark, dim3(gw), dim3(kThreads), 0, s, ev, ix.state, tgt.slots,
                       (const int32_t*)tgt.parent);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_ev_scan, dim3(1), dim3(1024), 0, s, ev, ix.state, tgt.capacity,
                       ix.slot_mask + 1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_ev_list, dim3(gw), dim3(kThreads), 0, s, ev, ix.state);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_rebuild_clear, dim3(grid_for((int64_t)(ix.slot_mask + 1), 2048)), dim3(kThreads),
                       0, s, ix.state, tgt.slots, ix.slot_mask + 1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_rebuild_insert, dim3(g), dim3(kThreads), 0, s, ev, ix.state, tgt.slots,
                       ix.slot_mask, (const int32_t*)tgt.parent, ix.ht);
    return hipGetLastError();
}

hipError_t launch_replicate(const IndexView& ix, const EvictView& ev, const CopyPlan& p,
                            hipStream_t s) {
    hipError_t e;
    const TierView& t = ev.tier;
    hipLaunchKernelGGL(k_rep_setup, dim3(1), dim3(64), 0, s, ix.state, t);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const unsigned g = grid_for((t.host_blocks + 3) / 4, kSelGroups);
    hipLaunchKernelGGL(k_sel_range, dim3(g), dim3(kThreads), 0, s, ev, ix.state);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    for (int k = 0; k < kSelPasses; ++k) {
        hipLaunchKernelGGL(k_sel_pass, dim3(g), dim3(kThreads), 0, s, ev, ix.state, k);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const unsigned gw = grid_for(((t.host_blocks + kWave - 1) / kWave) * kWave, 2048);
    hipLaunchKernelGGL(k_rep_diff, dim3(gw), dim3(kThreads), 0, s, ev, ix.state);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_rep_assign, dim3(1), dim3(1024), 0, s, ev, ix.state);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_copy_rows(p, t.copies, &ix.state->rep_new, t.replicas, s);
}

hipError_t launch_touch_paths(const IndexView& ix, const EvictView& ev, const int32_t* m,
                              const int32_t* ids, int32_t R, int32_t max_blocks, hipStream_t s) {
    const unsigned grid = (unsigned)((R + (kThreads / kWave) - 1) / (kThreads / kWave));
    hipLaunchKernelGGL(k_touch, dim3(grid), dim3(kThreads), 0, s, ev, ix.state, m, ids, R, max_blocks);
    return hipGetLastError();
}

}  // namespace ptsd
