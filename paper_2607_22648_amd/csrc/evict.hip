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
// So the victims are the `want` smallest 128-bit keys (H, 2^31-1-depth, id)
// among the unmatched blocks, found by a radix select: 16 passes, each a
// 256-bin histogram of the next 8-bit digit among the keys that agree with
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

__device__ inline void evict_key(const EvictView& ev, int64_t id, uint64_t* hi, uint64_t* lo) {
    *hi = ev.prio[id];
    *lo = ((uint64_t)(uint32_t)(0x7FFFFFFF - ev.depth[id]) << 32) | (uint32_t)id;
}

__device__ inline unsigned long long lanes_below(int lane) {
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// One digit pass of the threshold search.
__global__ __launch_bounds__(kThreads) void k_sel_pass(EvictView ev, DevState* st, int pass) {
    if (st->ev_want == 0 || st->ev_all) return;  // uniform over the grid
    __shared__ unsigned int h[256];
    __shared__ int last;
    const int t = threadIdx.x;
    h[t] = 0;
    __syncthreads();
    const int64_t old = (int64_t)st->insert_old_count;
    const uint64_t phi = st->sel_hi, plo = st->sel_lo;
    // bits above the digit must equal the threshold's
    const int word = pass < 8 ? 0 : 1;
    const int sh = 56 - 8 * (pass & 7);
    const uint64_t above = (pass & 7) == 0 ? 0ull : (~0ull << (sh + 8));
    for (int64_t id = (int64_t)blockIdx.x * kThreads + t; id < old; id += (int64_t)gridDim.x * kThreads) {
        if (ev.prot[id] == ev.epoch) continue;
        uint64_t hi, lo;
        evict_key(ev, id, &hi, &lo);
        bool match;
        unsigned digit;
        if (word == 0) {
            match = (hi & above) == (phi & above);
            digit = (unsigned)(hi >> sh) & 255u;
        } else {
            match = hi == phi && (lo & above) == (plo & above);
            digit = (unsigned)(lo >> sh) & 255u;
        }
        if (match) atomicAdd(&h[digit], 1u);
    }
    __syncthreads();
    uint32_t* gh = ev.hist + pass * 256;
    if (h[t]) atomicAdd(&gh[t], h[t]);
    __threadfence();
    __syncthreads();
    if (t == 0) last = atomicAdd(&st->sel_done[pass], 1u) == gridDim.x - 1;
    __syncthreads();
    if (!last) return;
    __threadfence();
    h[t] = __hip_atomic_load(&gh[t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (t != 0) return;
    const uint64_t want = st->ev_want;
    if (pass == 0) {
        uint64_t total = 0;
        for (int d = 0; d < 256; ++d) total += h[d];
        if (total <= want) {  // every candidate goes
            st->ev_all = 1;
            return;
        }
    }
    uint64_t need = st->sel_need, cum = 0;
    int d = 0;
    for (; d < 255; ++d) {
        if (cum + h[d] >= need) break;
        cum += h[d];
    }
    st->sel_need = need - cum;
    if (word == 0)
        st->sel_hi = phi | ((uint64_t)d << sh);
    else
        st->sel_lo = plo | ((uint64_t)d << sh);
}

// Marks the victims (one bit per id), deletes their index entries, takes a
// child from their parents and raises the clock to their largest priority.
__global__ __launch_bounds__(kThreads) void k_ev_mark(EvictView ev, DevState* st, Slot* slots,
                                                      const int32_t* parent) {
    if (st->ev_want == 0) return;
    const int lane = threadIdx.x & (kWave - 1);
    const bool all = st->ev_all != 0;
    const uint64_t thi = st->sel_hi, tlo = st->sel_lo;
    const int64_t old = (int64_t)st->insert_old_count;
    const int64_t span = ev.words * kWave;
    uint64_t maxp = 0;
    for (int64_t base = (int64_t)blockIdx.x * kThreads; base < span; base += (int64_t)gridDim.x * kThreads) {
        const int64_t id = base + threadIdx.x;
        bool sel = false;
        if (id < old && ev.prot[id] != ev.epoch) {
            uint64_t hi, lo;
            evict_key(ev, id, &hi, &lo);
            sel = all || hi < thi || (hi == thi && lo <= tlo);
            if (sel) {
                maxp = hi > maxp ? hi : maxp;
                slots[ev.spos[id]].key = kTombKey;
                const int32_t p = parent[id];
                if (p >= 0) atomicSub(&ev.live[p], 1);
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
        if (st->ev_new > fresh + nv) st->full_events += 1;
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
    const unsigned g = grid_for(tgt.capacity, 2048);
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

hipError_t launch_touch_paths(const IndexView& ix, const EvictView& ev, const int32_t* m,
                              const int32_t* ids, int32_t R, int32_t max_blocks, hipStream_t s) {
    const unsigned grid = (unsigned)((R + (kThreads / kWave) - 1) / (kThreads / kWave));
    hipLaunchKernelGGL(k_touch, dim3(grid), dim3(kThreads), 0, s, ev, ix.state, m, ids, R, max_blocks);
    return hipGetLastError();
}

}  // namespace ptsd
