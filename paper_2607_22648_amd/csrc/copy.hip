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
//           the counts, then write a dense descriptor list of (id, cache
//           block) pairs, compacted with a wave ballot (three kernels; one
//           workgroup does all three for a small batch). Entries with an id
//           or cache block out of range are dropped here and counted.
//   copy    workgroups walk (descriptor, group of chunks) units; the number
//           of units is read on the device, so no host round trip separates
//           the parts. Threads move 16-byte vectors with non-temporal loads
//           and stores (the stream is touched once).
// Only blocks that are really copied cost work, however sparse they are in
// the [request][block] arrays (a few created blocks per insert, half the
// requests missing the store). The default copy shape gives each
// 1024-thread workgroup one chunk per unit (two vectors per thread for a
// 32 KiB chunk). The copies are pure HBM streaming: no MFMA, and LDS only for
// the per-layer kernel's table of layer bases.
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
        if (dev) a.sc.pairs[pos + __popcll(mask & lanes_below(lane))] = p;
        if (sel && !dev) a.sc.pairs[pos_h + __popcll(mask_h & lanes_below(lane))] = p;
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
    if (t == 0) {
        *a.sc.total = (unsigned long long)carry;
        *a.sc.total_h = (unsigned long long)carry_h;
    }
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

// Small batches: count, scan and fill in one workgroup, the counts and
// bases in LDS, so that building the list costs one launch instead of
// three. Wave w takes requests w, w+16, ...; with at most 4 requests of at
// most 2 windows per wave (the host's condition) its serial walk stays as
// short as the three kernels' launch gaps.
constexpr int kSmallThreads = 1024;
constexpr int kSmallWaves = kSmallThreads / kWave;
constexpr int32_t kSmallMaxR = 64;
constexpr int64_t kSmallMaxEntries = 8192;

template <bool GATHER>
__global__ __launch_bounds__(kSmallThreads) void k_select_small(SelectArgs a) {
    __shared__ int32_t base[kSmallMaxR], base_h[kSmallMaxR];
    __shared__ int32_t total_dev;
    const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
    const unsigned long long count = a.state->count;
    int32_t bad = 0;
    for (int r = wv; r < a.R; r += kSmallWaves) {
        int32_t c, ch;
        count_row<GATHER>(a, r, lane, count, &c, &ch, &bad);
        if (lane == 0) {
            base[r] = c;
            base_h[r] = ch;
        }
    }
    if (lane == 0 && bad) atomicAdd(&a.state->bad_entries, (unsigned long long)bad);
    __syncthreads();
    // exclusive scan over the requests, thread t holding request t (R <= 64:
    // the first wave); totals of at most kSmallMaxEntries fit in 32 bits
    const int t = threadIdx.x;
    if (wv == 0) {
        const int32_t v = t < a.R ? base[t] : 0, vh = t < a.R ? base_h[t] : 0;
        int32_t s = v, sh = vh;
        for (int d = 1; d < kWave; d <<= 1) {
            const int32_t x = __shfl_up(s, d, kWave), xh = __shfl_up(sh, d, kWave);
            if (lane >= d) {
                s += x;
                sh += xh;
            }
        }
        if (t < a.R) {
            base[t] = s - v;
            base_h[t] = sh - vh;
        }
        if (lane == kWave - 1) {
            total_dev = s;
            *a.sc.total = (unsigned long long)s;
            *a.sc.total_h = (unsigned long long)sh;
        }
    }
    __syncthreads();
    const int64_t total = total_dev;  // host rows after all device rows
    for (int r = wv; r < a.R; r += kSmallWaves)
        fill_row<GATHER>(a, r, lane, count, base[r], total + base_h[r]);
}

struct CopyArgs {
    uint8_t* pool;
    uint8_t* host;      // host tier: rows dev_rows.. of the pool's row space
    int64_t dev_rows;
    uint8_t* cache;
    const Pair* pairs;
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
// 2048 times what the device holds at once, so the dense front of the list
// runs in hardware dispatch order (neighbouring workgroups copy neighbouring
// chunks; past the cap a workgroup also takes the unit one grid further on,
// and workgroups past the end exit at once); a scatter, whose created blocks
// are sparse, launches 16 times what the device holds, looping.
// Uniform slabs: a unit is (descriptor, group of chunks_per_group slabs).
template <bool GATHER>
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
            uint8_t* src = blk + (int64_t)c * a.chunk_bytes;
            uint8_t* dst = a.cache + ((int64_t)c * a.cache_blocks + p.cb) * a.chunk_bytes;
            if (GATHER)
                copy_span(reinterpret_cast<const v4u*>(src), reinterpret_cast<v4u*>(dst), n16);
            else
                copy_span(reinterpret_cast<const v4u*>(dst), reinterpret_cast<v4u*>(src), n16);
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

// Pool and cache addresses of the 16 bytes at range offset o of layer li
// (lb relative to the first layer of the call, l0).
__device__ inline void span_vec(const CopyArgs& a, const int64_t* lb, int li, int64_t o, int32_t cb,
                                uint8_t* blk, v4u** pv, v4u** cv) {
    const int64_t ch = (lb[li + 1] - lb[li]) >> 1;  // the layer's K (or V) slab
    const int64_t in = o - lb[li];
    const int kv = in >= ch ? 1 : 0;
    *pv = reinterpret_cast<v4u*>(blk + o);
    *cv = reinterpret_cast<v4u*>(a.cache + a.cache_blocks * lb[li] +
                                 ((int64_t)kv * a.cache_blocks + cb) * ch + (in - kv * ch));
}

template <bool GATHER>
__global__ __launch_bounds__(1024) void k_copy_spans(CopyArgs a) {
    __shared__ int64_t lb[kMaxVarLayers + 1];
    const unsigned long long spans = (unsigned)a.groups;  // kSpanBytes units per descriptor
    const unsigned long long units = *a.total * spans;
    const Pair* pairs = a.pairs + (a.first ? *a.first : 0ull);
    if (blockIdx.x >= units) return;  // the whole workgroup: nothing to move
    const int l0 = a.c_lo >> 1, l1 = a.c_hi >> 1, n = l1 - l0;
    for (int l = l0 + (int)threadIdx.x; l <= l1; l += blockDim.x) lb[l - l0] = a.lbase[l];
    __syncthreads();
    const int64_t b0 = lb[0], b1 = lb[n];
    const int64_t step = 16 * (int64_t)blockDim.x;
    for (unsigned long long unit = blockIdx.x; unit < units; unit += gridDim.x) {
        const unsigned long long d = unit / spans;
        const int64_t s0 = b0 + (int64_t)(unit - d * spans) * kSpanBytes;
        const int64_t s1 = min(s0 + (int64_t)kSpanBytes, b1);
        const Pair p = pairs[d];
        uint8_t* blk = p.row < a.dev_rows ? a.pool + (int64_t)p.row * a.block_bytes
                                          : a.host + (int64_t)(p.row - a.dev_rows) * a.block_bytes;
        // two vectors per thread in flight: both loaded before either is stored
        int li = 0;
        for (int64_t o = s0 + 16 * (int64_t)threadIdx.x; o < s1; o += 2 * step) {
            const bool two = o + step < s1;
            li = slab_from(lb, li, n, o);
            v4u *pv0, *cv0, *pv1 = nullptr, *cv1 = nullptr;
            span_vec(a, lb, li, o, p.cb, blk, &pv0, &cv0);
            int li1 = li;
            if (two) {
                li1 = slab_from(lb, li, n, o + step);
                span_vec(a, lb, li1, o + step, p.cb, blk, &pv1, &cv1);
            }
            const v4u x0 = ld_nt(GATHER ? pv0 : cv0);
            v4u x1;
            if (two) x1 = ld_nt(GATHER ? pv1 : cv1);
            st_nt(GATHER ? cv0 : pv0, x0);
            if (two) st_nt(GATHER ? cv1 : pv1, x1);
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
    SelectArgs a{ids, m, created, bt, R, max_blocks, cache_blocks, p.state, sc, p.tier};
    if (R <= kSmallMaxR && (int64_t)R * max_blocks <= kSmallMaxEntries) {
        hipLaunchKernelGGL(k_select_small<GATHER>, dim3(1), dim3(kSmallThreads), 0, s, a);
        return hipGetLastError();
    }
    const unsigned grid = (unsigned)((R + kSelWaves - 1) / kSelWaves);
    hipLaunchKernelGGL(k_select_count<GATHER>, dim3(grid), dim3(kSelThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_select_scan, dim3(1), dim3(1024), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_select_fill<GATHER>, dim3(grid), dim3(kSelThreads), 0, s, a);
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
    a.total = sc.total;
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
    else
        hipLaunchKernelGGL(k_copy_pairs<GATHER>, dim3((unsigned)grid), dim3(p.threads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.tier.host_blocks == 0) return e;
    // host-tier rows: bound by the host link, so a small looping grid moves
    // them and the device's other compute units stay free for device rows
    // (of this call or of calls on other streams)
    CopyArgs h = a;
    h.first = sc.total;
    h.total = sc.total_h;
    int64_t hg = p.host_grid;
    if (hg > bound) hg = bound;
    if (hg > cap) hg = cap;
    if (p.lbase)
        hipLaunchKernelGGL(k_copy_spans<GATHER>, dim3((unsigned)hg), dim3(p.threads), 0, s, h);
    else
        hipLaunchKernelGGL(k_copy_pairs<GATHER>, dim3((unsigned)hg), dim3(p.threads), 0, s, h);
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

size_t copy_scratch_bytes(int32_t R, int32_t max_blocks) {
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    return up((size_t)R * max_blocks * sizeof(Pair)) + 2 * up((size_t)R * 4) + 2 * up((size_t)R * 8) + 256;
}

void copy_scratch_carve(void* base, int32_t R, int32_t max_blocks, CopyScratch* out) {
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    uint8_t* q = static_cast<uint8_t*>(base);
    out->pairs = reinterpret_cast<Pair*>(q);
    q += up((size_t)R * max_blocks * sizeof(Pair));
    out->row_cnt = reinterpret_cast<int32_t*>(q);
    q += up((size_t)R * 4);
    out->row_cnt_h = reinterpret_cast<int32_t*>(q);
    q += up((size_t)R * 4);
    out->row_base = reinterpret_cast<int64_t*>(q);
    q += up((size_t)R * 8);
    out->row_base_h = reinterpret_cast<int64_t*>(q);
    q += up((size_t)R * 8);
    out->total = reinterpret_cast<unsigned long long*>(q);
    out->total_h = out->total + 1;
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
