// KV block movement between the store's pool and a caller's paged cache.
//
// Gather is the load of Section 4.1 (iterate over an object's ids and copy
// their tensors into application-supplied GPU memory); scatter stores the
// tensors of blocks an insert created. Both move whole (layer, K|V) chunks
// of heads x slots x dim elements, which are contiguous on both sides:
//   pool  [id][layer][K|V][head][slot][dim]        chunk c at id*block + c*chunk
//   cache [layer][K|V][cache block][head][slot][dim] chunk c at (c*NB + cb)*chunk
//
// The work is flattened over (request, block, group of chunks) units so that
// requests with very different match lengths balance across the GPU; a unit
// whose block is not copied exits at once. Threads move 16-byte vectors with
// non-temporal loads and stores (the stream is touched once). The default
// launch gives each 1024-thread workgroup one chunk (two vectors per thread
// for a 32 KiB chunk): measured on MI355X it kept ~6.2-6.6 TB/s whatever the
// physical placement of pool and cache, where fatter workgroups (8 chunks,
// 256 threads, an 8-deep unrolled stripe per thread) swung between 5.5 and
// 6.6 TB/s. Pure HBM streaming: no LDS, no MFMA.
#include "kernels.hpp"

namespace ptsd {
namespace {

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

constexpr int kUnroll = 8;

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

struct CopyArgs {
    uint8_t* pool;
    uint8_t* cache;
    const int32_t* ids;
    const int32_t* m;          // gather: blocks b < m[r] are copied
    const uint8_t* created;    // scatter: blocks with created != 0 are copied
    const int32_t* block_table;
    int64_t block_bytes;
    int64_t chunk_bytes;
    int64_t cache_blocks;
    int32_t max_blocks;
    int32_t chunks_per_block;
    int32_t chunks_per_group;
    int32_t groups;            // ceil(chunks_per_block / chunks_per_group)
    int64_t units;             // R * max_blocks * groups
    DevState* state;
};

// One unit: group g of the chunks of block b of request r.
template <bool GATHER>
__device__ inline void copy_unit(const CopyArgs& a, int64_t unit) {
    const int64_t rb = unit / a.groups;
    const int g = (int)(unit - rb * a.groups);
    const int64_t r = rb / a.max_blocks;
    const int b = (int)(rb - r * a.max_blocks);
    if (GATHER) {
        if (b >= a.m[r]) return;
    } else {
        if (!a.created[rb]) return;
    }
    const int64_t id = a.ids[rb];
    const int64_t cb = a.block_table[rb];
    if (cb < 0) return;
    if (cb >= a.cache_blocks || id < 0 || id >= (int64_t)a.state->count) {
        if (threadIdx.x == 0 && g == 0) atomicAdd(&a.state->bad_entries, 1ull);
        return;
    }
    const int c0 = g * a.chunks_per_group;
    const int c1 = min(c0 + a.chunks_per_group, a.chunks_per_block);
    const int n16 = (int)(a.chunk_bytes >> 4);
    for (int c = c0; c < c1; ++c) {
        uint8_t* p = a.pool + id * a.block_bytes + (int64_t)c * a.chunk_bytes;
        uint8_t* q = a.cache + ((int64_t)c * a.cache_blocks + cb) * a.chunk_bytes;
        if (GATHER)
            copy_span(reinterpret_cast<const v4u*>(p), reinterpret_cast<v4u*>(q), n16);
        else
            copy_span(reinterpret_cast<const v4u*>(q), reinterpret_cast<v4u*>(p), n16);
    }
}

// Units are visited grid-stride: the grid is capped so that it never exceeds
// the launch limit on total work-items, and is usually one unit per group.
template <bool GATHER>
__global__ __launch_bounds__(1024) void k_copy(CopyArgs a) {
    for (int64_t unit = blockIdx.x; unit < a.units; unit += gridDim.x) copy_unit<GATHER>(a, unit);
}

CopyArgs make_args(const CopyPlan& p, int32_t max_blocks, int64_t cache_blocks) {
    CopyArgs a{};
    a.pool = p.pool;
    a.block_bytes = p.block_bytes;
    a.chunk_bytes = p.chunk_bytes;
    a.cache_blocks = cache_blocks;
    a.max_blocks = max_blocks;
    a.chunks_per_block = p.chunks_per_block;
    a.chunks_per_group = p.chunks_per_group;
    a.groups = (p.chunks_per_block + p.chunks_per_group - 1) / p.chunks_per_group;
    a.state = p.state;
    return a;
}

hipError_t launch(CopyArgs a, bool gather, int32_t R, int threads, hipStream_t s) {
    a.units = (int64_t)R * a.max_blocks * a.groups;
    if (a.units == 0) return hipSuccess;
    const int64_t max_groups = (1ll << 31) / threads;
    const unsigned grid = (unsigned)(a.units < max_groups ? a.units : max_groups);
    if (gather)
        hipLaunchKernelGGL(k_copy<true>, dim3(grid), dim3(threads), 0, s, a);
    else
        hipLaunchKernelGGL(k_copy<false>, dim3(grid), dim3(threads), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gather(const CopyPlan& p, const int32_t* ids, const int32_t* m,
                         const int32_t* block_table, int32_t R, int32_t max_blocks,
                         uint8_t* cache, int64_t cache_blocks, hipStream_t s) {
    CopyArgs a = make_args(p, max_blocks, cache_blocks);
    a.cache = cache;
    a.ids = ids;
    a.m = m;
    a.block_table = block_table;
    return launch(a, true, R, p.threads, s);
}

hipError_t launch_scatter(const CopyPlan& p, const int32_t* ids, const uint8_t* created,
                          const int32_t* block_table, int32_t R, int32_t max_blocks,
                          const uint8_t* cache, int64_t cache_blocks, hipStream_t s) {
    CopyArgs a = make_args(p, max_blocks, cache_blocks);
    a.cache = const_cast<uint8_t*>(cache);
    a.ids = ids;
    a.created = created;
    a.block_table = block_table;
    return launch(a, false, R, p.threads, s);
}

}  // namespace ptsd
