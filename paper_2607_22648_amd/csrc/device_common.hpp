// Device-side building blocks shared by the prefix-store kernels (gfx950).
//
// Keys. A request's block b gets a chained key k_b that depends on all of
// its tokens up to the end of block b: k_b = P * k_{b-1} + c_b (mod 2^61-1),
// where c_b is a 64-bit mix of the block's tokens reduced mod 2^61-1 and
// k_{-1} is a seed-derived root key. Because the chain is affine, the keys of
// a 64-block window come out of one wavefront prefix scan instead of 64
// dependent steps. Keys only steer probing: a hit is accepted only after its
// block's tokens and parent id are compared, so results never depend on the
// hash (the store is exact, as the paper's id lists are).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ptsd {

constexpr uint64_t kM61 = (1ull << 61) - 1;
constexpr uint64_t kEmptyKey = ~0ull;  // never a key: keys are < 2^61
constexpr uint64_t kTombKey = ~1ull;   // slot of an evicted block: probing goes on past it
constexpr int kWave = 64;

// One slot of the open-addressing block index. The parent id rides along
// so that a probe learns a candidate's parent without another load.
struct alignas(16) Slot {
    uint64_t key;    // index key, kEmptyKey if free
    int32_t id;      // block id
    int32_t parent;  // id of the block's parent, -1 for a child of the root
};

// Per-store constants of the key chain, in device memory.
struct HashTables {
    uint64_t pow_lane[kWave];  // P^(j+1), j = 0..63
    uint64_t pow0[kWave];      // P^j
    uint64_t inv_pow[kWave];   // P^-j (mod 2^61-1)
    uint64_t p;                // P
    uint64_t root_key;         // k_{-1}
    uint64_t content_seed;
    uint64_t slot_seed;
    uint32_t weak;             // 1: index keys masked to 8 bits
    uint32_t weak_tag;         // 1: insert batch-table tags keep only the depth's parity
};

// Event counters a lookup adds to are spread over this many slots, each on
// its own 128-byte line, so that thousands of waves adding at once do not
// serialise on one address; readers sum the slots.
constexpr int kCounterSlots = 64;

struct alignas(128) CounterSlot {
    unsigned long long probes;
    unsigned long long token_compares;
    unsigned long long cas_attempts;
    unsigned long long cas_failures;
    unsigned long long pad[12];
};

// Eviction threshold search: at most this many digit passes of kSelBits bits
// each over a key of at most 128 bits.
constexpr int kSelBits = 11;
constexpr int kSelBins = 1 << kSelBits;
constexpr int kSelPasses = (128 + kSelBits - 1) / kSelBits;

// Device-side counters and status of a store.
struct DevState {
    unsigned long long count;         // blocks stored (= next id)
    unsigned long long full_events;
    unsigned long long bad_entries;
    unsigned long long insert_old_count;  // scratch: count before the running insert
    unsigned long long insert_fallbacks;  // inserts that took the exact sequential claim
    // eviction (state)
    unsigned long long clock;         // L: largest priority evicted so far
    unsigned long long evictions;
    unsigned long long tombstones;    // upper bound on deleted index slots
    unsigned long long rebuilds;
    unsigned long long ev_epoch;      // protection mark of the running insert (>= 1),
                                      // advanced by the insert's first kernel
    unsigned long long insert_full;   // 1: the last insert refused blocks for lack of room
    // eviction (scratch of the running insert)
    unsigned long long ev_new;        // distinct new blocks the batch needs
    unsigned long long ev_want;       // blocks to evict
    unsigned long long ev_all;        // 1: every candidate goes (no more than ev_want)
    unsigned long long ev_nv;         // blocks evicted
    unsigned long long ev_rebuild;    // 1: rebuild the index in this insert
    // key layout: only the bits in which candidates differ are kept
    unsigned long long sel_pbase, sel_dmax, sel_imin;  // H base, largest depth, smallest id
    unsigned int sel_wd, sel_wi;        // bit widths of the depth and id fields
    unsigned int sel_w, sel_npass;      // key width, digit passes it needs
    unsigned long long sel_hi, sel_lo;  // threshold key found so far (left-aligned)
    unsigned long long sel_need;        // rank of the threshold among what matches it
    unsigned int sel_range_done;        // workgroups finished the range pass
    unsigned int sel_done[kSelPasses];  // workgroups finished per digit pass
    // what the search ranks: 0 = eviction candidates (ids below sel_hi_id
    // that the batch did not match, key (H, deeper, id)); 1 = the host tier,
    // ids sel_lo_id .. sel_hi_id-1, key (H descending, id)
    unsigned int sel_hot, sel_pad;
    unsigned long long sel_lo_id, sel_hi_id;
    // replication
    unsigned long long rep_count;       // host-tier blocks with a device replica
    unsigned long long rep_copies;      // blocks copied into replica slots so far
    unsigned long long rep_new;         // blocks the running replicate copies
    CounterSlot slot[kCounterSlots];
};

__host__ __device__ inline uint64_t mix64(uint64_t z) {
    // SplitMix64 finaliser (Steele, Lea, Flood 2014)
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__host__ __device__ inline uint64_t mod61(uint64_t x) {
    x = (x & kM61) + (x >> 61);
    return x >= kM61 ? x - kM61 : x;
}

__device__ inline uint64_t mulmod61(uint64_t a, uint64_t b) {
    uint64_t lo = a * b;
    uint64_t hi = __umul64hi(a, b);
    uint64_t x = (lo & kM61) + ((lo >> 61) | (hi << 3));
    return mod61(x);
}

__device__ inline uint64_t addmod61(uint64_t a, uint64_t b) { return mod61(a + b); }

// Content hash of one block of bt tokens: tokens are taken in pairs (i, i+1)
// (the last one alone when bt is odd), each pair mixed into the state; the
// result is reduced mod 2^61-1. The three steps below are the only
// definition, so every caller (whole block in registers, streamed from LDS,
// read from memory) gets the same value.
__device__ inline uint64_t content_hash_init(uint64_t seed, int bt) {
    return seed ^ (0x9E3779B97F4A7C15ull * (uint64_t)bt);
}
__device__ inline uint64_t content_hash_pair(uint64_t h, int32_t lo, int32_t hi, int i) {
    const uint64_t w = (uint64_t)(uint32_t)lo | ((uint64_t)(uint32_t)hi << 32);
    return mix64(h ^ (w + 0x632BE59BD9B4E019ull * (uint64_t)(i + 1)));
}
__device__ inline uint64_t content_hash_final(uint64_t h) { return mod61(mix64(h)); }

__device__ inline uint64_t content_hash_mem(const int32_t* __restrict__ blk, int bt, uint64_t seed) {
    uint64_t h = content_hash_init(seed, bt);
    for (int i = 0; i < bt; i += 2) h = content_hash_pair(h, blk[i], i + 1 < bt ? blk[i + 1] : 0, i);
    return content_hash_final(h);
}

// One index slot in one 16-byte load: a probe learns the key, the id and the
// parent of a slot at once, with no second dependent load.
__device__ inline Slot load_slot(const Slot* p) {
    typedef unsigned int v4u_t __attribute__((ext_vector_type(4)));
    const v4u_t v = *reinterpret_cast<const v4u_t*>(p);
    Slot s;
    s.key = ((uint64_t)v.y << 32) | (uint64_t)v.x;
    s.id = (int32_t)v.z;
    s.parent = (int32_t)v.w;
    return s;
}

__device__ inline uint64_t index_key(uint64_t k, const HashTables& ht) {
    return ht.weak ? (k & 0xFFull) : k;
}

__device__ inline uint64_t slot_of(uint64_t ikey, uint64_t seed, uint64_t mask) {
    return mix64(ikey ^ seed) & mask;
}

// 64-bit wavefront shuffles built from 32-bit ones.
__device__ inline uint64_t shfl_u64(uint64_t v, int src) {
    uint32_t lo = __shfl((int)(uint32_t)v, src, kWave);
    uint32_t hi = __shfl((int)(uint32_t)(v >> 32), src, kWave);
    return ((uint64_t)hi << 32) | lo;
}

__device__ inline uint64_t shfl_up_u64(uint64_t v, int d) {
    uint32_t lo = __shfl_up((int)(uint32_t)v, d, kWave);
    uint32_t hi = __shfl_up((int)(uint32_t)(v >> 32), d, kWave);
    return ((uint64_t)hi << 32) | lo;
}

// The constants of the key chain a lane uses, read from HashTables once per
// kernel and then held in registers, so that no table read sits between a
// window's tokens and its probes.
struct ChainConsts {
    uint64_t lane_pow;  // P^(lane+1)
    uint64_t pow0;      // P^lane
    uint64_t inv;       // P^-lane
    uint64_t p;         // P
    uint64_t root_key;
    uint64_t content_seed;
    uint64_t slot_seed;
    uint32_t weak;
};

__device__ inline ChainConsts chain_consts(const HashTables* __restrict__ ht, int lane) {
    ChainConsts c;
    c.lane_pow = ht->pow_lane[lane];
    c.pow0 = ht->pow0[lane];
    c.inv = ht->inv_pow[lane];
    c.p = ht->p;
    c.root_key = ht->root_key;
    c.content_seed = ht->content_seed;
    c.slot_seed = ht->slot_seed;
    c.weak = ht->weak;
    return c;
}

__device__ inline uint64_t index_key(uint64_t k, const ChainConsts& c) {
    return c.weak ? (k & 0xFFull) : k;
}

// The affine key chain over one 64-block window. With c_i the content hash
// of block w0+i (0 past the request's end) and carry = k_{w0-1}, lane j's key
//   k_{w0+j} = P^(j+1) carry + sum_{i<=j} P^(j-i) c_i
//            = P^j (P carry + sum_{i<=j} P^-i c_i)          (mod 2^61-1),
// so one product per lane turns the hashes into terms P^-i c_i, a wave
// prefix sum of plain modular additions adds them up, and one more product
// (P carry is the same in every lane) gives the key: the same values as
// folding the chain block by block, with 2 products per lane instead of 7.
__device__ inline uint64_t window_chain(uint64_t c, uint64_t carry, const ChainConsts& cc, int lane) {
    uint64_t s = mulmod61(c, cc.inv);
#pragma unroll
    for (int t = 0; t < 6; ++t) {
        const int d = 1 << t;
        const uint64_t sp = shfl_up_u64(s, d);
        if (lane >= d) s = addmod61(s, sp);
    }
    return mulmod61(cc.pow0, addmod61(mulmod61(cc.p, carry), s));
}

__device__ inline unsigned long long ballot64(bool p) { return __ballot(p); }

// Sum of a per-lane count over the wave, the same in every lane. Counts
// are mostly 0, 1 or 2 (probes, comparisons, CAS attempts), so the sum is
// first taken as the number of lanes whose count reaches k, for k = 1..4:
// one ballot each and no lane shuffles. What larger counts hold beyond 4
// goes through a shuffle tree, only when some lane has such a count.
__device__ inline unsigned long long wave_sum(unsigned long long v, int lane) {
    unsigned long long sum = 0;
#pragma unroll
    for (unsigned k = 1; k <= 4; ++k) sum += __popcll(ballot64(v >= k));
    if (ballot64(v > 4)) {
        unsigned long long x = v > 4 ? v - 4 : 0;
#pragma unroll
        for (int d = 32; d >= 1; d >>= 1) x += (unsigned long long)shfl_u64(x, lane ^ d);
        sum += x;
    }
    return sum;
}

// Sum of a per-lane count over the wave, added once to a device counter.
__device__ inline void wave_count(unsigned long long* ctr, unsigned long long v, int lane) {
    const unsigned long long t = wave_sum(v, lane);
    if (lane == 0 && t) atomicAdd(ctr, t);
}

// Sum of a per-lane count over the wave, taken once from a device counter.
__device__ inline void wave_sub(unsigned long long* ctr, unsigned long long v, int lane) {
    const unsigned long long t = wave_sum(v, lane);
    if (lane == 0 && t) atomicSub(ctr, t);
}

// The counter slot a wave adds to.
__device__ inline CounterSlot* counter_slot(DevState* st) {
    const unsigned w = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    return &st->slot[w & (kCounterSlots - 1)];
}

}  // namespace ptsd
