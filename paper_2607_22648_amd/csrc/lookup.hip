// Batched longest-common-prefix lookup (PTStore Section 4.1, the LCP query:
// the longest prefix of a request that is stored, and the ids along it).
//
// One wavefront per request, lane j owns block w0+j of a 64-block window:
//   1. the wave copies the window's tokens into LDS with coalesced loads and
//      each lane hashes its block from there;
//   2. a wave prefix scan chains the hashes into per-block prefix keys;
//   3. each lane probes the open-addressing index for its key up to the
//      first key hit; the hits' stored tokens are compared by four lanes per
//      row, and a lane whose hit holds other tokens probes on, so it accepts
//      the first slot whose stored block has the same tokens;
//   4. the candidate of lane j must have as parent the id accepted by lane
//      j-1 (the root, -1, for block 0; the slot carries the parent id, so this
//      costs no extra load); a ballot finds the first lane that
//      fails, which is the end of the match. If that lane did find a block
//      with the right tokens but the wrong parent (two prefixes whose keys
//      collide), it keeps probing for one with the right parent before the
//      window is decided, so the answer never depends on the hash.
// Windows are walked in order and the walk stops at the first miss; for
// requests with room for more than one window, k_lookup_wide gives each
// window of a round its own wave instead.
// With eviction on, every matched block counts one access: its frequency F
// grows by one and its priority becomes max(H, L + F), which is L + F for
// the final F whatever order the atomics land in.
#include "kernels.hpp"

namespace ptsd {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerGroup = kThreads / kWave;

// Makes a wave's LDS writes visible to its other lanes and keeps the
// compiler from moving LDS accesses across this point. A wave's LDS
// operations are performed in the order it issues them, so no other wave
// takes part.
__device__ inline void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// All four bits of each 4-bit group of b set -> one bit per group (16 bits).
__device__ inline uint64_t quads_all(uint64_t b) {
    uint64_t t = b & (b >> 1);
    t = t & (t >> 2) & 0x1111111111111111ull;
    t = (t | (t >> 3)) & 0x0303030303030303ull;
    t = (t | (t >> 6)) & 0x000F000F000F000Full;
    t = (t | (t >> 12)) & 0x000000FF000000FFull;
    return (t | (t >> 24)) & 0xFFFFull;
}

constexpr int kQuads = 4;  // 16-byte pieces of a block of 16 tokens

// A window of up to 64 blocks of 16 tokens of one request, staged in the
// wave's own LDS area. The request is read with coalesced 16-byte loads
// (consecutive lanes, consecutive bytes: a 4 KiB window costs 64 requests to
// the L2 instead of 256 when each lane read its own block), and each lane
// then hashes and compares its block from LDS. Stored rows are compared four
// lanes to a row, so one load instruction reads 16 whole 64-byte rows.
struct Window16 {
    int4* sh;  // [kWave][kQuads], this wave's area
    int lane;

    // area: the workgroup's LDS, kWave * kQuads int4 per wave
    __device__ inline void init(int4* area, int wave, int l) {
        sh = area + wave * (kWave * kQuads);
        lane = l;
    }

    // n > w0. All of a lane's loads are issued before any is waited for:
    // pieces past the window's end re-read its last piece (always inside the
    // request) and land in LDS rows no lane reads.
    __device__ inline void stage(const int32_t* __restrict__ seq, int w0, int n, int) {
        wave_lds_sync();  // the previous window's reads are issued
        const int nq = (n - w0 < kWave ? n - w0 : kWave) * kQuads;
        const int32_t* base = seq + (int64_t)w0 * 16;
        if ((reinterpret_cast<uintptr_t>(base) & 15) == 0) {
            const int q0 = lane, q1 = kWave + lane, q2 = 2 * kWave + lane, q3 = 3 * kWave + lane;
            const int4 v0 = *reinterpret_cast<const int4*>(base + 4 * (q0 < nq ? q0 : nq - 1));
            const int4 v1 = *reinterpret_cast<const int4*>(base + 4 * (q1 < nq ? q1 : nq - 1));
            const int4 v2 = *reinterpret_cast<const int4*>(base + 4 * (q2 < nq ? q2 : nq - 1));
            const int4 v3 = *reinterpret_cast<const int4*>(base + 4 * (q3 < nq ? q3 : nq - 1));
            sh[q0] = v0;
            sh[q1] = v1;
            sh[q2] = v2;
            sh[q3] = v3;
        } else {
            int32_t* d = reinterpret_cast<int32_t*>(sh);
            for (int q = lane; q < 4 * nq; q += kWave) d[q] = base[q];
        }
        wave_lds_sync();
    }
    // streamed from LDS a piece at a time (four tokens live, not sixteen)
    __device__ inline uint64_t hash(uint64_t seed, int) const {
        uint64_t h = content_hash_init(seed, 16);
#pragma unroll
        for (int i = 0; i < kQuads; ++i) {
            const int4 v = sh[lane * kQuads + i];
            h = content_hash_pair(h, v.x, v.y, 4 * i);
            h = content_hash_pair(h, v.z, v.w, 4 * i + 2);
        }
        return content_hash_final(h);
    }
    // This lane's block against one stored row (64-byte aligned). Only the
    // rare paths (a key hit with other tokens, a key collision between
    // prefixes) compare one lane at a time, so this takes one piece per step
    // to keep the kernel's register count down.
    __device__ inline bool equals(const int32_t* __restrict__ s, int) const {
        bool eq = true;
#pragma unroll 1
        for (int i = 0; i < kQuads; ++i) {
            const int4 v = *reinterpret_cast<const int4*>(s + 4 * i);
            const int4 w = sh[lane * kQuads + i];
            eq &= (v.x == w.x) & (v.y == w.y) & (v.z == w.z) & (v.w == w.w);
        }
        return eq;
    }
    // Token check of every lane's candidate (-1: none); called by the whole
    // wave. Returns whether this lane's candidate row holds its tokens. The
    // four row loads are issued together; a lane of a block without a
    // candidate reads row 0 (always allocated) and ignores it.
    __device__ inline bool verify(const int32_t* __restrict__ tokens, int32_t cand, int) const {
        constexpr int G = kWave / 16;
        int32_t id[G];
        int4 v[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            id[g] = __shfl(cand, g * 16 + (lane >> 2), kWave);
            const int64_t row = id[g] >= 0 ? id[g] : 0;
            v[g] = *reinterpret_cast<const int4*>(tokens + row * 16 + 4 * (lane & 3));
        }
        uint64_t ok = 0;  // bit j: block j's candidate row holds block j's tokens
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int4 w = sh[(g * 16 + (lane >> 2)) * kQuads + (lane & 3)];
            const bool eq = (id[g] >= 0) & (v[g].x == w.x) & (v[g].y == w.y) & (v[g].z == w.z) &
                            (v[g].w == w.w);
            ok |= quads_all(ballot64(eq)) << (16 * g);
        }
        return (ok >> lane) & 1;
    }
};

// Any block size: each lane reads its own block from the request.
struct WindowAny {
    const int32_t* p;  // this lane's block (meaningful for lanes inside the request)
    int lane;

    __device__ inline void init(int4*, int, int l) { lane = l; }

    __device__ inline void stage(const int32_t* __restrict__ seq, int w0, int, int bt) {
        p = seq + (int64_t)(w0 + lane) * bt;
    }
    __device__ inline uint64_t hash(uint64_t seed, int bt) const { return content_hash_mem(p, bt, seed); }
    __device__ inline bool equals(const int32_t* __restrict__ s, int bt) const {
        for (int i = 0; i < bt; ++i)
            if (s[i] != p[i]) return false;
        return true;
    }
    __device__ inline bool verify(const int32_t* __restrict__ tokens, int32_t cand, int bt) const {
        return cand >= 0 && equals(tokens + (int64_t)cand * bt, bt);
    }
};

// The window type for a compile-time block size (0: a run-time one).
template <int BT>
struct WindowOf {
    static_assert(BT == 0 || BT == 16, "block sizes: 16, or any at run time");
    typedef WindowAny type;
};
template <>
struct WindowOf<16> {
    typedef Window16 type;
};

// First slot along the probe sequence from `pos` that holds `ikey`, its
// tokens not yet compared; -1 at the first empty slot. *pos_out is the slot
// and *parent_out the block's parent id.
__device__ inline int32_t probe_key(const IndexView& ix, uint64_t ikey, uint64_t pos, uint64_t* pos_out,
                                    int32_t* parent_out, unsigned* probes) {
    while (true) {
        const Slot s = load_slot(ix.slots + pos);
        ++*probes;
        if (s.key == kEmptyKey) {
            *pos_out = pos;
            return -1;
        }
        if (s.key == ikey) {
            *pos_out = pos;
            *parent_out = s.parent;
            return s.id;
        }
        pos = (pos + 1) & ix.slot_mask;
    }
}

// Linear probing from `pos` for a slot holding `ikey` whose block has the
// lane's tokens (and, if need_parent, parent id `want_parent`), comparing as
// it goes. Returns the block id or -1 at the first empty slot.
template <class Win>
__device__ inline int32_t probe(const IndexView& ix, uint64_t ikey, uint64_t pos, const Win& win,
                                bool need_parent, int32_t want_parent, uint64_t* pos_out,
                                int32_t* parent_out, unsigned* probes, unsigned* cmps) {
    const int bt = ix.block_tokens;
    while (true) {
        const Slot s = load_slot(ix.slots + pos);
        ++*probes;
        if (s.key == kEmptyKey) {
            *pos_out = pos;
            return -1;
        }
        if (s.key == ikey && (!need_parent || s.parent == want_parent)) {
            ++*cmps;
            if (win.equals(ix.tokens + (int64_t)s.id * bt, bt)) {
                *pos_out = pos;
                *parent_out = s.parent;
                return s.id;
            }
        }
        pos = (pos + 1) & ix.slot_mask;
    }
}

// Every lane's first block along its key's probe sequence that holds its
// tokens (-1: none); called by the whole wave. All lanes find their first
// key hit, the hits' tokens are compared together, and a lane whose hit
// holds other tokens (a content-hash collision) probes on alone.
template <class Win>
__device__ inline int32_t find_block(const IndexView& ix, const Win& win, bool active, uint64_t ik,
                                     uint64_t slot_seed, uint64_t* pos, int32_t* par, unsigned* probes,
                                     unsigned* cmps) {
    int32_t cand = -1;
    if (active) {
        cand = probe_key(ix, ik, slot_of(ik, slot_seed, ix.slot_mask), pos, par, probes);
        if (cand >= 0) ++*cmps;
    }
    const bool same = win.verify(ix.tokens, cand, ix.block_tokens);
    if (cand >= 0 && !same)
        cand = probe(ix, ik, (*pos + 1) & ix.slot_mask, win, false, 0, pos, par, probes, cmps);
    return cand;
}

// Request bounds; a malformed request is empty and counted.
__device__ inline int32_t request_blocks(const Batch& b, int64_t r, int bt, int lane,
                                         DevState* st, int64_t* o0) {
    int64_t a = b.offsets[r], e = b.offsets[r + 1];
    if (a < 0 || e < a || e > b.n_tokens) {
        if (lane == 0) atomicAdd(&st->bad_entries, 1ull);
        *o0 = 0;
        return 0;
    }
    *o0 = a;
    int64_t n = (e - a) / bt;
    return (int32_t)(n < b.max_blocks ? n : b.max_blocks);
}

// TOUCH: count accesses (eviction on); a variant of its own so that the
// plain lookup keeps its register count.
template <int BT, bool TOUCH>
__global__ __launch_bounds__(kThreads) void k_lookup(IndexView ix, Batch bat, int32_t* __restrict__ m_out,
                                                     int32_t* __restrict__ ids_out) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r = (int64_t)blockIdx.x * kWavesPerGroup + (threadIdx.x / kWave);
    if (r >= bat.R) return;  // uniform per wave
    const int bt = BT ? BT : ix.block_tokens;
    const ChainConsts cc = chain_consts(ix.ht, lane);
    int64_t o0;
    const int32_t n = request_blocks(bat, r, bt, lane, ix.state, &o0);
    const int32_t* __restrict__ seq = bat.tokens + o0;
    int32_t* __restrict__ row = ids_out + r * bat.max_blocks;
    __shared__ int4 sh_tok[BT == 16 ? kThreads * kQuads : 1];
    typename WindowOf<BT>::type win;
    win.init(sh_tok, threadIdx.x / kWave, lane);

    const uint64_t clock = TOUCH ? ix.state->clock : 0;
    uint64_t carry_key = cc.root_key;
    int32_t carry_id = -1;  // the root
    int32_t m = 0;
    unsigned probes = 0, cmps = 0;
    int w0 = 0;
    bool done = false;
    for (; w0 < n && !done; w0 += kWave) {
        const int b = w0 + lane;
        const bool active = b < n;
        win.stage(seq, w0, n, bt);
        const uint64_t c = active ? win.hash(cc.content_seed, bt) : 0;
        const uint64_t k = window_chain(c, carry_key, cc, lane);
        const uint64_t ik = index_key(k, cc);
        int32_t cpar = -2;
        uint64_t pos = 0;
        int32_t cand = find_block(ix, win, active, ik, cc.slot_seed, &pos, &cpar, &probes, &cmps);
        int first_bad = kWave;
        while (true) {
            int32_t prev = __shfl_up(cand, 1, kWave);
            if (lane == 0) prev = carry_id;
            const int32_t par = cand >= 0 ? cpar : -2;
            const bool ok = active && cand >= 0 && par == prev;
            const unsigned long long bad = ballot64(!ok);
            if (bad == 0) break;
            const int f = __ffsll((long long)bad) - 1;
            const int retry = __shfl((active && cand >= 0 && par != prev) ? 1 : 0, f, kWave);
            if (!retry) {
                first_bad = f;
                break;
            }
            // keys of two different prefixes collided: lane f looks further
            // along its probe sequence for the block with the right parent
            if (lane == f)
                cand = probe(ix, ik, (pos + 1) & ix.slot_mask, win, true, prev, &pos, &cpar,
                             &probes, &cmps);
        }
        if (active) row[b] = lane < first_bad ? cand : -1;
        if (TOUCH && active && lane < first_bad) {
            const uint64_t f = atomicAdd((unsigned long long*)&ix.freq[cand], 1ull) + 1ull;
            atomicMax((unsigned long long*)&ix.prio[cand], (unsigned long long)(clock + f));
        }
        if (first_bad < kWave) {
            m = w0 + first_bad;
            done = true;
        } else {
            m = w0 + kWave;
            carry_id = __shfl(cand, kWave - 1, kWave);
            carry_key = shfl_u64(k, kWave - 1);
        }
    }
    const int fill_from = w0 < n ? w0 : n;
    for (int b = fill_from + lane; b < bat.max_blocks; b += kWave) row[b] = -1;
    if (lane == 0) m_out[r] = m;
    if (ix.counters) {
        CounterSlot* cs = counter_slot(ix.state);
        wave_count(&cs->probes, probes, lane);
        wave_count(&cs->token_compares, cmps, lane);
    }
}

// Long requests: one workgroup of W waves per request, each wave on its
// own window, W windows per round instead of one after another. Within a
// round each wave scans its window's key chain from a zero carry; the affine
// chain makes window w's carry P^64 * (carry of window w-1) + (its offset),
// folded over the round's earlier windows from LDS, so every lane then has
// its key and probes at once. A position's parent check needs the candidate
// of the position before it, across a wave boundary through LDS. The round's
// first failing position decides; only when it found the right tokens under
// another parent (a key collision) does that lane probe on, and the round is
// checked again.
template <int BT, bool TOUCH, int W>
__global__ __launch_bounds__(W * kWave) void k_lookup_wide(IndexView ix, Batch bat,
                                                           int32_t* __restrict__ m_out,
                                                           int32_t* __restrict__ ids_out) {
    __shared__ uint64_t sh_off[W];   // each window's chain offset (zero carry)
    __shared__ int32_t sh_last[W];   // candidate of each window's last lane
    __shared__ int32_t sh_fail[W];   // first failing lane per window (kWave: none)
    __shared__ int32_t sh_retry[W];  // 1: that lane found the tokens under another parent
    __shared__ uint64_t sh_klast;    // key of the round's last position
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x / kWave;
    const int64_t r = blockIdx.x;
    if (r >= bat.R) return;  // uniform over the workgroup
    const int bt = BT ? BT : ix.block_tokens;
    const ChainConsts cc = chain_consts(ix.ht, lane);
    int64_t o0;
    const int32_t n = request_blocks(bat, r, bt, wv == 0 ? lane : 1, ix.state, &o0);
    const int32_t* __restrict__ seq = bat.tokens + o0;
    int32_t* __restrict__ row = ids_out + r * bat.max_blocks;
    const uint64_t clock = TOUCH ? ix.state->clock : 0;
    const uint64_t p64 = ix.ht->pow_lane[kWave - 1];  // P^64
    __shared__ int4 sh_tok[BT == 16 ? W * kWave * kQuads : 1];
    typename WindowOf<BT>::type win;
    win.init(sh_tok, wv, lane);
    uint64_t carry_key = cc.root_key;
    int32_t carry_id = -1;  // the root
    int32_t m = n;
    unsigned probes = 0, cmps = 0;
    int r0 = 0;  // first block of the round
    for (; r0 < n; r0 += W * kWave) {
        const int b = r0 + wv * kWave + lane;
        const bool active = b < n;
        win.stage(seq, r0 + wv * kWave, n, bt);
        const uint64_t c = active ? win.hash(cc.content_seed, bt) : 0;
        const uint64_t sl = window_chain(c, 0, cc, lane);  // zero-carry chain
        if (lane == kWave - 1) sh_off[wv] = sl;
        __syncthreads();
        uint64_t carry = carry_key;
        for (int i = 0; i < wv; ++i) carry = addmod61(mulmod61(p64, carry), sh_off[i]);
        const uint64_t k = addmod61(mulmod61(cc.lane_pow, carry), sl);
        const uint64_t ik = index_key(k, cc);
        int32_t cpar = -2;
        uint64_t pos = 0;
        int32_t cand = find_block(ix, win, active, ik, cc.slot_seed, &pos, &cpar, &probes, &cmps);
        if (wv == W - 1 && lane == kWave - 1) sh_klast = k;
        int fail = W * kWave;  // first failing position of the round, relative to r0
        while (true) {
            if (lane == kWave - 1) sh_last[wv] = cand;
            __syncthreads();
            int32_t prev = __shfl_up(cand, 1, kWave);
            if (lane == 0) prev = wv == 0 ? carry_id : sh_last[wv - 1];
            const int32_t par = cand >= 0 ? cpar : -2;
            const bool ok = active && cand >= 0 && par == prev;
            const unsigned long long bad = ballot64(!ok);
            const int f = bad ? __ffsll((long long)bad) - 1 : kWave;
            const int rt = f < kWave ? __shfl((active && cand >= 0 && par != prev) ? 1 : 0, f, kWave) : 0;
            if (lane == 0) {
                sh_fail[wv] = f;
                sh_retry[wv] = rt;
            }
            __syncthreads();
            int fw = -1;
            for (int i = 0; i < W; ++i)
                if (sh_fail[i] < kWave) {
                    fw = i;
                    break;
                }
            const int fl = fw >= 0 ? sh_fail[fw] : kWave;
            const bool again = fw >= 0 && sh_retry[fw];
            if (fw >= 0) fail = fw * kWave + fl;
            __syncthreads();  // every wave has read the round's flags
            if (!again) break;
            // keys of two different prefixes collided: that lane looks
            // further along its probe sequence for the block with the
            // right parent, then the round is checked again
            if (wv == fw && lane == fl)
                cand = probe(ix, ik, (pos + 1) & ix.slot_mask, win, true, prev, &pos, &cpar,
                             &probes, &cmps);
        }
        const int rel = wv * kWave + lane;
        if (active) row[b] = rel < fail ? cand : -1;
        if (TOUCH && active && rel < fail) {
            const uint64_t fq = atomicAdd((unsigned long long*)&ix.freq[cand], 1ull) + 1ull;
            atomicMax((unsigned long long*)&ix.prio[cand], (unsigned long long)(clock + fq));
        }
        if (fail < W * kWave) {
            m = r0 + fail < n ? r0 + fail : n;
            r0 += W * kWave;
            break;
        }
        carry_key = sh_klast;
        carry_id = sh_last[W - 1];
        __syncthreads();  // sh_klast and sh_last read before the next round writes them
    }
    const int fill_from = r0 < n ? r0 : n;
    for (int b = fill_from + (int)threadIdx.x; b < bat.max_blocks; b += W * kWave) row[b] = -1;
    if (threadIdx.x == 0) m_out[r] = m;
    if (ix.counters) {
        CounterSlot* cs = counter_slot(ix.state);
        wave_count(&cs->probes, probes, lane);
        wave_count(&cs->token_compares, cmps, lane);
    }
}

// Chained keys of every whole block of every request (no probing).
template <int BT>
__global__ __launch_bounds__(kThreads) void k_hash_all(IndexView ix, Batch bat, uint64_t* __restrict__ keys) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r = (int64_t)blockIdx.x * kWavesPerGroup + (threadIdx.x / kWave);
    if (r >= bat.R) return;
    const int bt = BT ? BT : ix.block_tokens;
    const ChainConsts cc = chain_consts(ix.ht, lane);
    int64_t o0;
    // malformed requests were already counted by the lookup of the same batch
    int64_t a = bat.offsets[r], e = bat.offsets[r + 1];
    int32_t n = 0;
    o0 = 0;
    if (!(a < 0 || e < a || e > bat.n_tokens)) {
        o0 = a;
        int64_t nb = (e - a) / bt;
        n = (int32_t)(nb < bat.max_blocks ? nb : bat.max_blocks);
    }
    const int32_t* __restrict__ seq = bat.tokens + o0;
    __shared__ int4 sh_tok[BT == 16 ? kThreads * kQuads : 1];
    typename WindowOf<BT>::type win;
    win.init(sh_tok, threadIdx.x / kWave, lane);
    uint64_t carry = cc.root_key;
    for (int w0 = 0; w0 < n; w0 += kWave) {
        const int b = w0 + lane;
        win.stage(seq, w0, n, bt);
        const uint64_t c = b < n ? win.hash(cc.content_seed, bt) : 0;
        const uint64_t k = window_chain(c, carry, cc, lane);
        if (b < n) keys[r * bat.max_blocks + b] = k;
        carry = shfl_u64(k, kWave - 1);
    }
}

}  // namespace

namespace {
template <int W>
void launch_wide(const IndexView& ix, const Batch& b, int32_t* m, int32_t* ids, hipStream_t s) {
    const dim3 grid((unsigned)b.R), block(W * kWave);
    const bool touch = ix.freq != nullptr;
    if (ix.block_tokens == 16) {
        if (touch)
            hipLaunchKernelGGL((k_lookup_wide<16, true, W>), grid, block, 0, s, ix, b, m, ids);
        else
            hipLaunchKernelGGL((k_lookup_wide<16, false, W>), grid, block, 0, s, ix, b, m, ids);
    } else {
        if (touch)
            hipLaunchKernelGGL((k_lookup_wide<0, true, W>), grid, block, 0, s, ix, b, m, ids);
        else
            hipLaunchKernelGGL((k_lookup_wide<0, false, W>), grid, block, 0, s, ix, b, m, ids);
    }
}

}  // namespace

hipError_t launch_lookup(const IndexView& ix, const Batch& b, int32_t* m, int32_t* ids, hipStream_t s) {
    // requests of more than one window: a workgroup per request, windows in
    // parallel (4 waves up to 256 blocks, 8 up to 512, 16 beyond)
    if (b.max_blocks > kWave) {
        if (b.max_blocks <= 4 * kWave)
            launch_wide<4>(ix, b, m, ids, s);
        else if (b.max_blocks <= 8 * kWave)
            launch_wide<8>(ix, b, m, ids, s);
        else
            launch_wide<16>(ix, b, m, ids, s);
        return hipGetLastError();
    }
    const unsigned grid = (unsigned)((b.R + kWavesPerGroup - 1) / kWavesPerGroup);
    const bool touch = ix.freq != nullptr;
    if (ix.block_tokens == 16) {
        if (touch)
            hipLaunchKernelGGL((k_lookup<16, true>), dim3(grid), dim3(kThreads), 0, s, ix, b, m, ids);
        else
            hipLaunchKernelGGL((k_lookup<16, false>), dim3(grid), dim3(kThreads), 0, s, ix, b, m, ids);
    } else {
        if (touch)
            hipLaunchKernelGGL((k_lookup<0, true>), dim3(grid), dim3(kThreads), 0, s, ix, b, m, ids);
        else
            hipLaunchKernelGGL((k_lookup<0, false>), dim3(grid), dim3(kThreads), 0, s, ix, b, m, ids);
    }
    return hipGetLastError();
}

hipError_t launch_hash_all(const IndexView& ix, const Batch& b, uint64_t* keys, hipStream_t s) {
    const unsigned grid = (unsigned)((b.R + kWavesPerGroup - 1) / kWavesPerGroup);
    if (ix.block_tokens == 16)
        hipLaunchKernelGGL(k_hash_all<16>, dim3(grid), dim3(kThreads), 0, s, ix, b, keys);
    else
        hipLaunchKernelGGL(k_hash_all<0>, dim3(grid), dim3(kThreads), 0, s, ix, b, keys);
    return hipGetLastError();
}

}  // namespace ptsd
