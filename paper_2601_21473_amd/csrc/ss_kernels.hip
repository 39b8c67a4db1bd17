// Device kernels of the invocation-distance memory manager for gfx950.
//
// Plan (per step, Section 3.3 of the paper and its Appendix A interface):
//   classification  one pass over the agents: distance of active agents
//                forced to 0, 64-bit priority keys (d, id), classification
//                into evictable residents / demand loads / prefetch
//                candidates, stream compaction of each class (wave64 ballot
//                + mbcnt ranks, one DPP scan per list over the waves' counts),
//                and the unit sums the plan needs;
//   plan core    one workgroup of 1024 threads: the distance-histogram
//                cuts of the evictable and candidate sets that can take part
//                in the plan, one register/LDS merge sort of both (and of the
//                demand loads), prefix sums, the prefetch acceptance rule in
//                closed form, the victim count, and the plan written to a
//                mapped host mirror, published by a sequence number written
//                last; then the pick of the pre-step free units.
//   k_plan_core      the plan core, classifying the agents itself
//                    (N <= kFuseAgents = 12,288);
//   k_classify_core  classification over N / 4096 workgroups, the last of
//                    which runs the plan core (larger N), in one launch.
//   Either way the core's workgroup updates the block table (release of the
//   victims' units, assignment of the loads' units) after publishing the plan.
// Data movement:
//   k_copy<pack>  gathers (pack) or scatters (unpack) whole units between the
//                pool's planes and a contiguous staging slot, one wave per
//                piece of at most 32 KiB moved as one burst of 16-byte
//                non-temporal accesses;
//   k_duplex     both directions of a small step in one launch, straight
//                between the pool's units and the pinned host copies.
//
// Nothing here is a dense contraction; all work is integer indexing and byte
// movement, so there is no MFMA.
#include "ss_internal.h"

namespace ss {

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ unsigned lane_id() { return __lane_id(); }

// Lane 0's value in every lane (a scalar read: every caller has all lanes
// active, so lane 0 is the first active lane).
__device__ __forceinline__ unsigned lane0(unsigned v) {
    return (unsigned)__builtin_amdgcn_readfirstlane((int)v);
}

__device__ __forceinline__ unsigned mbcnt(u64 mask) {
    return __builtin_amdgcn_mbcnt_hi((unsigned)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((unsigned)mask, 0u));
}

// Value of lane (lane ^ jl) for jl in {1, 2, 4, 8, 16, 32}, without LDS: DPP
// quad permutes (1, 2), row rotates (4: by 4 or 12 depending on the lane, 8)
// and the permlane swaps of 16- and 32-lane halves.
__device__ __forceinline__ unsigned lane_xor32(unsigned x, unsigned jl) {
    const unsigned l = lane_id();
    switch (jl) {
    case 1: return __builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false);     // quad_perm 1,0,3,2
    case 2: return __builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false);     // quad_perm 2,3,0,1
    case 4: {
        const unsigned dn = __builtin_amdgcn_mov_dpp(x, 0x124, 0xF, 0xF, false);   // row_ror:4
        const unsigned up = __builtin_amdgcn_mov_dpp(x, 0x12C, 0xF, 0xF, false);   // row_ror:12
        return (l & 4) ? dn : up;
    }
    case 8: return __builtin_amdgcn_mov_dpp(x, 0x128, 0xF, 0xF, false);    // row_ror:8
    case 16: {
        const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
        return (l & 16) ? r[0] : r[1];
    }
    default: {
        const auto q = __builtin_amdgcn_permlane32_swap(x, x, false, false);
        return (l & 32) ? q[0] : q[1];
    }
    }
}

__device__ __forceinline__ u64 lane_xor64(u64 v, unsigned jl) {
    return ((u64)lane_xor32((unsigned)(v >> 32), jl) << 32) | lane_xor32((unsigned)v, jl);
}

// Sum over the wave, in every lane (butterfly over lane_xor64).
__device__ __forceinline__ u64 wave_sum(u64 v) {
#pragma unroll
    for (unsigned o = 32; o > 0; o >>= 1) v += lane_xor64(v, o);
    return v;
}

// v of the lane `ctrl` selects (DPP row shift or row broadcast), 0 in lanes
// the move does not reach and in rows outside row_mask.
template <int ctrl, int row_mask>
__device__ __forceinline__ u64 dpp_move64(u64 v) {
    const unsigned lo = __builtin_amdgcn_update_dpp(0u, (unsigned)v, ctrl, row_mask, 0xF, false);
    const unsigned hi = __builtin_amdgcn_update_dpp(0u, (unsigned)(v >> 32), ctrl, row_mask, 0xF,
                                                    false);
    return ((u64)hi << 32) | lo;
}

// Inclusive scan over the wave (all lanes active): row-wise by DPP row shifts
// of 1, 2, 4 and 8 lanes, then row 0's total into row 1 and row 2's into row 3
// (row_bcast:15), then the first two rows' total into rows 2 and 3
// (row_bcast:31).  No LDS.
__device__ __forceinline__ u64 wave_incl_scan(u64 v) {
    v += dpp_move64<0x111, 0xF>(v);                  // row_shr:1
    v += dpp_move64<0x112, 0xF>(v);                  // row_shr:2
    v += dpp_move64<0x114, 0xF>(v);                  // row_shr:4
    v += dpp_move64<0x118, 0xF>(v);                  // row_shr:8
    v += dpp_move64<0x142, 0xA>(v);                  // row_bcast:15 into rows 1 and 3
    v += dpp_move64<0x143, 0xC>(v);                  // row_bcast:31 into rows 2 and 3
    return v;
}

// ---------------------------------------------------------------------------
// classification
// ---------------------------------------------------------------------------

// Agents classified per thread and pass: the loads of all of them are issued
// before any is used, so each thread has that many agents' reads in flight.
constexpr unsigned kClassBatch = 4;

// The inputs of agents first + u * kCoreThreads (u < kClassBatch) below end.
struct AgentBatch {
    unsigned D[kClassBatch], s[kClassBatch];
    unsigned char act[kClassBatch], res[kClassBatch];
};

__device__ __forceinline__ void load_agents(const PlanArgs& A, unsigned first, unsigned end,
                                            AgentBatch& b) {
#pragma unroll
    for (unsigned u = 0; u < kClassBatch; ++u) {
        const unsigned a = first + u * kCoreThreads;
        const bool v = a < end;
        b.D[u] = v ? A.dist[a] : 0u;
        b.act[u] = v ? A.active[a] : (unsigned char)0;
        b.res[u] = v ? A.resident[a] : (unsigned char)0;
        b.s[u] = v ? A.units[a] : 0u;
    }
}

// Class of agent a: its key (distance 0 when active, then the id), its
// membership of the evictable residents E, the demand loads L and the
// prefetch candidates C (distance below the threshold), the distance bucket
// of an inactive agent and a candidate's sub-list.
struct AgentClass {
    u64 key;
    bool isE, isL, isC;
    unsigned bucket, kl;
};

__device__ __forceinline__ AgentClass classify(const PlanArgs& A, unsigned a, bool valid,
                                               unsigned D, bool act, bool res) {
    AgentClass c;
    const u64 d = act ? 0ull : (u64)D;
    c.key = (d << A.idbits) | a;
    c.isE = valid && res && !act;
    c.isL = valid && act && !res;
    c.isC = valid && !res && !act && D < A.threshold;
    c.bucket = dist_bucket(D);
    c.kl = cand_list(c.bucket);
    return c;
}

// Per-thread unit sums of the classes, added to the block's counters once.
struct ClassSums {
    u64 act = 0, res = 0, dem = 0, evi = 0, can = 0;
    __device__ void add(const AgentClass& c, bool act_, bool res_, u64 s) {
        act += act_ ? s : 0;
        res += res_ ? s : 0;
        dem += c.isL ? s : 0;
        evi += c.isE ? s : 0;
        can += c.isC ? s : 0;
    }
};

// Block-local slot of this lane in a list (one LDS atomic per wave).
__device__ __forceinline__ unsigned wave_reserve(bool pred, unsigned* counter) {
    const u64 mask = __ballot(pred);
    if (mask == 0) return 0;                         // wave-uniform
    unsigned base = 0;
    if (lane_id() == 0) base = atomicAdd(counter, (unsigned)__popcll(mask));
    return lane0(base) + mbcnt(mask);
}

// List ids of the classification: the candidate sub-lists 0 .. kCandLists-1,
// then the evictable residents E and the demand loads L (an agent is in at
// most one of them).
constexpr unsigned kListE = kCandLists, kListL = kCandLists + 1, kLists = kCandLists + 2;
constexpr unsigned kNoList = 0xFFu;
// Counts of one pass (kClassBatch agents per thread): one per wave, agent
// slot and list; a list's counts fill one wave, which scans them.
constexpr unsigned kPassSlots = (kCoreThreads / 64) * kClassBatch;
static_assert(kPassSlots == 64, "one wave scans a list's counts");
constexpr unsigned kPassTab = kLists * kPassSlots;     // u32 entries per pass table

__device__ __forceinline__ unsigned list_of(const AgentClass& c) {
    return c.isC ? c.kl : c.isE ? kListE : c.isL ? kListL : kNoList;
}

__device__ __forceinline__ unsigned* list_counter(PlanCounters* c, unsigned k) {
    return k < kCandLists ? &c->n_C[k] : k == kListE ? &c->n_E : &c->n_L;
}

__device__ __forceinline__ u64* list_ptr(const PlanArgs& A, unsigned k) {
    return k < kCandLists ? A.listC + (u64)k * A.n : k == kListE ? A.listE : A.listL;
}

// Slots of one pass's agents in their lists (the whole workgroup, one agent
// per thread and u).  No atomic sits in the waves' path: each wave ranks its
// lanes within their lists (ballots, mbcnt) and stores its per-list counts
// in tab[list][wave, u]; after a barrier wave k scans list k's 64 counts (DPP)
// and adds the list's base, which is this workgroup's running count of the
// list (kGlobal false) or the range that one device-wide atomic reserves for
// the workgroup's whole list (kGlobal true: one pass per workgroup); after a
// second barrier every agent's slot is its table entry plus its rank.  Slots
// follow (wave, u, lane) order within a pass.  Callers alternate between two
// tables on consecutive passes, so a pass never overwrites a table that a
// thread of the previous pass has still to read.
template <bool kGlobal>
__device__ __forceinline__ void reserve_pass(const unsigned (&lst)[kClassBatch],
                                             unsigned (&slot)[kClassBatch], unsigned* tab,
                                             PlanCounters* local, PlanCounters* global) {
    const unsigned w = threadIdx.x >> 6, l = lane_id();
    static_assert(kLists <= 15, "list ids and kNoList's low bits fit four bits");
    unsigned rank[kClassBatch];
#pragma unroll
    for (unsigned u = 0; u < kClassBatch; ++u) {
        // The first two lists of the wave by one ballot each (in a single
        // workgroup's classification most waves hold one or two); if lanes
        // remain, a multi-split by the four bits of the list id: four
        // ballots, then the lanes of list k are those whose bits match k's.
        // The many-workgroup classification (large agent counts, whose waves
        // mostly hold three or more lists) goes to the multi-split directly.
        // Selects throughout, no branches per lane.
        const u64 valid = __ballot(lst[u] != kNoList);
        u64 rest = valid;
        unsigned r = 0, k0 = kNoList, k1 = kNoList, c0 = 0, c1 = 0;
        if (!kGlobal && rest) {                      // wave-uniform
            k0 = (unsigned)__builtin_amdgcn_readlane((int)lst[u], (int)__builtin_ctzll(rest));
            const u64 m = __ballot(lst[u] == k0);
            r = lst[u] == k0 ? mbcnt(m) : r;
            c0 = (unsigned)__popcll(m);
            rest &= ~m;
        }
        if (!kGlobal && rest) {
            k1 = (unsigned)__builtin_amdgcn_readlane((int)lst[u], (int)__builtin_ctzll(rest));
            const u64 m = __ballot(lst[u] == k1);
            r = lst[u] == k1 ? mbcnt(m) : r;
            c1 = (unsigned)__popcll(m);
            rest &= ~m;
        }
        unsigned cnt = l == k0 ? c0 : l == k1 ? c1 : 0u;
        if (rest) {
            const u64 m0 = __ballot(lst[u] & 1u), m1 = __ballot(lst[u] & 2u);
            const u64 m2 = __ballot(lst[u] & 4u), m3 = __ballot(lst[u] & 8u);
            auto lanes_of = [&](unsigned k) {
                return valid & ((k & 1u) ? m0 : ~m0) & ((k & 2u) ? m1 : ~m1) &
                       ((k & 4u) ? m2 : ~m2) & ((k & 8u) ? m3 : ~m3);
            };
            r = mbcnt(lanes_of(lst[u]));
            cnt = (unsigned)__popcll(lanes_of(l));
        }
        rank[u] = r;
        if (l < kLists) tab[l * kPassSlots + w * kClassBatch + u] = cnt;
    }
    __syncthreads();
    if (w < kLists) {                                // wave-uniform
        const unsigned v = tab[w * kPassSlots + l];
        const unsigned incl = (unsigned)wave_incl_scan((u64)v);
        const unsigned total = (unsigned)__builtin_amdgcn_readlane((int)incl, 63);
        unsigned base;
        if (kGlobal) {
            unsigned b = 0;
            if (l == 0 && total) b = atomicAdd(list_counter(global, w), total);
            base = lane0(b);
        } else {
            unsigned* ctr = list_counter(local, w);
            base = *ctr;                             // only this wave touches list w
            if (l == 0) *ctr = base + total;
        }
        tab[w * kPassSlots + l] = base + incl - v;
    }
    __syncthreads();
#pragma unroll
    for (unsigned u = 0; u < kClassBatch; ++u)
        slot[u] = lst[u] == kNoList ? 0u : tab[lst[u] * kPassSlots + w * kClassBatch + u] + rank[u];
}

// Add every thread's sums to the block counters *cnt (LDS): one reduction per
// wave and sum, one LDS atomic per wave.
__device__ __forceinline__ void flush_sums(const ClassSums& t, PlanCounters* cnt) {
    const u64 s_act = wave_sum(t.act);
    const u64 s_res = wave_sum(t.res);
    const u64 s_dem = wave_sum(t.dem);
    const u64 s_evi = wave_sum(t.evi);
    const u64 s_can = wave_sum(t.can);
    if (lane_id() == 0) {
        if (s_act) atomicAdd(&cnt->sum_active, s_act);
        if (s_res) atomicAdd(&cnt->sum_resident, s_res);
        if (s_dem) atomicAdd(&cnt->sum_demand, s_dem);
        if (s_evi) atomicAdd(&cnt->sum_evictable, s_evi);
        if (s_can) atomicAdd(&cnt->sum_cand, s_can);
    }
}

// ---------------------------------------------------------------------------
// k_plan_core helpers (blockDim.x == kCoreThreads)
// ---------------------------------------------------------------------------

struct CoreShared {
    u64 histw[kDistBuckets];        // candidate units per distance bucket (this workgroup)
    PlanCounters cnt;               // this workgroup's classification
    u64 wsum[kCoreThreads / 64 + 1];
    u64 scal[8];
    unsigned uscal[8];
};

// Exclusive block scan of one value per thread; returns the prefix and sets
// *total (same on every thread).
__device__ __forceinline__ u64 block_excl_scan(u64 v, CoreShared& S, u64* total) {
    const unsigned w = threadIdx.x >> 6, l = lane_id();
    const unsigned nw = blockDim.x >> 6;
    const u64 inc = wave_incl_scan(v);
    if (l == 63) S.wsum[w] = inc;
    __syncthreads();
    if (w == 0) {
        u64 x = (l < nw) ? S.wsum[l] : 0;
        u64 xi = wave_incl_scan(x);
        if (l < nw) S.wsum[l] = xi - x;
        if (l == nw - 1) S.wsum[nw] = xi;
    }
    __syncthreads();
    const u64 r = inc - v + S.wsum[w];
    *total = S.wsum[nw];
    __syncthreads();
    return r;
}

// out(i, f(0) + ... + f(i)) for i < n: the inclusive prefix of every element.
// Lists longer than the block: each thread takes kPrefixRun consecutive
// elements per round, so the f(i) of a round (often gathers) are in flight
// together and a block scan covers 4096 elements (shorter lists keep one
// element per thread: fewer instructions when most threads would idle).
constexpr unsigned kPrefixRun = 4;
template <class F, class Out>
__device__ __forceinline__ void block_prefix_to(unsigned n, F f, Out out, CoreShared& S) {
    u64 carry = 0;
    if (n <= blockDim.x) {
        const unsigned i = threadIdx.x;
        const u64 v = (i < n) ? f(i) : 0;
        u64 tot;
        const u64 ex = block_excl_scan(v, S, &tot);
        if (i < n) out(i, ex + v);
        __syncthreads();
        return;
    }
    for (unsigned base = 0; base < n; base += kPrefixRun * blockDim.x) {
        const unsigned i0 = base + threadIdx.x * kPrefixRun;
        u64 v[kPrefixRun];
        u64 sum = 0;
#pragma unroll
        for (unsigned u = 0; u < kPrefixRun; ++u) v[u] = (i0 + u < n) ? f(i0 + u) : 0;
#pragma unroll
        for (unsigned u = 0; u < kPrefixRun; ++u) sum += v[u];
        u64 tot;
        u64 run = carry + block_excl_scan(sum, S, &tot);
#pragma unroll
        for (unsigned u = 0; u < kPrefixRun; ++u) {
            run += v[u];
            if (i0 + u < n) out(i0 + u, run);
        }
        carry += tot;
    }
    __syncthreads();
}

// out[0] = 0, out[i+1] = out[i] + f(i) for i < n.
template <class F>
__device__ __forceinline__ void block_prefix(unsigned n, F f, u64* out, CoreShared& S) {
    if (threadIdx.x == 0) out[0] = 0;
    block_prefix_to(n, f, [&](unsigned i, u64 v) { out[i + 1] = v; }, S);
}

// Keys src[i] (i < n) with keep(key) appended to buf[*counter ...] (slots at
// or beyond cap are counted but not written), each stored or'ed with tag.
// Each thread loads kGatherLoads keys per round, and the next round's loads
// are issued before this round's keys are placed; each wave reserves the
// slots of a whole round with one LDS atomic.  The order of the appended keys
// is arbitrary.
constexpr unsigned kGatherLoads = 8;
template <class Keep>
__device__ __forceinline__ void gather_keys(const u64* src, unsigned n, Keep keep, u64* buf,
                                            unsigned cap, unsigned* counter, u64 tag = 0) {
    if (n <= blockDim.x) {
        const unsigned i = threadIdx.x;
        const u64 k = i < n ? src[i] : ~0ull;
        const bool take = k != ~0ull && keep(k);
        const unsigned pos = wave_reserve(take, counter);
        if (take && pos < cap) buf[pos] = k | tag;
        return;
    }
    const unsigned step = kGatherLoads * blockDim.x;
    u64 k[kGatherLoads];
#pragma unroll
    for (unsigned u = 0; u < kGatherLoads; ++u) {
        const unsigned i = u * blockDim.x + threadIdx.x;
        k[u] = i < n ? src[i] : ~0ull;
    }
    for (unsigned i0 = 0; i0 < n; i0 += step) {
        u64 kn[kGatherLoads];
#pragma unroll
        for (unsigned u = 0; u < kGatherLoads; ++u) {
            const unsigned i = i0 + step + u * blockDim.x + threadIdx.x;
            kn[u] = i < n ? src[i] : ~0ull;
        }
        u64 mask[kGatherLoads];
        unsigned total = 0;
#pragma unroll
        for (unsigned u = 0; u < kGatherLoads; ++u) {
            mask[u] = __ballot(k[u] != ~0ull && keep(k[u]));
            total += (unsigned)__popcll(mask[u]);
        }
        if (total) {                                 // wave-uniform
            unsigned off = 0;
            if (lane_id() == 0) off = atomicAdd(counter, total);
            off = lane0(off);
#pragma unroll
            for (unsigned u = 0; u < kGatherLoads; ++u) {
                const unsigned pos = off + mbcnt(mask[u]);
                if (((mask[u] >> lane_id()) & 1) && pos < cap) buf[pos] = k[u] | tag;
                off += (unsigned)__popcll(mask[u]);
            }
        }
#pragma unroll
        for (unsigned u = 0; u < kGatherLoads; ++u) k[u] = kn[u];
    }
}

// buf[0..n) = src[0..n), kGatherLoads loads per thread and round, the next
// round's loads issued before this round's stores.
__device__ __forceinline__ void copy_keys(const u64* src, unsigned n, u64* buf) {
    if (n <= blockDim.x) {
        if (threadIdx.x < n) buf[threadIdx.x] = src[threadIdx.x];
        return;
    }
    const unsigned step = kGatherLoads * blockDim.x;
    u64 k[kGatherLoads];
#pragma unroll
    for (unsigned u = 0; u < kGatherLoads; ++u) {
        const unsigned i = u * blockDim.x + threadIdx.x;
        if (i < n) k[u] = src[i];
    }
    for (unsigned i0 = 0; i0 < n; i0 += step) {
        u64 kn[kGatherLoads];
#pragma unroll
        for (unsigned u = 0; u < kGatherLoads; ++u) {
            const unsigned i = i0 + step + u * blockDim.x + threadIdx.x;
            if (i < n) kn[u] = src[i];
        }
#pragma unroll
        for (unsigned u = 0; u < kGatherLoads; ++u) {
            const unsigned i = i0 + u * blockDim.x + threadIdx.x;
            if (i < n) buf[i] = k[u];
        }
#pragma unroll
        for (unsigned u = 0; u < kGatherLoads; ++u) k[u] = kn[u];
    }
}

__device__ __forceinline__ unsigned pow2ceil(unsigned n) {
    unsigned p = 1;
    while (p < n) p <<= 1;
    return p;
}

// Ascending bitonic sort of buf[0..npad), npad a power of two.  buf is LDS or
// (for lists larger than the LDS budget) global memory private to this block.
__device__ void bitonic_asc(u64* buf, unsigned npad) {
    for (unsigned k = 2; k <= npad; k <<= 1) {
        for (unsigned j = k >> 1; j > 0; j >>= 1) {
            for (unsigned t = threadIdx.x; t < (npad >> 1); t += blockDim.x) {
                const unsigned i = ((t & ~(j - 1)) << 1) | (t & (j - 1));
                const unsigned p = i | j;
                const u64 a = buf[i], b = buf[p];
                const bool asc = (i & k) == 0;
                if ((a > b) == asc) {
                    buf[i] = b;
                    buf[p] = a;
                }
            }
            __syncthreads();
        }
    }
}

// Largest list sorted in LDS: 1024 threads with up to kRegKeys keys each.
constexpr unsigned kRegKeys = 8;

// Ascending sort of lds[0..npad), npad a power of two <= 1024 * kE, by a
// 1024-thread block, using lds[npad..2 npad) as scratch.
//
// Register stage: each wave sorts a run of 64 * kE keys, lane l holding the
// kE consecutive keys from l * kE, by a bitonic network (Batcher 1968):
// exchanges between keys of one lane are register moves, exchanges between
// lanes go through lane_xor64 (no LDS, no barrier); waves that hold only
// padding skip it.  Merge stage: runs are merged pairwise, one barrier per
// round, by merge path (Green, McColl and Bader 2012): thread t writes the kE
// consecutive outputs from t * kE; one binary search over the diagonal of its
// run pair finds how many of the outputs before it come from the left run,
// then it merges its kE outputs sequentially with the two run heads in
// registers.  Ties take the left run first, so the padding keys (all equal)
// keep a consistent order.  Only the first n keys are real (n <= npad): when
// lds[n..npad) and lds[npad + n..2 npad) hold padding, every round's outputs
// from n on are padding too (the real keys of a pair of runs precede its
// padding, and only the pair holding key n - 1 has both), so the waves and
// threads whose keys or outputs all lie there do nothing.
template <unsigned kE>
__device__ __forceinline__ void merge_sort_lds_e(u64* lds, unsigned npad, unsigned n) {
    constexpr unsigned W = 64 * kE;                  // keys per wave run
    const unsigned t = threadIdx.x, l = lane_id();
    const unsigned base = (t >> 6) * W;
    if (base < n) {                                  // wave-uniform: the wave holds real keys
        u64 x[kE];
#pragma unroll
        for (unsigned r = 0; r < kE; ++r) {
            const unsigned i = base + l * kE + r;
            x[r] = i < npad ? lds[i] : ~0ull;
        }
#pragma unroll
        for (unsigned k = 2; k <= W; k <<= 1) {
#pragma unroll
            for (unsigned j = k >> 1; j > 0; j >>= 1) {
                if (j < kE) {                        // partner in the same lane
#pragma unroll
                    for (unsigned r = 0; r < kE; ++r) {
                        if (r & j) continue;
                        const bool up = ((l * kE + r) & k) == 0;
                        const u64 a = x[r], b = x[r | j];
                        const bool sw = (a > b) == up;
                        x[r] = sw ? b : a;
                        x[r | j] = sw ? a : b;
                    }
                } else {                             // partner in lane l ^ (j / kE)
                    const unsigned i = l * kE;
                    const bool keep_min = ((i & j) == 0) == ((i & k) == 0);
#pragma unroll
                    for (unsigned r = 0; r < kE; ++r) {
                        const u64 p = lane_xor64(x[r], j / kE);
                        const bool take = (p < x[r]) == keep_min;
                        x[r] = take ? p : x[r];
                    }
                }
            }
        }
#pragma unroll
        for (unsigned r = 0; r < kE; ++r) {
            const unsigned i = base + l * kE + r;
            if (i < npad) lds[i] = x[r];
        }
    }
    __syncthreads();
    u64* src = lds;
    u64* dst = lds + npad;
    for (unsigned L = W; L < npad; L <<= 1) {
        const unsigned o = t * kE;                   // first output of this thread
        if (o < n) {
            const unsigned b0 = o & ~(2 * L - 1);
            const unsigned d = o - b0;               // outputs of the pair before o
            const u64* A = src + b0;
            const u64* B = src + b0 + L;
            unsigned lo = d > L ? d - L : 0, hi = d < L ? d : L;
            while (lo < hi) {
                const unsigned mid = (lo + hi) >> 1;
                if (A[mid] <= B[d - 1 - mid]) lo = mid + 1; else hi = mid;
            }
            unsigned i = lo, j = d - lo;
            u64 a = i < L ? A[i] : ~0ull, b = j < L ? B[j] : ~0ull;
#pragma unroll
            for (unsigned k = 0; k < kE; ++k) {
                const bool takeA = j >= L || (i < L && a <= b);
                dst[o + k] = takeA ? a : b;
                if (takeA) {
                    ++i;
                    a = i < L ? A[i] : ~0ull;
                } else {
                    ++j;
                    b = j < L ? B[j] : ~0ull;
                }
            }
        }
        __syncthreads();
        u64* tmp = src;
        src = dst;
        dst = tmp;
    }
    if (src != lds) {
        for (unsigned i = t; i < n; i += blockDim.x) lds[i] = src[i];
        __syncthreads();
    }
}

// Keys per lane by list size (measured on one 1024-thread workgroup: longer
// register runs save merge rounds until the register stage's exchanges cost
// more than the rounds they save).  Inlined wherever a plan sorts (its LDS
// accesses then stay LDS instructions, and the plan kernels make no calls: a
// call would give them a stack in scratch memory for the callee's saved
// registers, and a longer register allocation).
__device__ __forceinline__ void merge_sort_lds_inl(u64* lds, unsigned npad, unsigned n) {
    if (npad <= 512) merge_sort_lds_e<1>(lds, npad, n);
    else if (npad <= 2048) merge_sort_lds_e<2>(lds, npad, n);
    else if (npad == 4096) merge_sort_lds_e<4>(lds, npad, n);
    else merge_sort_lds_e<8>(lds, npad, n);
}

// (all npad keys treated as real: the callers pad only the first half)
__device__ __forceinline__ void merge_sort_lds(u64* lds, unsigned npad) {
    merge_sort_lds_inl(lds, npad, npad);
}

// The keys that gather(buf, cap, counter) appends (its calls of gather_keys
// with one LDS counter), sorted ascending into dst[0..m); returns m.  They are
// gathered into LDS and sorted there when they fit; otherwise they are
// gathered again, into dst (room for pow2ceil(N) keys), and sorted there.
template <class Gather>
__device__ __forceinline__ unsigned gather_sorted(Gather gather, u64* dst, u64* lds, CoreShared& S) {
    if (threadIdx.x == 0) S.uscal[7] = 0;
    __syncthreads();
    gather(lds, (unsigned)kLdsKeys, &S.uscal[7]);
    __syncthreads();
    const unsigned m = S.uscal[7];
    __syncthreads();                                 // every thread has m before the reuse below
    if (m == 0) return 0;
    const unsigned npad = pow2ceil(m);
    u64* buf = lds;
    if (m > (unsigned)kLdsKeys) {
        if (threadIdx.x == 0) S.uscal[7] = 0;
        __syncthreads();
        gather(dst, m, &S.uscal[7]);
        buf = dst;
        __syncthreads();
    }
    for (unsigned i = m + threadIdx.x; i < npad; i += blockDim.x) buf[i] = ~0ull;
    __syncthreads();
    if (buf == lds && npad <= 1024 * kRegKeys) merge_sort_lds(lds, npad);
    else bitonic_asc(buf, npad);
    if (buf == lds) {
        for (unsigned i = threadIdx.x; i < m; i += blockDim.x) dst[i] = lds[i];
        __syncthreads();
    }
    return m;
}

// Sort the keys src[i] < kstar (there are exactly m of them) ascending into
// dst[0..m).  dst has room for pow2ceil(N) keys and doubles as the sort buffer
// when m exceeds the LDS budget.
__device__ __forceinline__ void select_sort(const u64* src, unsigned n_src, u64 kstar, unsigned m,
                                            u64* dst, u64* lds, CoreShared& S) {
    if (m == 0) return;
    const unsigned npad = pow2ceil(m);
    u64* buf = (npad <= (unsigned)kLdsKeys) ? lds : dst;
    if (threadIdx.x == 0) S.uscal[7] = 0;
    __syncthreads();
    if (kstar == ~0ull) copy_keys(src, n_src, buf);
    else gather_keys(src, n_src, [&](u64 k) { return k < kstar; }, buf, m, &S.uscal[7]);
    for (unsigned i = m + threadIdx.x; i < npad; i += blockDim.x) buf[i] = ~0ull;
    __syncthreads();
    if (npad <= 1024 * kRegKeys) merge_sort_lds(lds, npad);
    else bitonic_asc(buf, npad);
    if (buf == lds) {
        for (unsigned i = threadIdx.x; i < m; i += blockDim.x) dst[i] = lds[i];
        __syncthreads();
    }
}

// Occupancy words per thread that the free-unit scan holds in registers
// (pools of up to 1024 * 16 * 32 = 524,288 units; larger pools loop).
constexpr unsigned kOccRegs = 16;

// The plan's first n_free_used free units in ascending order into free_old,
// each marked in use in the occupancy bitmap (thread t owns words
// [t * per, (t + 1) * per), per <= kR: all of them are loaded at once).
template <unsigned kR>
__device__ __forceinline__ void free_scan_regs(const PlanArgs& A, u64 n_free_used, unsigned per,
                                               CoreShared& S) {
    const unsigned w0 = threadIdx.x * per;
    unsigned word[kR];
#pragma unroll
    for (unsigned k = 0; k < kR; ++k) word[k] = k < per && w0 + k < A.occ_words ? A.occ[w0 + k] : ~0u;
    u64 cnt = 0;
#pragma unroll
    for (unsigned k = 0; k < kR; ++k) cnt += __popc(~word[k]);
    u64 tot;
    u64 pos = block_excl_scan(cnt, S, &tot);
#pragma unroll
    for (unsigned k = 0; k < kR; ++k) {
        unsigned bits = ~word[k], used = 0;
        while (bits && pos < n_free_used) {
            const unsigned b = __ffs(bits) - 1;
            bits &= bits - 1;
            used |= 1u << b;
            A.free_old[pos++] = (int)((w0 + k) * 32u + b);
        }
        if (used) A.occ[w0 + k] = word[k] | used;
    }
}

// The three key sets a plan sorts (evictable residents T, demand loads L,
// candidates C) as one array: a tag above the key bits makes T sort first,
// then L, then C, so one merge sort replaces three (each sort's rounds are
// barrier- and latency-bound on one workgroup, so three small sorts cost
// about three times one sort of their union).  Keys are below
// 2^(32 + idbits), so the tags fit when idbits <= kTagShift - 32.
constexpr unsigned kTagShift = 62;
constexpr u64 kTagL = 1ull << kTagShift, kTagC = 2ull << kTagShift;
constexpr u64 kKeyBits = kTagL - 1;
constexpr unsigned kJointKeys = 1024 * kRegKeys;   // largest joint sort (LDS: twice this)
static_assert(2 * kJointKeys <= (unsigned)kLdsKeys, "joint sort and its merge scratch fit");

// Sorts lds[0..n) (tagged keys) and writes each set, untagged and ascending,
// to its array: sortE[0..nT), sortL[0..nL), sortC[0..n - nT - nL).
__device__ __forceinline__ void joint_sort_out(u64* lds, unsigned n, unsigned nT, unsigned nL,
                                               u64* sortE, u64* sortL, u64* sortC) {
    if (n == 0) return;
    const unsigned npad = pow2ceil(n);
    for (unsigned i = n + threadIdx.x; i < npad; i += kCoreThreads) {
        lds[i] = ~0ull;                              // padding, and the same range of
        lds[npad + i] = ~0ull;                       // the merge rounds' second buffer
    }
    __syncthreads();
    merge_sort_lds_inl(lds, npad, n);
    for (unsigned i = threadIdx.x; i < n; i += kCoreThreads) {
        const u64 k = lds[i] & kKeyBits;
        u64* dst = i < nT ? sortE + i : i < nT + nL ? sortL + (i - nT) : sortC + (i - nT - nL);
        *dst = k;
    }
    __syncthreads();
}

// ---------------------------------------------------------------------------
// k_plan_core
// ---------------------------------------------------------------------------

// Classification of all agents by the plan core's workgroup: candidate units
// into the LDS histogram S.histw, evictable residents' units into the LDS
// histogram `he`, counts and sums into S.cnt, list entries at the slots
// reserve_pass gives them (tab: two pass tables in LDS).
__device__ __forceinline__ void classify_fused(const PlanArgs& A, CoreShared& S, unsigned* he,
                                               unsigned* tab) {
    ClassSums t;
    constexpr unsigned step = kClassBatch * kCoreThreads;
    AgentBatch b;
    load_agents(A, threadIdx.x, A.n, b);
    unsigned pass = 0;
    for (unsigned base = 0; base < A.n; base += step, ++pass) {
        AgentBatch nb;                               // next pass's loads in flight
        load_agents(A, base + step + threadIdx.x, A.n, nb);
        u64 key[kClassBatch];
        unsigned lst[kClassBatch], slot[kClassBatch];
#pragma unroll
        for (unsigned u = 0; u < kClassBatch; ++u) {
            const unsigned a = base + u * kCoreThreads + threadIdx.x;
            const AgentClass c = classify(A, a, a < A.n, b.D[u], b.act[u] != 0, b.res[u] != 0);
            if (c.isC) atomicAdd(&S.histw[c.bucket], (u64)b.s[u]);
            if (c.isE) atomicAdd(&he[c.bucket], b.s[u]);
            key[u] = c.key;
            lst[u] = list_of(c);
            t.add(c, b.act[u] != 0, b.res[u] != 0, b.s[u]);
        }
        reserve_pass<false>(lst, slot, tab + (pass & 1) * kPassTab, &S.cnt, nullptr);
#pragma unroll
        for (unsigned u = 0; u < kClassBatch; ++u)
            if (lst[u] != kNoList) list_ptr(A, lst[u])[slot[u]] = key[u];
        b = nb;
    }
    flush_sums(t, &S.cnt);
}

// Items (victims or loads) of the block-table update handled together: every
// lane loads its entries of all of them before it stores any, so a group
// costs one memory round trip per 64 of its logical units.
constexpr unsigned kBtGroup = 4;

// Release the units of a group of victims (block-table row base[g], s[g]
// units, eviction-order offset o[g], written back w[g] at offset ow[g], host
// copy at hoff[g]); lanes take logical units j: record each unit in eviction
// order for the loads (and, for a victim that is written back, for the pack)
// and clear its block-table entry.  (Occupancy bits: see bt_update_block.)
__device__ __forceinline__ void bt_release_group(const BtArgs& B, const u64 (&base)[kBtGroup],
                                                 const unsigned (&s)[kBtGroup],
                                                 const u64 (&o)[kBtGroup],
                                                 const bool (&w)[kBtGroup],
                                                 const u64 (&ow)[kBtGroup],
                                                 const u64 (&hoff)[kBtGroup], unsigned smax) {
    for (unsigned j = lane_id(); j < smax; j += 64) {
        int u[kBtGroup];
#pragma unroll
        for (unsigned g = 0; g < kBtGroup; ++g) u[g] = j < s[g] ? B.bt[base[g] + j] : -1;
#pragma unroll
        for (unsigned g = 0; g < kBtGroup; ++g) {
            if (j >= s[g]) continue;
            B.vunits[o[g] + j] = u[g];
            if (w[g]) {
                B.wunits[ow[g] + j] = u[g];
                if (B.whost) B.whost[ow[g] + j] = hoff[g] + (u64)j * B.unit_bytes;
                if (B.wrel) B.wrel[ow[g] + j] = (unsigned)(o[g] + j);
            }
            if (B.rhost) B.rhost[o[g] + j] = w[g] ? hoff[g] + (u64)j * B.unit_bytes : ~0ull;
            B.bt[base[g] + j] = -1;
        }
    }
}

// Hand a group of loads their units (row base[g], s[g] units, load-order
// offset o[g], host copy at hoff[g]): the pre-step free units first, then the
// victims' units in eviction order (nF = free units used).
__device__ __forceinline__ void bt_assign_group(const BtArgs& B, const u64 (&base)[kBtGroup],
                                                const unsigned (&s)[kBtGroup],
                                                const u64 (&o)[kBtGroup],
                                                const u64 (&hoff)[kBtGroup], u64 nF,
                                                unsigned smax) {
    for (unsigned j = lane_id(); j < smax; j += 64) {
        int u[kBtGroup];
#pragma unroll
        for (unsigned g = 0; g < kBtGroup; ++g) {
            const u64 q = o[g] + j;
            u[g] = j >= s[g] ? -1 : q < nF ? B.free_old[q] : B.vunits[q - nF];
        }
#pragma unroll
        for (unsigned g = 0; g < kBtGroup; ++g) {
            if (j >= s[g]) continue;
            const u64 q = o[g] + j;
            B.bt[base[g] + j] = u[g];
            B.lunits[q] = u[g];
            if (B.lhost) B.lhost[q] = hoff[g] + (u64)j * B.unit_bytes;
        }
    }
}

__device__ __forceinline__ unsigned lane_bcast(unsigned x, unsigned k) {
    return (unsigned)__builtin_amdgcn_readlane((int)x, (int)k);
}
__device__ __forceinline__ u64 lane_bcast(u64 x, unsigned k) {
    return ((u64)lane_bcast((unsigned)(x >> 32), k) << 32) | lane_bcast((unsigned)x, k);
}

// The block-table update inside one workgroup.  Wave w takes victims (then
// loads) w, w + nw, ...; lane k of a batch loads the k-th of them first, so
// the item-level loads of up to 64 items are in flight at once; the wave then
// takes the batch's items kBtGroup at a time, lanes over their units.
// Occupancy: the plan core already marked the pre-step free units the loads
// take; the released units that no load takes, released positions
// [units_in - nF, units_out), are freed here.  (Clearing every released unit's
// bit and setting every loaded unit's bit had cost about 0.4 ms at 50,000
// agents: consecutive units share a 32-bit word, so a wave's atomics
// serialized on two or three addresses.)
__device__ __forceinline__ void bt_update_block(const BtArgs& B, unsigned n_v, unsigned n_l,
                                                u64 nF, u64 units_in, u64 units_out) {
    const unsigned wid = threadIdx.x >> 6, nw = blockDim.x >> 6, lane = lane_id();
    for (unsigned i0 = wid; i0 < n_v; i0 += 64 * nw) {
        const unsigned ik = i0 + lane * nw;
        unsigned v = 0, w = 0, s = 0;
        u64 o = 0, ow = 0, base = 0, hoff = 0;
        if (ik < n_v) {
            v = B.victims[ik];
            o = B.voff[ik];
            ow = B.woff[ik];
            w = B.vwritten[ik];
            base = B.agent_off[v];
            s = B.units[v];
            if (B.whost) hoff = B.host_off[v];
        }
        const unsigned rounds = min(64u, (n_v - i0 + nw - 1) / nw);
        for (unsigned k0 = 0; k0 < rounds; k0 += kBtGroup) {
            u64 gb[kBtGroup], go[kBtGroup], gow[kBtGroup], gh[kBtGroup];
            unsigned gs[kBtGroup], smax = 0;
            bool gw[kBtGroup];
#pragma unroll
            for (unsigned g = 0; g < kBtGroup; ++g) {
                const bool in = k0 + g < rounds;
                const unsigned k = in ? k0 + g : k0;       // a lane of the batch either way
                gb[g] = lane_bcast(base, k);
                gs[g] = in ? lane_bcast(s, k) : 0u;
                go[g] = lane_bcast(o, k);
                gw[g] = lane_bcast(w, k) != 0;
                gow[g] = lane_bcast(ow, k);
                gh[g] = lane_bcast(hoff, k);
                smax = max(smax, gs[g]);
            }
            bt_release_group(B, gb, gs, go, gw, gow, gh, smax);
        }
    }
    __syncthreads();                                 // the victims' units, before the loads take them
    for (u64 q = (units_in > nF ? units_in - nF : 0) + threadIdx.x; q < units_out; q += blockDim.x) {
        const int u = B.vunits[q];
        if ((u64)(unsigned)u < B.capacity)
            atomicAnd(&B.occ[(unsigned)u >> 5], ~(1u << ((unsigned)u & 31u)));
    }
    for (unsigned i0 = wid; i0 < n_l; i0 += 64 * nw) {
        const unsigned ik = i0 + lane * nw;
        unsigned s = 0;
        u64 o = 0, base = 0, hoff = 0;
        if (ik < n_l) {
            const unsigned a = B.loads[ik];
            o = B.loff[ik];
            base = B.agent_off[a];
            s = B.units[a];
            if (B.lhost) hoff = B.host_off[a];
        }
        const unsigned rounds = min(64u, (n_l - i0 + nw - 1) / nw);
        for (unsigned k0 = 0; k0 < rounds; k0 += kBtGroup) {
            u64 gb[kBtGroup], go[kBtGroup], gh[kBtGroup];
            unsigned gs[kBtGroup], smax = 0;
#pragma unroll
            for (unsigned g = 0; g < kBtGroup; ++g) {
                const bool in = k0 + g < rounds;
                const unsigned k = in ? k0 + g : k0;
                gb[g] = lane_bcast(base, k);
                gs[g] = in ? lane_bcast(s, k) : 0u;
                go[g] = lane_bcast(o, k);
                gh[g] = lane_bcast(hoff, k);
                smax = max(smax, gs[g]);
            }
            bt_assign_group(B, gb, gs, go, gh, nF, smax);
        }
    }
}

// The plan core's tail; its arguments come from the pool's device copy, not
// from the kernel's.  Inlined like the rest of the plan (no call, so no stack
// in scratch memory).
__device__ __forceinline__ void bt_tail(const BtArgs* Bp, unsigned n_v, unsigned n_l,
                                                  u64 nF, u64 units_in, u64 units_out) {
    const BtArgs B = *Bp;
    bt_update_block(B, n_v, n_l, nF, units_in, units_out);
}

// Publish the plan to the host: every thread's host-visible writes are made
// visible at system scope, then one thread writes the plan's sequence number
// to the mapped flag word, which the host polls.  The fences only release:
// nothing after them reads what the host writes (a full fence also
// invalidates the L2 at system scope, in every wave).
__device__ __forceinline__ void publish_plan(const PlanArgs& A) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
    __syncthreads();
    if (threadIdx.x == 0)
        __hip_atomic_store(A.flag_host, A.seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// The plan core: one workgroup of kCoreThreads threads; `lds` holds kLdsKeys
// keys.  Inlined into both kernels below so that its LDS accesses stay LDS
// instructions.  kFused: its workgroup classified the agents (k_plan_core;
// histograms and counters in LDS); otherwise it runs in the last classifying
// workgroup of k_classify_core (histograms and counters in global memory).
// After publishing the plan it updates the block table.
//
// Only the keys that can take part in the plan are sorted.  Write need for the
// units the demand loads lack (demand units minus free units), HC[b] and HE[b]
// for the units of the candidates and of the evictable residents whose
// distance falls in bucket b (dist_bucket is monotone in the distance).
//  * Candidates.  The capacity a candidate of distance x may use is
//    free1 + G(x) = max(P(lo), P(n_d)) - need, with P the unit prefix over the
//    eviction order, lo the evictable residents farther than x and n_d the
//    demand victims; P(lo) <= HEsuf(b) (units of buckets >= b) and
//    P(n_d) < need + smax when need > 0 (0 otherwise).  A candidate of bucket b
//    uses at least HCbefore(b) + 1 units, so if that exceeds
//    min(budget, max(HEsuf(b) - need, free1 bound)) no candidate of bucket b
//    or later is accepted (the left side grows with b, the right side
//    shrinks).  The buckets below b_cut, the first such bucket, hold every
//    accepted candidate; only they are gathered and sorted.
//  * Evictable residents.  Accepted candidates use at most
//    Cmax = min(budget, HCbefore(b_cut)) units, so every victim has less than
//    R = need + Cmax units of evictable residents before it in eviction order.
//    With b_E the last bucket whose HEsuf reaches R, all victims lie in the
//    buckets >= b_E (T): a resident of a lower bucket comes after all of T,
//    whose units reach R.  T is gathered and sorted instead of all residents.
//    The acceptance test stays exact: a candidate nearer than every key of T
//    has free1 + G >= units(T) - need >= Cmax, which is what the test then
//    computes from T as well.  (R <= 0: no victims, T is empty; HEsuf(0) < R:
//    T is every evictable resident.)
template <bool kFused>
__device__ __forceinline__ void plan_core(const PlanArgs& A, u64* lds, CoreShared& S) {
    const unsigned tid = threadIdx.x;
    auto stamp = [&](int k) {
        if (A.phase && tid == 0) A.phase[k] = wall_clock64();
    };
    const u64 idmask = (1ull << A.idbits) - 1;
    const unsigned idb = A.idbits;
    const unsigned* units = A.units;
    unsigned* he_lds = reinterpret_cast<unsigned*>(lds);
    // the histograms and counters: this workgroup's LDS when it classified the
    // agents itself, else the global sums of all classifying workgroups (the
    // counters copied into LDS)
    const u64* histw = kFused ? S.histw : A.hist_w;
    const unsigned* histe = kFused ? he_lds : A.hist_e;
    if (!kFused && tid == 0) S.cnt = *A.cnt;
    __syncthreads();
    const PlanCounters& c = S.cnt;
    stamp(1);

    static_assert(kDistBuckets == 2 * kCoreThreads, "two buckets per thread");
    const unsigned b0 = 2 * tid;
    const u64 hc0 = histw[b0], hc1 = histw[b0 + 1];
    const u64 he0 = histe[b0], he1 = histe[b0 + 1];
    if (!kFused) {                                   // each thread clears what it read
        A.hist_w[b0] = 0;
        A.hist_w[b0 + 1] = 0;
        A.hist_e[b0] = 0;
        A.hist_e[b0 + 1] = 0;
    }
    if (c.sum_active > A.capacity) {                 // overcommit: change nothing
        if (tid == 0) {
            PlanResult r = {};
            r.status = 1;
            *A.res = r;
            *A.res_host = r;
            if (!kFused) *A.cnt = PlanCounters{};
        }
        publish_plan(A);
        stamp(8);
        return;
    }
    const u64 free_before = A.capacity - c.sum_resident;
    const long long need = (long long)c.sum_demand - (long long)free_before;
    const unsigned nE = c.n_E, nL = c.n_L;

    // the cuts (see above): one scan of both histograms (packed into one word
    // when their totals fit 32 bits), then the first bucket that fails and the
    // first that does not reach R, each the minimum of a per-wave candidate
    // (lanes hold ascending buckets) by one LDS atomic per wave
    if (tid == 0) {
        S.uscal[0] = kDistBuckets;
        S.uscal[1] = kDistBuckets;
    }
    u64 hcb, heb, tot_c, tot_e;                      // HCbefore(b0), HEbefore(b0), totals
    if (c.sum_cand < (1ull << 32) && c.sum_evictable < (1ull << 32)) {   // block-uniform
        u64 tot;
        const u64 x = block_excl_scan(((hc0 + hc1) << 32) | (he0 + he1), S, &tot);
        hcb = x >> 32;
        heb = x & 0xFFFFFFFFull;
        tot_c = tot >> 32;
        tot_e = tot & 0xFFFFFFFFull;
    } else {
        hcb = block_excl_scan(hc0 + hc1, S, &tot_c);
        heb = block_excl_scan(he0 + he1, S, &tot_e);
    }
    auto wave_first = [&](unsigned b, unsigned* dst) {
        const u64 m = __ballot(b < kDistBuckets);
        if (m && lane_id() == (unsigned)__ffsll((long long)m) - 1) atomicMin(dst, b);
    };
    const long long f1ub = need > 0 ? (long long)A.smax - 1 : -need;
    auto fails = [&](u64 hc_before, u64 he_before) {
        long long lim = (long long)(tot_e - he_before) - need;  // HEsuf(b) - need
        if (lim < f1ub) lim = f1ub;
        const u64 cap = A.budget < (u64)lim ? A.budget : (u64)lim;
        return hc_before >= cap;                                // hc_before + 1 > cap
    };
    // the buckets that do not fail form the prefix [0, b_cut)
    wave_first(fails(hcb, heb) ? b0 : fails(hcb + hc0, heb + he0) ? b0 + 1 : kDistBuckets,
               &S.uscal[0]);
    __syncthreads();
    const unsigned b_cut = S.uscal[0];
    if (b_cut < kDistBuckets && tid == b_cut / 2) S.wsum[0] = (b_cut & 1) ? hcb + hc0 : hcb;
    __syncthreads();
    const u64 hc_cut = b_cut < kDistBuckets ? S.wsum[0] : tot_c;       // HCbefore(b_cut)
    const u64 cmax = A.budget < hc_cut ? A.budget : hc_cut;
    const long long R = need + (long long)cmax;
    unsigned b_E = kDistBuckets;                     // R <= 0: no victims
    if (R > 0) {
        // the buckets whose HEsuf reaches R form a prefix [0, b_E]
        const u64 r = (u64)R;
        wave_first(tot_e - heb < r ? b0 : tot_e - heb - he0 < r ? b0 + 1 : kDistBuckets,
                   &S.uscal[1]);
        __syncthreads();
        const unsigned fr = S.uscal[1];
        b_E = fr ? fr - 1 : 0;                       // none reaches R: every evictable resident
        // units of the evictable residents of buckets >= b_E (the set sorted
        // below): HEsuf(b_E), from the thread that holds bucket b_E
        if (tid == b_E / 2) S.scal[0] = tot_e - ((b_E & 1) ? heb + he0 : heb);
        __syncthreads();
    }
    const u64 units_T = b_E < kDistBuckets ? S.scal[0] : 0;

    // The sorted sets: the evictable residents of buckets >= b_E (ascending;
    // eviction order is descending key = the reversed array), the demand loads
    // by id (their distance is 0, so key order is id order) and the candidates
    // of buckets < b_cut, from the sub-lists whose distance range starts below
    // b_cut.  Jointly in LDS when they fit (their counts are known once they
    // are gathered), else one by one with the global-memory fallbacks.
    auto keepT = [&](u64 k) { return dist_bucket((unsigned)(k >> idb)) >= b_E; };
    auto keepC = [&](u64 k) { return dist_bucket((unsigned)(k >> idb)) < b_cut; };
    auto gatherC = [&](u64* buf, unsigned cap, unsigned* counter, u64 tag) {
        for (unsigned k = 0; k < kCandLists; ++k)
            if (cand_list_start(k) < b_cut && c.n_C[k])
                gather_keys(A.listC + (u64)k * A.n, c.n_C[k], keepC, buf, cap, counter, tag);
    };
    unsigned nT = 0, m = 0;
    bool joint = idb + 32 <= kTagShift;              // kernel-uniform
    if (joint) {
        if (tid == 0) {
            S.uscal[6] = 0;
            S.uscal[7] = 0;
        }
        __syncthreads();
        if (b_E < kDistBuckets) gather_keys(A.listE, nE, keepT, lds, kJointKeys, &S.uscal[7]);
        __syncthreads();
        nT = S.uscal[7];
        if (nT + nL <= kJointKeys) {                 // block-uniform
            for (unsigned i = tid; i < nL; i += kCoreThreads) lds[nT + i] = A.listL[i] | kTagL;
            gatherC(lds + nT + nL, kJointKeys - nT - nL, &S.uscal[6], kTagC);
        }
        __syncthreads();
        m = S.uscal[6];
        if (nT + nL + m <= kJointKeys) joint_sort_out(lds, nT + nL + m, nT, nL, A.sortE, A.sortL, A.sortC);
        else joint = false;
    }
    if (!joint) {
        select_sort(A.listL, nL, ~0ull, nL, A.sortL, lds, S);
        nT = b_E >= kDistBuckets ? 0u : gather_sorted(
            [&](u64* buf, unsigned cap, unsigned* counter) {
                gather_keys(A.listE, nE, keepT, buf, cap, counter);
            }, A.sortE, lds, S);
        m = gather_sorted(
            [&](u64* buf, unsigned cap, unsigned* counter) { gatherC(buf, cap, counter, 0); },
            A.sortC, lds, S);
    }
    const u64* sortE = A.sortE;
    const u64* sortC = A.sortC;
    // The three unit prefixes in one pass over the evictable keys in eviction
    // order (descending), then the demand keys, then the candidates: prefE
    // over the first, loff and prefC over the others, each from 0 (the bases
    // are the units of the evictable set, HEsuf(b_E), and of the demand loads,
    // sum_demand).  The keys come from the joint sort's LDS array where it ran
    // (evictable keys at [0, nT), demand keys after them, then the candidates;
    // tags lie above idmask).
    {
        const unsigned nTL = nT + nL;
        const u64 baseL = units_T, baseC = units_T + c.sum_demand;
        if (tid == 0) {
            A.prefE[0] = 0;
            A.loff[0] = 0;
            A.prefC[0] = 0;
        }
        block_prefix_to(nTL + m, [&](unsigned i) {
            u64 k;
            if (joint) k = lds[i < nT ? nT - 1 - i : i];
            else k = i < nT ? sortE[nT - 1 - i] : i < nTL ? A.sortL[i - nT] : sortC[i - nTL];
            return (u64)units[k & idmask];
        }, [&](unsigned i, u64 v) {
            if (i < nT) A.prefE[i + 1] = v;
            else if (i < nTL) A.loff[i - nT + 1] = v - baseL;
            else A.prefC[i - nTL + 1] = v - baseC;
        }, S);
    }
    stamp(2);

    // demand victims: shortest prefix of the eviction order covering `need`.
    // prefE is non-decreasing and prefE[nT] >= R >= need, so its length is the
    // number of prefix values below need (prefE[0] = 0 among them): counted by
    // the whole block instead of one thread's chain of dependent loads.
    unsigned n_d = 0;
    if (need > 0) {                                  // block-uniform
        u64 below = 0;
#pragma unroll 4
        for (unsigned i = tid; i < nT; i += blockDim.x) below += (long long)A.prefE[i] < need;
        u64 tot;
        (void)block_excl_scan(below, S, &tot);
        n_d = (unsigned)tot;
    }
    const u64 free1 = free_before + A.prefE[n_d] - c.sum_demand;

    stamp(3);

    // acceptance: S_i <= budget and S_i <= free1 + (units of the remaining
    // evictable residents with distance strictly larger than d_i)
    if (tid == 0) S.uscal[3] = m;
    // the evictable keys and their unit prefix in LDS for the searches below
    // when both fit (the joint sort left the keys there; the sort buffer is
    // free otherwise)
    const bool in_lds = 2 * nT + 1 <= (unsigned)kLdsKeys;   // block-uniform
    if (in_lds) {
        if (!joint) for (unsigned i = tid; i < nT; i += blockDim.x) lds[i] = sortE[i];
        for (unsigned i = tid; i <= nT; i += blockDim.x) lds[nT + i] = A.prefE[i];
    }
    const u64* keysE = in_lds ? lds : sortE;
    const u64* pref = in_lds ? lds + nT : A.prefE;
    __syncthreads();
    stamp(4);
    // (the search runs on LDS or on global memory; each instance sees which,
    // so the LDS one uses LDS instructions)
    auto accept = [&](const u64* keysE, const u64* pref) __attribute__((always_inline)) {
        // kAccept candidates per thread at once: their binary searches run in
        // lockstep (ceil(log2(nT + 1)) steps), so the loads of one overlap the
        // others'
        constexpr unsigned kAccept = 4;
        const unsigned steps = nT ? 32u - (unsigned)__clz(nT) : 0u;
        const u64 base_units = pref[n_d];
        for (unsigned i0 = tid; i0 < m; i0 += kAccept * blockDim.x) {
            u64 di[kAccept], Si[kAccept];
            unsigned lo[kAccept], hi[kAccept];
#pragma unroll
            for (unsigned u = 0; u < kAccept; ++u) {
                const unsigned i = i0 + u * blockDim.x;
                di[u] = i < m ? sortC[i] >> idb : 0;
                Si[u] = i < m ? A.prefC[i + 1] : 0;
                lo[u] = 0;                           // first eviction index with d <= di
                hi[u] = i < m ? nT : 0;
            }
            for (unsigned it = 0; it < steps; ++it) {
#pragma unroll
                for (unsigned u = 0; u < kAccept; ++u) {
                    if (lo[u] < hi[u]) {
                        const unsigned mid = (lo[u] + hi[u]) >> 1;
                        if ((keysE[nT - 1 - mid] >> idb) > di[u]) lo[u] = mid + 1;
                        else hi[u] = mid;
                    }
                }
            }
#pragma unroll
            for (unsigned u = 0; u < kAccept; ++u) {
                // the wave's first failing candidate (lanes hold consecutive
                // i) goes to one LDS atomic per wave: most candidates past the
                // accepted prefix fail, and same-address atomics serialize
                const unsigned i = i0 + u * blockDim.x;
                const u64 G = lo[u] > n_d ? pref[lo[u]] - base_units : 0;
                const bool fail = i < m && !(Si[u] <= A.budget && Si[u] <= free1 + G);
                const u64 fm = __ballot(fail);
                if (fm && lane_id() == (unsigned)__ffsll((long long)fm) - 1)
                    atomicMin(&S.uscal[3], i);
            }
        }
    };
    if (in_lds) accept(lds, lds + nT);
    else accept(sortE, A.prefE);
    __syncthreads();
    stamp(5);
    const unsigned n_p = S.uscal[3];
    // victims: the demand victims, extended while the accepted loads need
    // room: to the first eviction index past n_d whose prefix reaches the
    // target, i.e. n_d + 1 plus the prefix values below it (counted by the
    // whole block), at most nT
    unsigned n_v = n_d;
    if (n_p > 0 && A.prefC[n_p] > free1) {           // block-uniform
        const u64 target = pref[n_d] + (A.prefC[n_p] - free1);
        u64 below = 0;
#pragma unroll 4
        for (unsigned i = n_d + 1 + tid; i < nT; i += blockDim.x) below += pref[i] < target;
        u64 tot;
        (void)block_excl_scan(below, S, &tot);
        n_v = min(nT, n_d + 1 + (unsigned)tot);
    }
    const unsigned n_l = nL + n_p;
    const u64 units_out = pref[n_v];
    const u64 units_in = c.sum_demand + A.prefC[n_p];

    // plan lists, load offsets, residency (victims and loads are disjoint)
    for (unsigned i = tid; i < n_l; i += blockDim.x) {
        const unsigned a = (unsigned)((i < nL ? A.sortL[i] : sortC[i - nL]) & idmask);
        A.loads[i] = a;
        A.loads_host[i] = a;
        A.resident[a] = 1;
        if (i >= nL) A.loff[i + 1] = c.sum_demand + A.prefC[i - nL + 1];
    }
    // the victims, and the offsets of the written-back victims' units (all of
    // them without a mask): with at most one victim per thread, from the same
    // loads in one pass
    auto victim = [&](unsigned i, u64* wunits) {
        const unsigned v = (unsigned)(keysE[nT - 1 - i] & idmask);
        const unsigned char w = (!A.dirty || A.dirty[v]) ? 1 : 0;
        A.victims[i] = v;
        A.victims_host[i] = v;
        A.vwritten[i] = w;
        A.vwritten_host[i] = w;
        A.resident[v] = 0;
        *wunits = w ? (u64)units[v] : 0ull;
    };
    if (n_v <= blockDim.x) {
        u64 wv = 0;
        if (tid < n_v) victim(tid, &wv);
        u64 tot;
        const u64 ex = block_excl_scan(wv, S, &tot);
        if (tid == 0) A.woff[0] = 0;
        if (tid < n_v) A.woff[tid + 1] = ex + wv;
        __syncthreads();
    } else {
        u64 wv;
        for (unsigned i = tid; i < n_v; i += blockDim.x) victim(i, &wv);
        block_prefix(n_v, [&](unsigned i) {
            const unsigned v = (unsigned)(keysE[nT - 1 - i] & idmask);
            return (!A.dirty || A.dirty[v]) ? (u64)units[v] : 0ull;
        }, A.woff, S);
    }

    stamp(6);
    // pre-step free units, as many as the loads can use (the host needs only
    // their count)
    const u64 n_free_used = units_in < free_before ? units_in : free_before;
    __syncthreads();
    if (tid == 0) {
        PlanResult r = {};
        r.status = 0;
        r.n_victims = n_v;
        r.n_loads = n_l;
        r.n_demand = nL;
        r.n_demand_victims = n_d;
        r.units_out = units_out;
        r.units_in = units_in;
        r.free_before = free_before;
        r.n_free_used = n_free_used;
        r.units_written = A.woff[n_v];
        *A.res = r;
        *A.res_host = r;
        if (!kFused) *A.cnt = PlanCounters{};
    }
    publish_plan(A);
    stamp(7);
    // The host has the plan; the workgroup goes on to pick the pre-step free
    // units (ascending) and to update the block table (waves over victims,
    // then over loads), off the plan's return path.  The update saves the
    // step the launches of separate update kernels (queueing those two
    // kernels behind the multi-workgroup plan kernel cost the host about
    // 0.1 ms per call).  The free units all go to this step's loads, so the
    // thread that owns their occupancy word marks them in use there (plain
    // stores: one owner per word); the update then only frees the released
    // units that no load takes.  Every list the update reads was written above
    // by this workgroup; the barriers inside publish_plan and below order
    // those writes before its reads.
    const unsigned occ_per = (A.occ_words + blockDim.x - 1) / blockDim.x;
    if (n_free_used > 0 && occ_per <= 2) {
        free_scan_regs<2>(A, n_free_used, occ_per, S);
    } else if (n_free_used > 0 && occ_per <= kOccRegs) {
        free_scan_regs<kOccRegs>(A, n_free_used, occ_per, S);
    } else if (n_free_used > 0) {
        const unsigned W = A.occ_words;
        const unsigned per = occ_per;
        const unsigned w0 = tid * per;
        const unsigned w1 = min(W, w0 + per);
        u64 cnt = 0;
        for (unsigned w = w0; w < w1; ++w) cnt += __popc(~A.occ[w]);
        u64 tot;
        u64 pos = block_excl_scan(cnt, S, &tot);
        for (unsigned w = w0; w < w1 && pos < n_free_used; ++w) {
            const unsigned word = A.occ[w];
            unsigned bits = ~word, used = 0;
            while (bits && pos < n_free_used) {
                const unsigned b = __ffs(bits) - 1;
                bits &= bits - 1;
                used |= 1u << b;
                A.free_old[pos++] = (int)(w * 32u + b);
            }
            if (used) A.occ[w] = word | used;
        }
    }

    __syncthreads();
    bt_tail(A.bt, n_v, n_l, n_free_used, units_in, units_out);
    if (A.phase) {                                   // kernel-uniform
        __syncthreads();
        stamp(8);                                    // the whole plan kernel, tail included
    }
}

typedef const __attribute__((address_space(4))) PlanArgs PlanArgsK;

// The kernel's arguments read afresh from the kernel-argument segment,
// through a pointer the compiler cannot trace back to earlier loads: the plan
// core takes its arguments from it after the classification, otherwise the
// compiler keeps the argument block that the classification's loads merged
// live across the whole core, spilled to lanes of a vector register and
// reloaded as a unit (thousands of v_readlane).
__device__ __forceinline__ const PlanArgs& fresh_args() {
    u64 bits = (u64)__builtin_amdgcn_kernarg_segment_ptr();
    asm volatile("" : "+s"(bits));
    bits = ((u64)(unsigned)__builtin_amdgcn_readfirstlane((int)(bits >> 32)) << 32) |
           (unsigned)__builtin_amdgcn_readfirstlane((int)bits);
    return *(const PlanArgs*)(PlanArgsK*)bits;      // constant segment: scalar loads
}

__global__ void __launch_bounds__(kCoreThreads) k_plan_core(PlanArgs A) {
    __shared__ u64 lds[kLdsKeys];
    __shared__ CoreShared S;
    if (A.phase && threadIdx.x == 0) A.phase[0] = wall_clock64();
    unsigned* he = reinterpret_cast<unsigned*>(lds);  // evictable units per bucket
    if (threadIdx.x == 0) S.cnt = PlanCounters{};
    for (unsigned b = threadIdx.x; b < kDistBuckets; b += kCoreThreads) {
        S.histw[b] = 0;
        he[b] = 0;
    }
    __syncthreads();
    classify_fused(A, S, he, he + kDistBuckets);
    __syncthreads();
    plan_core<true>(fresh_args(), lds, S);
}

// Classification over many workgroups, then the plan core in the workgroup
// that finishes last (N > kFuseAgents).  Each workgroup classifies
// kClassBatch * 1024 agents, gathers its counts and sums in LDS and reaches
// the global counters with one atomic per counter; its list entries go to the
// ranges those atomics reserve.  Every workgroup then publishes its writes
// (device-scope release) and counts itself done; the one that counts last
// acquires them all and runs the plan core, so no workgroup ever waits for
// another and the core starts without a second launch.  It resets the count
// for the next step.  (Same-address atomics across workgroups serialize, so
// fewer, larger workgroups reach the core sooner.)
__global__ void __launch_bounds__(kCoreThreads) k_classify_core(PlanArgs A) {
    __shared__ u64 lds[kLdsKeys];
    __shared__ CoreShared S;
    const unsigned first = blockIdx.x * (kClassBatch * kCoreThreads) + threadIdx.x;
    if (A.phase && blockIdx.x == 0 && threadIdx.x == 0) A.phase[0] = wall_clock64();
    AgentBatch b;
    load_agents(A, first, A.n, b);                   // in flight while LDS is cleared
    unsigned* he = reinterpret_cast<unsigned*>(lds);  // evictable units per bucket (this workgroup)
    unsigned* tab = he + kDistBuckets;                // reserve_pass's table
    if (threadIdx.x == 0) S.cnt = PlanCounters{};
    for (unsigned k = threadIdx.x; k < kDistBuckets; k += kCoreThreads) {
        S.histw[k] = 0;
        he[k] = 0;
    }
    __syncthreads();
    u64 key[kClassBatch];
    unsigned lst[kClassBatch], slot[kClassBatch];
    ClassSums t;
#pragma unroll
    for (unsigned u = 0; u < kClassBatch; ++u) {
        const unsigned a = first + u * kCoreThreads;
        const AgentClass c = classify(A, a, a < A.n, b.D[u], b.act[u] != 0, b.res[u] != 0);
        // candidate and evictable units per distance bucket: LDS first
        // (distances concentrate on few buckets, where global atomics would
        // serialize), one global atomic per non-empty bucket and workgroup
        // below
        if (c.isC) atomicAdd(&S.histw[c.bucket], (u64)b.s[u]);
        if (c.isE) atomicAdd(&he[c.bucket], b.s[u]);
        key[u] = c.key;
        lst[u] = list_of(c);
        t.add(c, b.act[u] != 0, b.res[u] != 0, b.s[u]);
    }
    flush_sums(t, &S.cnt);                           // complete at reserve_pass's first barrier
    reserve_pass<true>(lst, slot, tab, &S.cnt, A.cnt);
    if (threadIdx.x < 5) {                           // the workgroup's unit sums, one lane each
        const PlanCounters& lc = S.cnt;
        PlanCounters* g = A.cnt;
        const unsigned l = threadIdx.x;
        const u64 v = l == 0 ? lc.sum_active : l == 1 ? lc.sum_resident : l == 2 ? lc.sum_demand
                    : l == 3 ? lc.sum_evictable : lc.sum_cand;
        u64* dst = l == 0 ? &g->sum_active : l == 1 ? &g->sum_resident : l == 2 ? &g->sum_demand
                 : l == 3 ? &g->sum_evictable : &g->sum_cand;
        if (v) atomicAdd(dst, v);
    }
#pragma unroll
    for (unsigned u = 0; u < kClassBatch; ++u)
        if (lst[u] != kNoList) list_ptr(A, lst[u])[slot[u]] = key[u];
    for (unsigned k = threadIdx.x; k < kDistBuckets; k += kCoreThreads) {
        if (S.histw[k]) atomicAdd(&A.hist_w[k], S.histw[k]);
        if (he[k]) atomicAdd(&A.hist_e[k], he[k]);
    }
    // Every wave has issued its list entries and atomics before the barrier;
    // one thread's device-scope release then covers them (the L2 write-back
    // it issues completes behind the requests the compute unit issued before
    // it), and it counts the workgroup done.  The last workgroup's thread
    // acquires every workgroup's writes the same way before the barrier that
    // lets its workgroup read them.
    __syncthreads();
    if (threadIdx.x == 0) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        const bool last = atomicAdd(A.done, 1u) == gridDim.x - 1;
        if (last) {
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            *A.done = 0;
        }
        S.uscal[3] = last;
    }
    __syncthreads();
    if (!S.uscal[3]) return;                         // workgroup-uniform
    plan_core<false>(fresh_args(), lds, S);
}

// ---------------------------------------------------------------------------
// pack / unpack
// ---------------------------------------------------------------------------

// Pointers into global memory.  The pool's planes arrive as 64-bit integers,
// so without the address space the compiler emits flat instructions for them;
// with flat accesses the deeper bursts below did not pay (5.5 TB/s for the
// gather instead of 6.0).
typedef __attribute__((address_space(1))) v4u gv4u;

// One wave copies len bytes (multiple of 16, at most kItemBytes): lane l moves
// the 16-byte words l, l+64, l+128, ...; eight words per lane are loaded
// before any is stored so that each wave keeps 8 KiB in flight.  Loads and
// stores are non-temporal: every byte is touched once.
__device__ __forceinline__ void wave_copy(char* dst, const char* src, unsigned len) {
    const gv4u* s = (const gv4u*)src;
    gv4u* d = (gv4u*)dst;
    const unsigned n16 = len >> 4;
    unsigned i = lane_id();
    for (; i + 7 * 64 < n16; i += 8 * 64) {
        v4u r[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) r[k] = __builtin_nontemporal_load(s + i + k * 64);
#pragma unroll
        for (int k = 0; k < 8; ++k) __builtin_nontemporal_store(r[k], d + i + k * 64);
    }
    for (; i < n16; i += 64) __builtin_nontemporal_store(__builtin_nontemporal_load(s + i), d + i);
}

// A full kItemBytes piece moves as one burst: every lane loads all of its
// words (32 KiB per wave in flight) before the first store, so the piece's
// stores also leave the wave back to back.  On the round-robin layout (32 KiB
// pieces scattered over 64 planes) this ran the gather at 6.0 TB/s and the
// scatter at 5.6 TB/s, against 5.6 and 5.2 with 8 KiB rounds.  Shorter pieces
// take the rounds.  The burst is branch-free: per-word conditions make the
// compiler wait for each store before the next.
__device__ __forceinline__ void wave_copy_burst(char* dst, const char* src, unsigned len) {
    if (len != kItemBytes) {
        wave_copy(dst, src, len);
        return;
    }
    constexpr int kWords = kItemBytes / 1024;     // 16-byte words per lane
    const gv4u* s = (const gv4u*)src + lane_id();
    gv4u* d = (gv4u*)dst + lane_id();
    v4u r[kWords];
#pragma unroll
    for (int k = 0; k < kWords; ++k) r[k] = __builtin_nontemporal_load(s + k * 64);
#pragma unroll
    for (int k = 0; k < kWords; ++k) __builtin_nontemporal_store(r[k], d + k * 64);
}

// One item (a piece of one plane's chunk) per wave.
// Pack: block b copies items [g*8, g*8+8) of logical unit p = b / item_groups
// (g = b % item_groups), so consecutive blocks walk a unit's bytes in order and
// a block's stores fill 8 consecutive pieces of the staging slot.
// Unpack with run_order (set when every plane's chunk is a single item):
// block b copies item r = b % n_items of the 8 logical units [t*8, t*8+8),
// t = b / n_items, one unit per wave.  The loads' units mostly come in runs of
// consecutive physical units (allocation hands out free units in index
// order), and consecutive units of a plane are adjacent, so a block's stores
// fill one run of a plane: on the round-robin workload's unit lists this ran
// at 5.7-5.8 TB/s against 5.6 for the pack order (and 5.2 against 5.4 on
// random lists).  Without run_order (chunks of several items, which already
// give each block a contiguous range) the unpack takes the pack order.
// Direct mode (stage_off set): the "staging" side is each unit's place in its
// agent's pinned host copy, so the same kernel moves the bytes over the host
// link itself.
// The item index is wave-uniform, so its descriptor and the plane's base and
// stride are scalar loads.
template <bool kPack>
__global__ void __launch_bounds__(kCopyThreads) k_copy(CopyArgs A) {
    const unsigned b = blockIdx.x;
    const unsigned wid = threadIdx.x >> 6;
    unsigned p, r;
    if (kPack || !A.run_order) {
        p = b / A.item_groups;
        r = __builtin_amdgcn_readfirstlane((b - p * A.item_groups) * kCopyWavesPerBlock + wid);
        if (r >= A.n_items) return;
    } else {
        const unsigned t = b / A.n_items;
        r = b - t * A.n_items;
        p = __builtin_amdgcn_readfirstlane(t * kCopyWavesPerBlock + wid);
        if (p >= A.count) return;
    }
    const u64 u = (u64)(unsigned)A.units_list[A.first + p];
    if (u >= A.capacity) return;
    const CopyItem it = A.items[r];
    char* chunk = reinterpret_cast<char*>(A.plane_base[it.plane]) + u * A.chunk_bytes[it.plane] +
                  it.chunk_off;
    char* stage = A.staging + (A.stage_off ? A.stage_off[A.first + p] : (u64)p * A.unit_bytes) +
                  it.unit_off;
    if (kPack) wave_copy_burst(stage, chunk, it.len);
    else wave_copy_burst(chunk, stage, it.len);
}

__global__ void __launch_bounds__(kCopyThreads) k_probe_copy(char* dst, const char* src, u64 bytes) {
    const u64 w = (u64)blockIdx.x * kCopyWavesPerBlock + (threadIdx.x >> 6);
    const u64 off = w * kItemBytes;
    if (off >= bytes) return;
    const u64 rem = bytes - off;
    wave_copy(dst + off, src + off, rem < kItemBytes ? (unsigned)rem : kItemBytes);
}

__global__ void k_nop() {}

__global__ void k_zero_u32(unsigned* p, u64 n) {
    for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (u64)gridDim.x * blockDim.x)
        p[i] = 0;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

hipError_t launch_plan(const PlanArgs& a, hipStream_t st) {
    if (a.fused) {
        hipLaunchKernelGGL(k_plan_core, dim3(1), dim3(kCoreThreads), 0, st, a);
    } else {
        const unsigned per = kClassBatch * kCoreThreads;
        const unsigned blocks = (a.n + per - 1) / per;
        hipLaunchKernelGGL(k_classify_core, dim3(blocks), dim3(kCoreThreads), 0, st, a);
    }
    return hipGetLastError();
}

static hipError_t launch_copy(const CopyArgs& a, hipStream_t st, bool pack) {
    if (a.count == 0) return hipSuccess;
    if (a.item_groups == 0 || a.n_items == 0) return hipErrorInvalidValue;
    const u64 blocks = (pack || !a.run_order)
                           ? a.count * a.item_groups
                           : (a.count + kCopyWavesPerBlock - 1) / kCopyWavesPerBlock * a.n_items;
    if (blocks > 0x7fffffffull) return hipErrorInvalidValue;
    if (pack) hipLaunchKernelGGL(k_copy<true>, dim3((unsigned)blocks), dim3(kCopyThreads), 0, st, a);
    else hipLaunchKernelGGL(k_copy<false>, dim3((unsigned)blocks), dim3(kCopyThreads), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_pack(const CopyArgs& a, hipStream_t st) { return launch_copy(a, st, true); }
hipError_t launch_unpack(const CopyArgs& a, hipStream_t st) { return launch_copy(a, st, false); }

hipError_t launch_zero_u32(unsigned* p, u64 n, hipStream_t st) {
    if (n == 0) return hipSuccess;
    u64 blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(k_zero_u32, dim3((unsigned)blocks), dim3(256), 0, st, p, n);
    return hipGetLastError();
}

hipError_t launch_nop(hipStream_t st) {
    hipLaunchKernelGGL(k_nop, dim3(1), dim3(64), 0, st);
    return hipGetLastError();
}

hipError_t launch_probe_copy(void* dst, const void* src, u64 bytes, hipStream_t st) {
    const u64 items = (bytes + kItemBytes - 1) / kItemBytes;
    const u64 blocks = (items + kCopyWavesPerBlock - 1) / kCopyWavesPerBlock;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_probe_copy, dim3((unsigned)blocks), dim3(kCopyThreads), 0, st,
                       static_cast<char*>(dst), static_cast<const char*>(src), bytes);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// direct two-way copies
// ---------------------------------------------------------------------------

// Both directions of a direct step in one launch, so that the host link
// carries them at once: position p < n_in is load position p, whose unit
// first gives its old bytes to the host copy of the victim that released it
// (when that victim is written back) and then takes the load's bytes from its
// host copy; the positions after those are the written-back units that no
// load takes (written back only).  One wave per (position, item) in the pack
// order.  A unit's write-back and its load are the same wave's, in program
// order: the load's stores into the unit are issued after the write-back's
// loads from it have returned (the write-back's stores wait for their data).
__global__ void __launch_bounds__(kCopyThreads) k_duplex(DuplexArgs A) {
    const unsigned b = blockIdx.x;
    const unsigned wid = threadIdx.x >> 6;
    const u64 p = b / A.item_groups;
    const unsigned r =
        __builtin_amdgcn_readfirstlane((b - (unsigned)p * A.item_groups) * kCopyWavesPerBlock + wid);
    if (r >= A.n_items) return;
    const CopyItem it = A.items[r];
    auto chunk = [&](u64 u) {
        return reinterpret_cast<char*>(A.plane_base[it.plane]) + u * A.chunk_bytes[it.plane] +
               it.chunk_off;
    };
    if (p < A.n_in) {
        const u64 u = (u64)(unsigned)A.lunits[p];
        if (u >= A.capacity) return;
        if (p >= A.n_free) {
            const u64 h = A.rhost[p - A.n_free];
            if (h != ~0ull) wave_copy_burst(A.host + h + it.unit_off, chunk(u), it.len);
        }
        wave_copy_burst(chunk(u), A.host + A.lhost[p] + it.unit_off, it.len);
    } else {
        const u64 w = p - A.n_in;
        if (w >= A.n_written) return;
        if ((u64)A.wrel[w] + A.n_free < A.n_in) return;   // its load position wrote it back
        const u64 u = (u64)(unsigned)A.wunits[w];
        if (u >= A.capacity) return;
        wave_copy_burst(A.host + A.whost[w] + it.unit_off, chunk(u), it.len);
    }
}

hipError_t launch_duplex(const DuplexArgs& a, hipStream_t st) {
    const u64 positions = a.n_in + a.n_written;
    if (positions == 0) return hipSuccess;
    if (a.item_groups == 0 || a.n_items == 0) return hipErrorInvalidValue;
    const u64 blocks = positions * a.item_groups;
    if (blocks > 0x7fffffffull) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_duplex, dim3((unsigned)blocks), dim3(kCopyThreads), 0, st, a);
    return hipGetLastError();
}

}  // namespace ss
