// Distance kernels for gfx950: invocation distances of shared memory objects
// and the on-device distance estimators of Section 3.2.
//
// ss_object_distances (Appendix A, fine-grained distance assignment): an
// object referenced by several agents takes the smallest distance among them,
// and is needed now when any of them is active.  With v(a) = 0 for an active
// agent and D(a) otherwise, the object's distance is min over its referencing
// agents of v(a) and its activity is the OR of theirs, so one segmented
// min/or over the CSR map object -> agents computes both.
//
// The map is skewed (the root of a prefix tree is referenced by every agent,
// a leaf by one), so the work is split evenly over the merge of the two
// sorted lists "row ends" (obj_off[1..M]) and "reference indices" (0..R-1),
// the merge-path decomposition of Merrill and Garland (SC'16) for sparse
// products: every workgroup takes 2048 merge items, whatever the row lengths.
//   k_obj_prep  merge-path coordinates of every workgroup boundary (16 lanes
//               per boundary, 16 probes per round) and, in the same launch,
//               w[a] = 0 if a is active else 2 D[a] + 1, one word per agent.
//   k_obj_min   per workgroup: coalesced staging of its row ends and of
//               w of its references into LDS (the gather of the agents'
//               words happens here, one load per reference; every thread
//               issues all its loads before using any), an 8-item walk
//               per thread, LDS atomics for rows split between threads,
//               coalesced stores of the rows that end in the block and one
//               carry record for the row that continues past it.
//   k_obj_fix   applies the carry records with global atomic min / stores,
//               after every k_obj_min block has written its rows.
// No dense contraction here; the kernel is bound by HBM bytes and by the rate
// of random gathers.
//
// ss_hop_distances (predefined activation paths): multi-source breadth-first
// hop counts over a CSR graph in one cooperative launch.
//   k_bfs       level-synchronous, frontier queues in device memory; every
//               thread takes one frontier vertex and claims its unvisited
//               out-neighbours eight edges at a time with atomic
//               compare-and-swap, appending winners to the next queue with one
//               counter atomic per wave; a grid barrier (atomic arrival
//               counter and generation word, bounded spin) separates levels,
//               so the whole search is one launch and needs no host round
//               trip per level.
//
// ss_interaction_distances (interaction-involved simulations): D =
// min(D_action, floor(max(0, isqrt(d2) - radius) / velocity)) with d2 the
// squared distance to the nearest other agent on an integer tile grid.
//   k_pair_min  all pairs, 256 agents per workgroup against a slice of the
//               others staged through LDS as packed 16-bit (x, y); per pair a
//               packed 16-bit subtract and a 16-bit dot product give dx^2 +
//               dy^2 exactly; one atomic min per agent and slice.
//   k_pair_fin  integer square root, radius, velocity and the min with
//               D_action.
// Both are plain integer ALU work (no contraction), so no MFMA.
#include "scalesim.h"
#include "ss_internal.h"

#include <algorithm>
#include <mutex>

namespace ss {
namespace {

constexpr int kObjThreads = 256;
constexpr int kObjItems = 8;                          // merge items per thread
constexpr int kObjTile = kObjThreads * kObjItems;     // merge items per workgroup
constexpr unsigned kNone = 0xFFFFFFFFu;

struct ObjCarry {
    unsigned row;      // object, or kNone
    unsigned vmin;     // partial minimum of v over the block's references of row
    unsigned act;      // partial OR of activity
    unsigned pad;
};

struct ObjArgs {
    const unsigned* off;              // [M + 1]
    const unsigned* agents;           // [R]
    const unsigned* dist;             // [N]
    const unsigned char* active;      // [N]
    unsigned M, R, N;
    unsigned* out_dist;               // [M]
    unsigned char* out_act;           // [M]
    ObjCarry* carry;                  // [blocks]
    unsigned* coord;                  // [blocks + 1] rows consumed at each block boundary
    u64* w;                           // [N] 0 if active, else 2 * distance + 1
};

// Merge-path coordinate (rows consumed) at diagonal d: the first p in
// [max(0, d - R), min(d, M)) whose row end comes after reference d - p - 1,
// i.e. off[p + 1] + p + 1 > d (strictly increasing in p), else the upper
// bound.  A group of 16 lanes searches one diagonal, 16 probes per round, so
// a wave serves four boundaries and a search takes a few dependent loads.
__device__ unsigned group_path_search(const unsigned* __restrict__ off, unsigned M, unsigned R,
                                      unsigned d, bool valid) {
    const unsigned lane = __lane_id(), g = lane >> 4, gl = lane & 15u;
    unsigned lo = d > R ? d - R : 0u;
    unsigned hi = d < M ? d : M;
    if (!valid) lo = hi = 0;
    for (;;) {
        const bool busy = lo < hi;
        if (__ballot(busy) == 0) break;
        const unsigned step = busy ? (hi - lo + 15u) / 16u : 1u;
        const unsigned p = lo + gl * step;
        bool after = false;
        if (busy && p < hi) after = (u64)min(off[p + 1], R) + p + 1 > d;
        const unsigned gm = (unsigned)(__ballot(after) >> (g * 16u)) & 0xFFFFu;
        if (busy) {
            if (gm == 0) {
                const unsigned n_probe = (hi - lo + step - 1) / step;   // lanes with p < hi
                lo = lo + (n_probe - 1) * step + 1;
            } else {
                const unsigned f = __ffs(gm) - 1;
                hi = lo + f * step;
                if (f > 0) lo = lo + (f - 1) * step + 1;
            }
        }
    }
    return lo;
}

// Two independent preparations in one launch.  Blocks [0, part_blocks): the
// merge-path coordinate of every workgroup boundary b * kObjTile,
// b = 0..blocks (16 per block).  The rest: w[a] = 0 if agent a is active,
// else 2 D[a] + 1, so that k_obj_min gathers one word per reference that
// carries both the distance (w >> 1) and the activity (w == 0).
__global__ void __launch_bounds__(256) k_obj_prep(ObjArgs A, unsigned n_bounds,
                                                  unsigned part_blocks) {
    if (blockIdx.x < part_blocks) {
        const unsigned b = (blockIdx.x * 256u + threadIdx.x) >> 4;
        const bool valid = b < n_bounds;
        const unsigned d = valid ? (unsigned)min((u64)b * kObjTile, (u64)A.M + A.R) : 0u;
        const unsigned x = group_path_search(A.off, A.M, A.R, d, valid);
        if (valid && (threadIdx.x & 15u) == 0) A.coord[b] = x;
        return;
    }
    // 2048 agents per block and round, eight per thread, loads before stores
    const u64 stride = (u64)(gridDim.x - part_blocks) * 2048u;
    for (u64 base = (u64)(blockIdx.x - part_blocks) * 2048u + threadIdx.x; base < A.N;
         base += stride) {
        unsigned dv[8];
        unsigned char ac[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const u64 a = base + k * 256u;
            dv[k] = 0;
            ac[k] = 0;
            if (a < A.N) {
                dv[k] = A.dist[a];
                ac[k] = A.active[a];
            }
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const u64 a = base + k * 256u;
            if (a < A.N) A.w[a] = ac[k] ? 0ull : 2ull * dv[k] + 1ull;
        }
    }
}

// Persistent workgroups: the grid is a multiple of the eight XCDs, and
// workgroups are dispatched to the XCDs in turn (block b to XCD b % 8).  XCD x
// owns one contiguous range of tiles, which its workgroups walk side by side,
// so the objects of one subtree and the agent words they gather stay in that
// XCD's L2; a workgroup lives for many tiles, so the dispatcher is not the
// limit.
__global__ void __launch_bounds__(kObjThreads) k_obj_min(ObjArgs A, unsigned n_tiles) {
    // s_item[0, nrow) = row ends (absolute), s_item[nrow, nrow + nref) = v of
    // the block's references; nrow + nref = the block's merge items.  s_flag
    // has the same split: activity of the rows ending in the block (output),
    // then activity of the references.
    __shared__ unsigned s_item[kObjTile];
    __shared__ unsigned s_outd[kObjTile];     // rows ending in the block: min
    __shared__ unsigned char s_flag[kObjTile];
    __shared__ unsigned s_bmin, s_bact;

    constexpr unsigned kXcds = 8;
    const unsigned tid = threadIdx.x;
    const unsigned total = A.M + A.R;
    const unsigned xcd = blockIdx.x % kXcds, per_xcd = gridDim.x / kXcds;
    const unsigned q = n_tiles / kXcds, rem = n_tiles % kXcds;
    const unsigned t_lo = xcd < rem ? xcd * (q + 1) : rem * (q + 1) + (xcd - rem) * q;
    const unsigned t_hi = t_lo + (xcd < rem ? q + 1 : q);
    for (unsigned tile = t_lo + blockIdx.x / kXcds; tile < t_hi; tile += per_xcd) {
        const unsigned d0 = tile * (unsigned)kObjTile;
        const unsigned d1 = min(d0 + (unsigned)kObjTile, total);
        const unsigned o0 = A.coord[tile], o1 = A.coord[tile + 1];
        const unsigned r0 = d0 - o0, r1 = d1 - o1;
        const unsigned nrow = o1 - o0, nref = r1 - r0;
        if (tid == 0) {
            s_bmin = kNone;
            s_bact = 0;
        }

        // Staging: every thread owns items i = tid + k * kObjThreads of the
        // block's merge range; all loads of a kind are issued before any is used.
        unsigned val[kObjItems];
    #pragma unroll
        for (int k = 0; k < kObjItems; ++k) {
            const unsigned i = tid + k * kObjThreads;
            val[k] = kNone;
            if (i < nrow) val[k] = min(A.off[o0 + 1 + i], A.R);
            else if (i < nrow + nref) val[k] = A.agents[r0 + (i - nrow)];
        }
        // one 64-bit word per reference: e = 0 if the agent is active, else 2 D + 1
        unsigned char act[kObjItems];
    #pragma unroll
        for (int k = 0; k < kObjItems; ++k) {
            const unsigned i = tid + k * kObjThreads;
            act[k] = 0;
            if (i >= nrow && i < nrow + nref) {
                const unsigned a = val[k];
                val[k] = kNone;
                if (a < A.N) {
                    const u64 e = A.w[a];
                    act[k] = e == 0;
                    val[k] = (unsigned)(e >> 1);
                }
            }
        }
    #pragma unroll
        for (int k = 0; k < kObjItems; ++k) {
            const unsigned i = tid + k * kObjThreads;
            if (i < nrow + nref) s_item[i] = val[k];
            if (i >= nrow && i < nrow + nref) s_flag[i] = act[k];
        }
        __syncthreads();

        // this thread's start on the block's merge path (binary search in LDS)
        const unsigned k0 = tid * (unsigned)kObjItems;
        const unsigned n_items = d1 - d0;
        const unsigned* s_val = s_item + nrow;
        const unsigned char* s_act = s_flag + nrow;
        unsigned char* s_outa = s_flag;
        unsigned o = 0, r = 0, vmin = kNone, vact = 0;
        if (k0 < n_items) {
            unsigned lo = k0 > nref ? k0 - nref : 0u, hi = min(k0, nrow);
            while (lo < hi) {
                const unsigned mid = (lo + hi) >> 1;
                if (s_item[mid] + mid + 1 > r0 + k0) hi = mid;
                else lo = mid + 1;
            }
            o = lo;
            r = k0 - lo;
            const unsigned k1 = min(k0 + (unsigned)kObjItems, n_items);
            for (unsigned k = k0; k < k1; ++k) {
                if (o < nrow && (s_item[o] <= r0 + r || r >= nref)) {     // row o ends here
                    s_outd[o] = vmin;
                    s_outa[o] = (unsigned char)vact;
                    vmin = kNone;
                    vact = 0;
                    ++o;
                } else if (r < nref) {
                    vmin = min(vmin, s_val[r]);
                    vact |= s_act[r];
                    ++r;
                }
            }
        }
        __syncthreads();
        // references of a row that ends in a later thread (or block)
        if (k0 < n_items && (vmin != kNone || vact)) {
            if (o < nrow) {
                atomicMin(&s_outd[o], vmin);
                if (vact) s_outa[o] = 1;
            } else {
                atomicMin(&s_bmin, vmin);
                if (vact) s_bact = 1;
            }
        }
        __syncthreads();
        for (unsigned i = tid; i < nrow; i += kObjThreads) {
            A.out_dist[o0 + i] = s_outd[i];
            A.out_act[o0 + i] = s_outa[i];
        }
        if (tid == 0) {
            ObjCarry c{kNone, kNone, 0u, 0u};
            if (o1 < A.M && (s_bmin != kNone || s_bact)) c = ObjCarry{o1, s_bmin, s_bact, 0u};
            A.carry[tile] = c;
        }
        __syncthreads();          // LDS is refilled by the next tile
    }
}

__global__ void __launch_bounds__(256) k_obj_fix(const ObjCarry* __restrict__ carry,
                                                unsigned n, unsigned M, unsigned* out_dist,
                                                unsigned char* out_act) {
    const unsigned i = blockIdx.x * 256u + threadIdx.x;
    if (i >= n) return;
    const ObjCarry c = carry[i];
    if (c.row >= M) return;
    atomicMin(&out_dist[c.row], c.vmin);
    if (c.act) out_act[c.row] = 1;
}

// ---------------------------------------------------------------------------
// Hop counts
// ---------------------------------------------------------------------------

constexpr int kBfsThreads = 256;
constexpr int kBfsEdges = 8;                 // edges claimed per vertex per round
constexpr int kBfsVerts = 2;                 // frontier vertices per thread per round
constexpr unsigned kBfsSpin = 1u << 24;      // barrier spin bound (about 0.5 s)

struct BfsArgs {
    const unsigned* row_off;                 // [V + 1]
    const unsigned* col;                     // [E]
    const unsigned* src;                     // [n_src]
    unsigned V, E, n_src, max_hops;
    unsigned* hops;                          // [V]
    uint2* q0;                               // [V] frontier queues: edge ranges
    uint2* q1;
    unsigned* ctl;                           // [8] see kCtl*
};
constexpr int kCtlCnt = 0;                   // [0..2] queue lengths, rotating
constexpr int kCtlBarCount = 3;              // grid barrier arrivals
constexpr int kCtlBarGen = 4;                // grid barrier generation
constexpr int kCtlError = 5;                 // 1 if a barrier wait hit its bound
constexpr int kCtlLevels = 6;                // levels expanded

// Grid-wide barrier for a cooperative launch (all workgroups resident).
// Thread 0 of each workgroup publishes the workgroup's writes with one
// agent-scope release fence and arrives on a counter; the last arrival bumps
// the generation word.  Waiters poll the generation with relaxed loads (an
// acquire per poll would invalidate the XCD's L2 each time) and take one
// acquire fence when it changes.  Returns false for every thread of a
// workgroup whose wait exceeded the bound; the caller then leaves the kernel,
// so every wave exits.
__device__ bool grid_barrier(unsigned* ctl) {
    __shared__ int s_ok;
    __syncthreads();
    if (threadIdx.x == 0) {
        int ok = 1;
        const unsigned gen = __hip_atomic_load(&ctl[kCtlBarGen], __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        const unsigned arrived = __hip_atomic_fetch_add(&ctl[kCtlBarCount], 1u, __ATOMIC_RELAXED,
                                                        __HIP_MEMORY_SCOPE_AGENT) + 1;
        if (arrived == gridDim.x) {
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "agent");
            __hip_atomic_store(&ctl[kCtlBarCount], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_fetch_add(&ctl[kCtlBarGen], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
            unsigned spin = 0;
            while (__hip_atomic_load(&ctl[kCtlBarGen], __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT) == gen) {
                if (++spin > kBfsSpin) {
                    ok = 0;
                    __hip_atomic_store(&ctl[kCtlError], 1u, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                __builtin_amdgcn_s_sleep(2);
            }
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        }
        s_ok = ok;
    }
    __syncthreads();
    return s_ok != 0;
}

// Append the lanes' claimed vertices (claim[k] for k < n) to queue q as their
// edge ranges [row_off[v], row_off[v + 1]), with one counter atomic per wave;
// the range loads and the counter atomic are in flight together.  Entries at
// or beyond `cap` are dropped (a vertex is claimed once, so a queue never
// holds more than the vertex count).  Called by every lane of the wave.
template <int n>
__device__ __forceinline__ void wave_append(const bool (&claim)[n], const unsigned (&v)[n],
                                            const BfsArgs& A, uint2* q, unsigned* cnt) {
    u64 m[n];
    unsigned total = 0;
#pragma unroll
    for (int k = 0; k < n; ++k) {
        m[k] = __ballot(claim[k]);
        total += __popcll(m[k]);
    }
    if (total == 0) return;
    uint2 r[n];
#pragma unroll
    for (int k = 0; k < n; ++k) {
        r[k] = make_uint2(0u, 0u);
        if (claim[k]) r[k] = make_uint2(min(A.row_off[v[k]], A.E), min(A.row_off[v[k] + 1], A.E));
    }
    unsigned base = 0;
    if (__lane_id() == 0)
        base = __hip_atomic_fetch_add(cnt, total, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    base = __shfl(base, 0);
#pragma unroll
    for (int k = 0; k < n; ++k) {
        const unsigned below = __builtin_amdgcn_mbcnt_hi((unsigned)(m[k] >> 32),
                                                         __builtin_amdgcn_mbcnt_lo((unsigned)m[k], 0u));
        if (claim[k] && base + below < A.V) q[base + below] = r[k];
        base += __popcll(m[k]);
    }
}

// Every vertex unvisited, counters and barrier words zero.
__global__ void __launch_bounds__(kBfsThreads) k_bfs_init(BfsArgs A) {
    const unsigned v = blockIdx.x * kBfsThreads + threadIdx.x;
    if (v < A.V) A.hops[v] = kNone;
    if (blockIdx.x == 0 && threadIdx.x < 8) A.ctl[threadIdx.x] = 0;
}

// Sources: hop 0, each vertex once, into the first queue.
__global__ void __launch_bounds__(kBfsThreads) k_bfs_src(BfsArgs A) {
    const unsigned i = blockIdx.x * kBfsThreads + threadIdx.x;
    bool claim[1] = {false};
    unsigned v[1] = {kNone};
    if (i < A.n_src) {
        v[0] = A.src[i];
        if (v[0] < A.V) claim[0] = atomicCAS(&A.hops[v[0]], kNone, 0u) == kNone;
    }
    wave_append(claim, v, A, A.q0, &A.ctl[kCtlCnt + 0]);
}

// The levels, in one cooperative launch.
__global__ void __launch_bounds__(kBfsThreads) k_bfs(BfsArgs A) {
    const unsigned lane = __lane_id();
    const unsigned gsz = gridDim.x * kBfsThreads;
    const unsigned wbase = blockIdx.x * kBfsThreads + (threadIdx.x & ~63u);   // wave's first thread
    for (unsigned level = 0;; ++level) {
        // ordered by the kernel start or the barrier's acquire fence; capped
        // at the queue length
        const unsigned n = min(__hip_atomic_load(&A.ctl[kCtlCnt + level % 3], __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT), A.V);
        if (n == 0 || level >= A.max_hops) break;
        if (blockIdx.x == 0 && threadIdx.x == 0) {
            __hip_atomic_store(&A.ctl[kCtlCnt + (level + 2) % 3], 0u, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&A.ctl[kCtlLevels], level + 1, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
        const uint2* cur = (level & 1) ? A.q1 : A.q0;
        uint2* nxt = (level & 1) ? A.q0 : A.q1;
        unsigned* cnt = &A.ctl[kCtlCnt + (level + 1) % 3];
        // Large frontiers first read a vertex's state and try to claim it only
        // while unvisited (fewer atomics); small ones go straight to the
        // compare-and-swap (one dependent access less per level).
        const bool precheck = n > 32768u;
        // each lane expands kBfsVerts frontier vertices per round, eight of
        // their edges at a time, so that many independent loads are in flight
        for (unsigned b0 = wbase * kBfsVerts; b0 < n; b0 += gsz * kBfsVerts) {
            unsigned e[kBfsVerts], e1[kBfsVerts];
#pragma unroll
            for (int f = 0; f < kBfsVerts; ++f) {
                const unsigned i = b0 + f * 64u + lane;
                const uint2 r = i < n ? cur[i] : make_uint2(0u, 0u);
                e[f] = r.x;
                e1[f] = min(r.y, A.E);
            }
            bool more = false;
#pragma unroll
            for (int f = 0; f < kBfsVerts; ++f) more |= e[f] < e1[f];
            while (__ballot(more)) {
                unsigned v[kBfsVerts * kBfsEdges];
                bool claim[kBfsVerts * kBfsEdges];
#pragma unroll
                for (int f = 0; f < kBfsVerts; ++f)
#pragma unroll
                    for (int k = 0; k < kBfsEdges; ++k)
                        v[f * kBfsEdges + k] = e[f] + k < e1[f] ? A.col[e[f] + k] : kNone;
#pragma unroll
                for (int k = 0; k < kBfsVerts * kBfsEdges; ++k)
                    claim[k] = v[k] < A.V && (!precheck || A.hops[v[k]] == kNone);
#pragma unroll
                for (int k = 0; k < kBfsVerts * kBfsEdges; ++k)
                    if (claim[k]) claim[k] = atomicCAS(&A.hops[v[k]], kNone, level + 1) == kNone;
                wave_append(claim, v, A, nxt, cnt);
                more = false;
#pragma unroll
                for (int f = 0; f < kBfsVerts; ++f) {
                    e[f] += kBfsEdges;
                    more |= e[f] < e1[f];
                }
            }
        }
        if (!grid_barrier(A.ctl)) return;
    }
}

// ---------------------------------------------------------------------------
// Interaction distances
// ---------------------------------------------------------------------------

constexpr int kPairThreads = 256;            // agents i per workgroup
constexpr int kPairTile = 256;               // agents j staged per LDS round

typedef short short2_t __attribute__((ext_vector_type(2)));

// Squared distance of two grid points held as packed 16-bit (x, y): one packed
// subtract and one 16-bit dot product (coordinates below 2^15, so neither the
// differences nor the sum of squares overflow).  The dot product is written
// in its three-operand form with a zero addend; the compiler's two-operand
// form would need a register cleared before every pair.
__device__ __forceinline__ unsigned dist2(short2_t a, short2_t b) {
    const short2_t d = a - b;
    int r;
    asm("v_dot2_i32_i16 %0, %1, %1, 0" : "=v"(r) : "v"(d));
    return (unsigned)r;
}

// Partial minimum of the squared distance from each agent i of the workgroup
// to the agents j of slice [j_lo, j_hi), excluding j = i, into d2min[i].
__global__ void __launch_bounds__(kPairThreads) k_pair_min(const int* __restrict__ pos,
                                                           unsigned n, unsigned slice,
                                                           unsigned* __restrict__ d2min) {
    __shared__ __attribute__((aligned(16))) short2_t s_p[kPairTile];
    const unsigned i = blockIdx.x * kPairThreads + threadIdx.x;
    const unsigned j_lo = blockIdx.y * slice, j_hi = min(j_lo + slice, n);
    short2_t pi = {0, 0};
    if (i < n) pi = short2_t{(short)pos[2 * i], (short)pos[2 * i + 1]};
    unsigned best = kNone;
    // the next tile's position is loaded while the current tile is compared
    int2 nxt = make_int2(0, 0);
    if (j_lo + threadIdx.x < j_hi)
        nxt = make_int2(pos[2 * (j_lo + threadIdx.x)], pos[2 * (j_lo + threadIdx.x) + 1]);
    for (unsigned j0 = j_lo; j0 < j_hi; j0 += kPairTile) {
        const unsigned j = j0 + threadIdx.x;
        if (j < j_hi) s_p[threadIdx.x] = short2_t{(short)nxt.x, (short)nxt.y};
        __syncthreads();
        if (j + kPairTile < j_hi) nxt = make_int2(pos[2 * (j + kPairTile)], pos[2 * (j + kPairTile) + 1]);
        const unsigned cnt = min((unsigned)kPairTile, j_hi - j0);
        if (i - j0 < cnt) {                  // this tile holds i itself: skip the self pair
            for (unsigned k = 0; k < cnt; ++k)
                if (j0 + k != i) best = min(best, dist2(pi, s_p[k]));
        } else if (cnt == kPairTile) {
            // four positions per 16-byte LDS read (a broadcast: every lane reads
            // the same address), so the LDS issues a quarter of the reads
            const uint4* q = reinterpret_cast<const uint4*>(s_p);
#pragma unroll 8
            for (unsigned k = 0; k < kPairTile / 4; ++k) {
                const uint4 v = q[k];
                best = min(best, dist2(pi, __builtin_bit_cast(short2_t, v.x)));
                best = min(best, dist2(pi, __builtin_bit_cast(short2_t, v.y)));
                best = min(best, dist2(pi, __builtin_bit_cast(short2_t, v.z)));
                best = min(best, dist2(pi, __builtin_bit_cast(short2_t, v.w)));
            }
        } else {
            for (unsigned k = 0; k < cnt; ++k) best = min(best, dist2(pi, s_p[k]));
        }
        __syncthreads();
    }
    if (i < n && best != kNone) atomicMin(&d2min[i], best);
}

__global__ void __launch_bounds__(256) k_pair_init(unsigned* d2min, unsigned n) {
    const unsigned i = blockIdx.x * 256u + threadIdx.x;
    if (i < n) d2min[i] = kNone;
}

__device__ __forceinline__ unsigned isqrt_u32(unsigned x) {
    unsigned r = (unsigned)sqrt((double)x);
    while ((u64)r * r > x) --r;
    while ((u64)(r + 1) * (r + 1) <= x) ++r;
    return r;
}

__global__ void __launch_bounds__(256) k_pair_fin(const unsigned* __restrict__ d2min,
                                                  const unsigned* __restrict__ d_action,
                                                  unsigned n, unsigned velocity, unsigned radius,
                                                  unsigned* __restrict__ out) {
    const unsigned i = blockIdx.x * 256u + threadIdx.x;
    if (i >= n) return;
    unsigned d = d_action[i];
    const unsigned m = d2min[i];
    if (m != kNone) {
        const unsigned dist = isqrt_u32(m);
        d = min(d, (dist > radius ? dist - radius : 0u) / velocity);
    }
    out[i] = d;
}

inline unsigned obj_blocks(unsigned M, unsigned R) {
    return (unsigned)(((u64)M + R + kObjTile - 1) / kObjTile);
}

}  // namespace
}  // namespace ss

using namespace ss;

extern "C" {

uint64_t ss_object_distances_workspace(uint32_t n_objects, uint32_t n_refs, uint32_t n_agents) {
    const u64 blocks = obj_blocks(n_objects, n_refs);
    return blocks * sizeof(ObjCarry) + ((blocks + 1 + 3) & ~3ull) * 4 + (u64)n_agents * 8;
}

}  // extern "C"

namespace {

// Checks the arguments of ss_object_distances and fills the kernel arguments.
ss_status object_args(const uint32_t* obj_off, const uint32_t* obj_agents, uint32_t n_objects,
                      uint32_t n_refs, const uint32_t* distances, const uint8_t* active,
                      uint32_t n_agents, uint32_t* obj_distances, uint8_t* obj_active,
                      void* workspace, uint64_t workspace_bytes, ObjArgs* A) {
    if (n_objects >= (1u << 31) || n_refs >= (1u << 31))
        return set_err(SS_ERR_ARG, "n_objects and n_refs must be below 2^31");
    if (!obj_off || !obj_distances || !obj_active || !workspace ||
        (n_refs && !obj_agents) || (n_agents && (!distances || !active)))
        return set_err(SS_ERR_ARG, "NULL argument");
    const u64 need = ss_object_distances_workspace(n_objects, n_refs, n_agents);
    if (workspace_bytes < need)
        return set_err(SS_ERR_ARG, "workspace_bytes %llu < %llu", (unsigned long long)workspace_bytes,
                       (unsigned long long)need);
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return set_err(SS_ERR_ARG, "no current device");
    }
    if (!device_range_ok(obj_off, ((u64)n_objects + 1) * 4, dev) ||
        (n_refs && !device_range_ok(obj_agents, (u64)n_refs * 4, dev)) ||
        (n_agents && (!device_range_ok(distances, (u64)n_agents * 4, dev) ||
                      !device_range_ok(active, n_agents, dev))) ||
        !device_range_ok(obj_distances, (u64)n_objects * 4, dev) ||
        !device_range_ok(obj_active, n_objects, dev) ||
        !device_range_ok(workspace, need, dev))
        return set_err(SS_ERR_ARG, "every array must be device memory of the current device (%d)",
                       dev);
    A->off = obj_off;
    A->agents = obj_agents;
    A->dist = distances;
    A->active = active;
    A->M = n_objects;
    A->R = n_refs;
    A->N = n_agents;
    A->out_dist = obj_distances;
    A->out_act = obj_active;
    const u64 blocks = obj_blocks(n_objects, n_refs);
    A->carry = static_cast<ObjCarry*>(workspace);
    A->coord = reinterpret_cast<unsigned*>(A->carry + blocks);
    A->w = reinterpret_cast<u64*>(A->coord + ((blocks + 1 + 3) & ~3ull));
    return SS_OK;
}

hipError_t object_launch(const ObjArgs& A, hipStream_t st) {
    const unsigned blocks = obj_blocks(A.M, A.R);
    const unsigned part_blocks = (blocks + 1 + 15) / 16;
    const unsigned pack_blocks = (unsigned)std::min<u64>(((u64)A.N + 2047) / 2048, 1024);
    hipLaunchKernelGGL(k_obj_prep, dim3(part_blocks + pack_blocks), dim3(256), 0, st, A,
                       blocks + 1, part_blocks);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        cus = 256;
    // eight resident workgroups per CU (LDS and registers allow eight)
    const unsigned grid = (unsigned)std::min<u64>(((u64)blocks + 7) / 8 * 8,
                                                  (u64)std::max(cus, 8) / 8 * 8 * 8);
    hipLaunchKernelGGL(k_obj_min, dim3(grid), dim3(kObjThreads), 0, st, A, blocks);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_obj_fix, dim3((blocks + 255) / 256), dim3(256), 0, st, A.carry, blocks,
                       A.M, A.out_dist, A.out_act);
    return hipGetLastError();
}

}  // namespace

extern "C" {

ss_status ss_object_distances(const uint32_t* obj_off, const uint32_t* obj_agents,
                              uint32_t n_objects, uint32_t n_refs, const uint32_t* distances,
                              const uint8_t* active, uint32_t n_agents, uint32_t* obj_distances,
                              uint8_t* obj_active, void* workspace, uint64_t workspace_bytes,
                              void* stream) {
    if (n_objects == 0 && n_refs < (1u << 31)) return SS_OK;
    ObjArgs A;
    ss_status st = object_args(obj_off, obj_agents, n_objects, n_refs, distances, active,
                               n_agents, obj_distances, obj_active, workspace, workspace_bytes, &A);
    if (st != SS_OK) return st;
    hipError_t e = object_launch(A, static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return set_err(SS_ERR_HIP, "object distance kernels: %s", hipGetErrorString(e));
    return SS_OK;
}

ss_status ss_probe_object_distances(const uint32_t* obj_off, const uint32_t* obj_agents,
                                    uint32_t n_objects, uint32_t n_refs,
                                    const uint32_t* distances, const uint8_t* active,
                                    uint32_t n_agents, uint32_t* obj_distances,
                                    uint8_t* obj_active, void* workspace,
                                    uint64_t workspace_bytes, int iters, float* ms_per_iter) {
    if (iters < 1 || !ms_per_iter || n_objects == 0)
        return set_err(SS_ERR_ARG, "bad probe arguments");
    ObjArgs A;
    ss_status st = object_args(obj_off, obj_agents, n_objects, n_refs, distances, active,
                               n_agents, obj_distances, obj_active, workspace, workspace_bytes, &A);
    if (st != SS_OK) return st;
    hipEvent_t a = nullptr, b = nullptr;
    hipStream_t s = nullptr;
    hipError_t e = hipEventCreate(&a);
    if (e == hipSuccess) e = hipEventCreate(&b);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
    if (e == hipSuccess) e = object_launch(A, s);                  // warm-up
    if (e == hipSuccess) e = hipEventRecord(a, s);
    for (int i = 0; i < iters && e == hipSuccess; ++i) e = object_launch(A, s);
    if (e == hipSuccess) e = hipEventRecord(b, s);
    if (e == hipSuccess) e = hipEventSynchronize(b);
    float t = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&t, a, b);
    if (s) (void)hipStreamDestroy(s);
    if (a) (void)hipEventDestroy(a);
    if (b) (void)hipEventDestroy(b);
    if (e != hipSuccess) return set_err(SS_ERR_HIP, "object distance probe: %s", hipGetErrorString(e));
    *ms_per_iter = t / iters;
    return SS_OK;
}

uint64_t ss_hop_distances_workspace(uint32_t n_vertices) {
    return 64 + 2 * (((uint64_t)n_vertices * 8 + 255) & ~255ull);
}

ss_status ss_hop_distances(const uint32_t* row_off, const uint32_t* col, uint32_t n_vertices,
                           uint32_t n_edges, const uint32_t* sources, uint32_t n_sources,
                           uint32_t max_hops, uint32_t* hops, void* workspace,
                           uint64_t workspace_bytes, void* stream) {
    if (n_vertices >= (1u << 31) || n_edges >= (1u << 31))
        return set_err(SS_ERR_ARG, "n_vertices and n_edges must be below 2^31");
    if (n_vertices == 0) return SS_OK;
    if (!row_off || !hops || !workspace || (n_edges && !col) || (n_sources && !sources))
        return set_err(SS_ERR_ARG, "NULL argument");
    const u64 need = ss_hop_distances_workspace(n_vertices);
    if (workspace_bytes < need)
        return set_err(SS_ERR_ARG, "workspace_bytes %llu < %llu", (unsigned long long)workspace_bytes,
                       (unsigned long long)need);
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return set_err(SS_ERR_ARG, "no current device");
    }
    if (!device_range_ok(row_off, ((u64)n_vertices + 1) * 4, dev) ||
        (n_edges && !device_range_ok(col, (u64)n_edges * 4, dev)) ||
        (n_sources && !device_range_ok(sources, (u64)n_sources * 4, dev)) ||
        !device_range_ok(hops, (u64)n_vertices * 4, dev) || !device_range_ok(workspace, need, dev))
        return set_err(SS_ERR_ARG, "every array must be device memory of the current device (%d)",
                       dev);
    int coop = 0, cus = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess ||
        !coop || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(k_bfs),
                                                     kBfsThreads, 0) != hipSuccess || per_cu < 1) {
        (void)hipGetLastError();
        return set_err(SS_ERR_HIP, "cooperative launch is not available on device %d", dev);
    }
    BfsArgs A;
    A.row_off = row_off;
    A.col = col;
    A.src = sources;
    A.V = n_vertices;
    A.E = n_edges;
    A.n_src = n_sources;
    A.max_hops = max_hops;
    A.hops = hops;
    char* ws = static_cast<char*>(workspace);
    A.ctl = reinterpret_cast<unsigned*>(ws);
    const u64 qbytes = ((u64)n_vertices * 8 + 255) & ~255ull;
    A.q0 = reinterpret_cast<uint2*>(ws + 64);
    A.q1 = reinterpret_cast<uint2*>(ws + 64 + qbytes);
    // one workgroup per 512 vertices, at most one per CU: every workgroup
    // pays an L2 write-back and invalidate at each grid barrier, so fewer,
    // wider workgroups (two vertices per thread per round) are cheaper
    const u64 want = ((u64)n_vertices + kBfsThreads * kBfsVerts - 1) / (kBfsThreads * kBfsVerts);
    const unsigned grid = (unsigned)std::max<u64>(1, std::min<u64>(want, (u64)cus));
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(k_bfs_init, dim3((n_vertices + kBfsThreads - 1) / kBfsThreads),
                       dim3(kBfsThreads), 0, st, A);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && n_sources) {
        hipLaunchKernelGGL(k_bfs_src, dim3((n_sources + kBfsThreads - 1) / kBfsThreads),
                           dim3(kBfsThreads), 0, st, A);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        void* args[] = {&A};
        e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(k_bfs), dim3(grid),
                                       dim3(kBfsThreads), args, 0, st);
    }
    if (e != hipSuccess) return set_err(SS_ERR_HIP, "hop distance kernels: %s", hipGetErrorString(e));
    return SS_OK;
}

uint64_t ss_interaction_distances_workspace(uint32_t n_agents) { return (uint64_t)n_agents * 4; }

}  // extern "C"

// Partial minima of ss_interaction_distances_static (4 MiB): one array per
// device, held from the library's load until the process ends, shared by
// every call on that device.  Host code never uses its name as an address:
// the device address is looked up once per device (scratch_addr) and kept.
static __device__ __align__(256) unsigned scratch[1u << 20];

namespace {

// Checks the arrays of an interaction-distance call (not its workspace) and
// returns the current device in *dev.
ss_status interaction_args(const int32_t* pos_xy, const uint32_t* d_action, uint32_t n_agents,
                           uint32_t velocity, const uint32_t* out, int* dev) {
    if (n_agents >= (1u << 31)) return set_err(SS_ERR_ARG, "n_agents must be below 2^31");
    if (velocity == 0) return set_err(SS_ERR_ARG, "velocity must be >= 1");
    if (n_agents == 0) return SS_OK;
    if (!pos_xy || !d_action || !out) return set_err(SS_ERR_ARG, "NULL argument");
    if (hipGetDevice(dev) != hipSuccess) {
        (void)hipGetLastError();
        return set_err(SS_ERR_ARG, "no current device");
    }
    if (!device_range_ok(pos_xy, (u64)n_agents * 8, *dev) ||
        !device_range_ok(d_action, (u64)n_agents * 4, *dev) ||
        !device_range_ok(out, (u64)n_agents * 4, *dev))
        return set_err(SS_ERR_ARG, "every array must be device memory of the current device (%d)",
                       *dev);
    return SS_OK;
}

// The three interaction kernels on `st`, with d2min [n_agents] as the
// partial minima (cleared by the first kernel).
ss_status interaction_launch(const int32_t* pos_xy, const uint32_t* d_action, uint32_t n_agents,
                             uint32_t velocity, uint32_t radius, uint32_t* out, unsigned* d2min,
                             int dev, hipStream_t st) {
    int cus = 256;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) cus = 256;
    const unsigned iblocks = (n_agents + kPairThreads - 1) / kPairThreads;
    // split the other agents into slices so that about 8 workgroups run per CU
    const unsigned want = (unsigned)std::max<u64>(1, (u64)cus * 8 / iblocks);
    const unsigned tiles = (n_agents + kPairTile - 1) / kPairTile;
    const unsigned slices = std::min(want, tiles);
    const unsigned slice = (tiles + slices - 1) / slices * kPairTile;
    const unsigned nslice = (n_agents + slice - 1) / slice;
    const unsigned b256 = (n_agents + 255) / 256;
    hipLaunchKernelGGL(k_pair_init, dim3(b256), dim3(256), 0, st, d2min, n_agents);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) {
        hipLaunchKernelGGL(k_pair_min, dim3(iblocks, nslice), dim3(kPairThreads), 0, st, pos_xy,
                           n_agents, slice, d2min);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        hipLaunchKernelGGL(k_pair_fin, dim3(b256), dim3(256), 0, st, d2min, d_action, n_agents,
                           velocity, radius, out);
        e = hipGetLastError();
    }
    if (e != hipSuccess)
        return set_err(SS_ERR_HIP, "interaction distance kernels: %s", hipGetErrorString(e));
    return SS_OK;
}

constexpr uint32_t kStaticPairAgents = 1u << 20;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
unsigned* g_scratch_addr[kMaxDevices] = {};

// Device address of `scratch` on device `dev` (current), looked up on the
// first call per device.
ss_status scratch_addr(int dev, unsigned** out) {
    if (dev < 0 || dev >= kMaxDevices) return set_err(SS_ERR_ARG, "device %d out of range", dev);
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_addr[dev]) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr)
            return set_err(SS_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                           hipGetErrorString(e));
        g_scratch_addr[dev] = static_cast<unsigned*>(ptr);
    }
    *out = g_scratch_addr[dev];
    return SS_OK;
}

}  // namespace

extern "C" {

ss_status ss_interaction_distances(const int32_t* pos_xy, const uint32_t* d_action,
                                   uint32_t n_agents, uint32_t velocity, uint32_t radius,
                                   uint32_t* out, void* workspace, uint64_t workspace_bytes,
                                   void* stream) {
    int dev = -1;
    ss_status st = interaction_args(pos_xy, d_action, n_agents, velocity, out, &dev);
    if (st != SS_OK || n_agents == 0) return st;
    if (!workspace) return set_err(SS_ERR_ARG, "NULL argument");
    const u64 need = ss_interaction_distances_workspace(n_agents);
    if (workspace_bytes < need)
        return set_err(SS_ERR_ARG, "workspace_bytes %llu < %llu", (unsigned long long)workspace_bytes,
                       (unsigned long long)need);
    if (!device_range_ok(workspace, need, dev))
        return set_err(SS_ERR_ARG, "every array must be device memory of the current device (%d)",
                       dev);
    return interaction_launch(pos_xy, d_action, n_agents, velocity, radius, out,
                              static_cast<unsigned*>(workspace), dev,
                              static_cast<hipStream_t>(stream));
}

ss_status ss_interaction_distances_static(const int32_t* pos_xy, const uint32_t* d_action,
                                          uint32_t n_agents, uint32_t velocity, uint32_t radius,
                                          uint32_t* out, void* stream) {
    static_assert(sizeof(scratch) == kStaticPairAgents * sizeof(unsigned), "scratch size");
    if (n_agents > kStaticPairAgents)
        return set_err(SS_ERR_ARG, "n_agents %u exceeds the %u agents of the static scratch "
                                   "(use ss_interaction_distances with a workspace)",
                       n_agents, kStaticPairAgents);
    int dev = -1;
    ss_status st = interaction_args(pos_xy, d_action, n_agents, velocity, out, &dev);
    if (st != SS_OK || n_agents == 0) return st;
    unsigned* d2min = nullptr;
    st = scratch_addr(dev, &d2min);
    if (st != SS_OK) return st;
    return interaction_launch(pos_xy, d_action, n_agents, velocity, radius, out, d2min, dev,
                              static_cast<hipStream_t>(stream));
}

}  // extern "C"
