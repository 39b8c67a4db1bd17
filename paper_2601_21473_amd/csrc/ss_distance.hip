// Distance kernels for gfx950: invocation distances of shared memory objects.
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
// No dense contraction here; the kernel is bound by HBM bytes.
#include "scalesim.h"
#include "ss_internal.h"

#include <algorithm>

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

}  // extern "C"
