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
//   k_obj_min   per workgroup: a 64-ary wave search of its two merge-path
//               coordinates in global memory, coalesced staging of its row
//               ends and of v/active of its references into LDS (the gather
//               of the agents' distances happens here, once per reference),
//               an 8-item walk per thread, LDS atomics for rows split between
//               threads, coalesced stores of the rows that end in the block
//               and one carry record for the row that continues past it.
//   k_obj_fix   applies the carry records with global atomic min / stores,
//               after every k_obj_min block has written its rows.
// No dense contraction here; the kernel is bound by HBM bytes.
#include "scalesim.h"
#include "ss_internal.h"

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
};

// Row ends consumed at merge diagonal d: the first p in [max(0, d - R),
// min(d, M)) whose row end comes after reference d - p - 1, i.e.
// off[p + 1] + p + 1 > d (a strictly increasing function of p), else the
// upper bound.  64 probes per round, so a few dependent loads per search.
__device__ unsigned wave_path_search(const unsigned* __restrict__ off, unsigned M, unsigned R,
                                     unsigned d) {
    const unsigned lane = __lane_id();
    unsigned lo = d > R ? d - R : 0u;
    unsigned hi = d < M ? d : M;
    while (lo < hi) {
        const unsigned step = (hi - lo + 63u) / 64u;
        const unsigned p = lo + lane * step;
        bool after = false;
        if (p < hi) {
            const unsigned e = min(off[p + 1], R);
            after = (unsigned long long)e + p + 1 > d;
        }
        const unsigned long long m = __ballot(after);
        if (m == 0) {
            const unsigned n_probe = (hi - lo + step - 1) / step;   // lanes with p < hi
            lo = lo + (n_probe - 1) * step + 1;
        } else {
            const unsigned f = __ffsll((long long)m) - 1;
            hi = lo + f * step;
            if (f > 0) lo = lo + (f - 1) * step + 1;
        }
    }
    return lo;
}

__global__ void __launch_bounds__(kObjThreads) k_obj_min(ObjArgs A) {
    __shared__ unsigned s_end[kObjTile];      // absolute row ends of the block's rows
    __shared__ unsigned s_val[kObjTile];      // v of the block's references
    __shared__ unsigned s_outd[kObjTile];     // rows ending in the block: min
    __shared__ unsigned char s_act[kObjTile];
    __shared__ unsigned char s_outa[kObjTile];
    __shared__ unsigned s_coord[2];
    __shared__ unsigned s_bmin, s_bact;

    const unsigned tid = threadIdx.x;
    const unsigned total = A.M + A.R;
    const unsigned d0 = blockIdx.x * (unsigned)kObjTile;
    const unsigned d1 = min(d0 + (unsigned)kObjTile, total);
    const unsigned wave = tid >> 6;
    if (wave < 2) {
        const unsigned x = wave_path_search(A.off, A.M, A.R, wave ? d1 : d0);
        if (__lane_id() == 0) s_coord[wave] = x;
    }
    if (tid == 0) {
        s_bmin = kNone;
        s_bact = 0;
    }
    __syncthreads();
    const unsigned o0 = s_coord[0], o1 = s_coord[1];
    const unsigned r0 = d0 - o0, r1 = d1 - o1;
    const unsigned nrow = o1 - o0, nref = r1 - r0;

    for (unsigned i = tid; i < nrow; i += kObjThreads) s_end[i] = min(A.off[o0 + 1 + i], A.R);
    for (unsigned i = tid; i < nref; i += kObjThreads) {
        const unsigned a = A.agents[r0 + i];
        unsigned v = kNone, act = 0;
        if (a < A.N) {
            act = A.active[a] != 0;
            v = act ? 0u : A.dist[a];
        }
        s_val[i] = v;
        s_act[i] = (unsigned char)act;
    }
    __syncthreads();

    // this thread's start on the block's merge path (binary search in LDS)
    const unsigned k0 = tid * (unsigned)kObjItems;
    const unsigned n_items = d1 - d0;
    unsigned o = 0, r = 0, vmin = kNone, vact = 0;
    if (k0 < n_items) {
        unsigned lo = k0 > nref ? k0 - nref : 0u, hi = min(k0, nrow);
        while (lo < hi) {
            const unsigned mid = (lo + hi) >> 1;
            if (s_end[mid] + mid + 1 > r0 + k0) hi = mid;
            else lo = mid + 1;
        }
        o = lo;
        r = k0 - lo;
        const unsigned k1 = min(k0 + (unsigned)kObjItems, n_items);
        for (unsigned k = k0; k < k1; ++k) {
            if (o < nrow && (s_end[o] <= r0 + r || r >= nref)) {      // row o ends here
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
        A.carry[blockIdx.x] = c;
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

uint64_t ss_object_distances_workspace(uint32_t n_objects, uint32_t n_refs) {
    return (uint64_t)obj_blocks(n_objects, n_refs) * sizeof(ObjCarry);
}

ss_status ss_object_distances(const uint32_t* obj_off, const uint32_t* obj_agents,
                              uint32_t n_objects, uint32_t n_refs, const uint32_t* distances,
                              const uint8_t* active, uint32_t n_agents, uint32_t* obj_distances,
                              uint8_t* obj_active, void* workspace, uint64_t workspace_bytes,
                              void* stream) {
    if (n_objects >= (1u << 31) || n_refs >= (1u << 31))
        return set_err(SS_ERR_ARG, "n_objects and n_refs must be below 2^31");
    if (n_objects == 0) return SS_OK;
    if (!obj_off || !obj_distances || !obj_active || !workspace ||
        (n_refs && !obj_agents) || (n_agents && (!distances || !active)))
        return set_err(SS_ERR_ARG, "NULL argument");
    const u64 need = ss_object_distances_workspace(n_objects, n_refs);
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
    ObjArgs A;
    A.off = obj_off;
    A.agents = obj_agents;
    A.dist = distances;
    A.active = active;
    A.M = n_objects;
    A.R = n_refs;
    A.N = n_agents;
    A.out_dist = obj_distances;
    A.out_act = obj_active;
    A.carry = static_cast<ObjCarry*>(workspace);
    const unsigned blocks = obj_blocks(n_objects, n_refs);
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(k_obj_min, dim3(blocks), dim3(kObjThreads), 0, st, A);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) {
        hipLaunchKernelGGL(k_obj_fix, dim3((blocks + 255) / 256), dim3(256), 0, st, A.carry,
                           blocks, n_objects, obj_distances, obj_active);
        e = hipGetLastError();
    }
    if (e != hipSuccess)
        return set_err(SS_ERR_HIP, "object distance kernels: %s", hipGetErrorString(e));
    return SS_OK;
}

}  // extern "C"
