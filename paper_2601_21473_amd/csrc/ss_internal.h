// Declarations shared by the device kernels (ss_kernels.hip), the host
// library (ss_pool.hip) and the distance kernels (ss_distance.hip).  Internal
// to libscalesim.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "scalesim.h"

namespace ss {

typedef unsigned long long u64;

// Prefetch candidates are listed in kCandLists sub-lists by distance range:
// sub-list k holds the candidates whose distance bucket (dist_bucket below)
// lies in [cand_list_start(k), cand_list_start(k + 1)), so a plan that can
// accept only near candidates reads only the first sub-lists.
constexpr unsigned kCandLists = 8;
__host__ __device__ inline unsigned cand_list(unsigned bucket) {
    if (bucket < 4u) return 0u;
    if (bucket < 64u) return (31u - (unsigned)__builtin_clz(bucket)) - 1u;   // 4, 8, 16, 32 ...
    if (bucket < 256u) return 5u;
    if (bucket < 1024u) return 6u;
    return 7u;
}
__host__ __device__ inline unsigned cand_list_start(unsigned k) {   // 0 4 8 16 32 64 256 1024
    return k == 0 ? 0u : k <= 5 ? (2u << k) : k == 6 ? 256u : 1024u;
}

// Per-step accumulators written by the classify kernel.  The plan-core
// kernel consumes and re-zeroes them, so they are zero between steps.
struct PlanCounters {
    u64 sum_active;      // units of active agents
    u64 sum_resident;    // units of resident agents
    u64 sum_demand;      // units of active, non-resident agents
    u64 sum_evictable;   // units of inactive, resident agents
    u64 sum_cand;        // units of prefetch candidates
    unsigned n_E, n_L;
    unsigned n_C[kCandLists];   // candidates per distance sub-list
};

// Outcome of a plan, written by the plan-core kernel to device memory and to
// a mapped pinned host mirror.
struct PlanResult {
    int status;                 // 0 ok, 1 overcommit (nothing changed)
    unsigned n_victims, n_loads, n_demand, n_demand_victims, pad;
    u64 units_out, units_in;
    u64 free_before;            // free units before the step
    u64 n_free_used;            // loads' units taken from the pre-step free units
    u64 units_written;          // victims' units written back
};

// One wave-sized piece of a unit: `len` bytes of plane `plane`, starting at
// `chunk_off` inside the plane's chunk and at `unit_off` inside the unit's
// serialised bytes (planes concatenated in order).
struct CopyItem {
    unsigned plane;
    unsigned len;
    u64 chunk_off;
    u64 unit_off;
};

struct BtArgs {
    const PlanResult* res;
    const unsigned* victims;
    const unsigned* loads;
    const unsigned* units;          // s[a]
    const u64* agent_off;           // [N+1] block-table CSR offsets
    int* bt;                        // [sum s]
    unsigned* occ;
    const u64* voff;                // = prefE: prefix units over victims
    const u64* loff;
    const int* free_old;
    int* vunits;                    // [U] victims' old units, victim then j order
    int* lunits;                    // [U] loads' new units, load then j order
    u64 capacity;                   // U
    const unsigned char* vwritten;  // [N] per victim: written back
    const u64* woff;                // [N+1] prefix units over written-back victims
    int* wunits;                    // [U] written-back victims' units (pack source)
    const u64* host_off;            // [N] host-copy byte offset per agent (direct mode, else null)
    u64 unit_bytes;
    u64* whost;                     // [U] host byte offset of each written-back unit (or null)
    u64* lhost;                     // [U] host byte offset of each loaded unit (or null)
    u64* rhost;                     // [U] per released position: the host byte offset of
                                    // its unit when written back, else ~0 (or null)
    unsigned* wrel;                 // [U] per written-back position: its released position
                                    // (or null)
};

struct PlanArgs {
    const unsigned* dist;           // [N] caller distances (device, or mapped pinned mirror)
    const unsigned char* active;    // [N] caller mask (device, or mapped pinned mirror)
    unsigned char* resident;        // [N] state
    const unsigned* units;          // [N] s[a]
    unsigned n;
    unsigned idbits;                // key = (d << idbits) | id
    unsigned threshold;
    unsigned smax;                  // largest agent size in units (pool constant)
    u64 budget;
    u64 capacity;
    PlanCounters* cnt;
    u64* listE;                     // [N] unsorted keys from classify
    u64* listC;                     // [kCandLists][N] candidate sub-lists by distance range
    u64* listL;
    u64* sortE;                     // [pow2 >= N] sorted keys (ascending), also global sort scratch
    u64* sortC;
    u64* sortL;
    u64* prefE;                     // [N+1] prefix units over E in eviction (descending) order
    u64* prefC;                     // [N+1] prefix units over selected candidates (ascending)
    u64* loff;                      // [N+1] prefix units over loads
    unsigned* victims;              // [N] device copy of the plan
    unsigned* loads;                // [N]
    unsigned* occ;                  // occupancy bitmap, bit u = unit u in use
    unsigned occ_words;
    unsigned pad1;
    int* free_old;                  // [U] pre-step free units, ascending
    PlanResult* res;                // device
    PlanResult* res_host;           // mapped pinned host
    unsigned* victims_host;         // mapped pinned host [N]
    unsigned* loads_host;           // mapped pinned host [N]
    unsigned fused;                 // 1: the plan core classifies the agents itself
    unsigned pad2;
    u64* phase;                     // [kPlanPhases] wall-clock stamps of the plan core, or null
    u64* hist_w;                    // [kDistBuckets] candidate units per distance bucket
    unsigned* hist_e;               // [kDistBuckets] evictable residents' units per bucket
                                    // (both global: multi-workgroup classification only)
    const unsigned char* dirty;     // [N] optional write-back mask (device, or mapped mirror)
    unsigned char* vwritten;        // [N] per victim: written back (device)
    unsigned char* vwritten_host;   // mapped pinned host [N]
    u64* woff;                      // [N+1] prefix units over written-back victims
    unsigned* done;                 // workgroups of k_classify_core finished (0 between steps)
    unsigned* flag_host;            // mapped pinned host word: `seq` is written there last
    unsigned seq;                   // this plan's sequence number (never 0)
    unsigned pad3;
    const BtArgs* bt;               // block-table update (device copy), run in the core's tail
};

// Candidate distance histogram: bucket(d) = d below 1024, then 32 buckets per
// power of two (monotone in d).
constexpr unsigned kDistBuckets = 2048;
__host__ __device__ inline unsigned dist_bucket(unsigned d) {
    if (d < 1024u) return d;
    const unsigned p = 31u - (unsigned)__builtin_clz(d);
    return 1024u + 32u * (p - 10u) + ((d >> (p - 5u)) & 31u);
}

constexpr int kPlanPhases = 10;


struct CopyArgs {
    const int* units_list;          // vunits (pack) or lunits (unpack)
    u64 first;                      // first position in units_list
    u64 count;                      // units in this launch
    const CopyItem* items;
    unsigned n_items;               // items per unit
    unsigned item_groups;           // ceil(n_items / kCopyWavesPerBlock) blocks per unit
    unsigned run_order;             // unpack: one block per (item, 8 consecutive units)
    unsigned pad1;
    const u64* plane_base;          // [P] device addresses
    const u64* chunk_bytes;         // [P]
    char* staging;                  // slot base (direct: device address of the host copies)
    const u64* stage_off;           // direct: [first + p] byte offset of logical unit p from
                                    // staging; null: unit p at staging + p * unit_bytes
    u64 unit_bytes;
    u64 capacity;                   // U; unit ids outside [0, U) are skipped
};

constexpr int kCopyThreads = 512;                 // 8 waves, one item per wave
constexpr int kCopyWavesPerBlock = kCopyThreads / 64;
constexpr unsigned kItemBytes = 32768;            // max bytes per item
static_assert(kItemBytes % 1024 == 0, "a wave moves 1 KiB per word round");
constexpr int kCoreThreads = 1024;
constexpr int kLdsKeys = 16384;                   // 128 KiB of u64 keys in LDS

// The plan kernels: the plan core alone (fused: it classifies the agents
// itself), or classification over many workgroups whose last one runs the core.
hipError_t launch_plan(const PlanArgs& a, hipStream_t st);
constexpr unsigned kFuseAgents = 12288;           // plan core classifies up to this many
// Both directions of a direct step in one launch (see k_duplex).
struct DuplexArgs {
    const int* lunits;              // [n_in] unit of each load position
    const u64* lhost;               // [n_in] host byte offset of each load position's bytes
    const int* wunits;              // [n_written] unit of each written-back position
    const u64* whost;               // [n_written] host byte offset it goes to
    const unsigned* wrel;           // [n_written] its released position
    const u64* rhost;               // [released] host byte offset if written back, else ~0
    u64 n_in;                       // load positions (units loaded)
    u64 n_written;                  // written-back positions (units written back)
    u64 n_free;                     // load positions < n_free take pre-step free units;
                                    // position q >= n_free takes released position q - n_free
    const CopyItem* items;
    unsigned n_items;               // items per unit
    unsigned item_groups;           // ceil(n_items / kCopyWavesPerBlock) blocks per position
    const u64* plane_base;          // [P] device addresses
    const u64* chunk_bytes;         // [P]
    char* host;                     // device address of the host copies
    u64 capacity;                   // U; unit ids outside [0, U) are skipped
};
hipError_t launch_duplex(const DuplexArgs& a, hipStream_t st);
hipError_t launch_pack(const CopyArgs& a, hipStream_t st);
hipError_t launch_unpack(const CopyArgs& a, hipStream_t st);
hipError_t launch_zero_u32(unsigned* p, u64 n, hipStream_t st);
hipError_t launch_probe_copy(void* dst, const void* src, u64 bytes, hipStream_t st);
hipError_t launch_nop(hipStream_t st);

// Host helpers defined in ss_pool.hip.
ss_status set_err(ss_status st, const char* fmt, ...);       // sets ss_last_error
// hipMemcpyAsync of the data-movement paths (pool steps, loader chunks); a
// copy armed to fail by ss_debug_fail_copy returns hipErrorUnknown unissued.
hipError_t copy_async(void* dst, const void* src, u64 bytes, hipMemcpyKind kind, hipStream_t st);
bool device_range_ok(const void* ptr, u64 bytes, int device); // one device allocation
bool pinned_range_ok(const void* ptr, u64 bytes);             // pinned host memory

}  // namespace ss
