// Host side of libscalesim: the C ABI declared in include/scalesim.h.
//
// Two library streams (non-blocking, default priority):
//   out   plan kernels, then per eviction ring slot: pack kernel ->
//         hipMemcpyAsync of the slot to the victims' host copies
//   in    per load ring slot: hipMemcpyAsync of the loads' host copies into
//         the slot -> unpack kernel
// Each stream is FIFO, so a ring slot is refilled only after the copy or
// kernel that last used it finished, and the two copy directions proceed side
// by side on the host link.  One cross-stream dependency remains: an unpack
// that writes units released by this step's victims waits for the pack that
// read them.  Loads take the pre-step free units first and then the released
// units in eviction order, so slot k of the loads depends on a single pack
// slot.  The next step's plan waits for the previous step's loads, its
// evictions (packs and device-to-host copies) and its block-table update.
//
// Direct transfers (direct_bytes): a direction whose bytes in the step are at
// most the pool's limit skips the staging ring and the copy commands; one
// pack (or unpack) launch reads (or writes) each unit's place in its agent's
// pinned host copy over the host link, at the addresses the block-table
// kernels record per moved unit.  Small steps are latency-bound, and one
// launch costs less than the copy commands of every agent.  A direct unpack
// that overwrites released units waits for the step's last pack.  A step
// whose moves are all direct runs on the caller's stream (block-table update,
// pack, unpack), so it crosses no hardware queue after the plan.
//
// The two streams are shared by all pools of a device, so any number of pools
// (plus the caller's stream) fits in the four hardware queues the HIP runtime
// gives a process by default and the two directions never share a queue.
// Every cross-stream wait refers to an event recorded earlier in host order,
// so sharing cannot form a cycle.
//
// ss_plan_step returns once the plan kernel has written the plan's sequence
// number into a mapped host word (its last write, after the lists), which the
// host polls; the runtime's completion event is the fallback.
#include "scalesim.h"
#include "ss_internal.h"

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <vector>

using namespace ss;

namespace {
thread_local std::string g_err;

// How long ss_plan_step polls the plan's mapped flag word before it waits on
// the plan's event instead (a plan queued behind long work on the caller's
// stream then costs no spinning host core).
constexpr long kPlanPollUs = 2000;
}  // namespace

namespace {
// Copies left before the armed one fails (0 = disarmed); see ss_debug_fail_copy.
std::atomic<uint32_t> g_fail_copy{0};
}  // namespace

namespace ss {
hipError_t copy_async(void* dst, const void* src, u64 bytes, hipMemcpyKind kind, hipStream_t st) {
    uint32_t n = g_fail_copy.load(std::memory_order_relaxed);
    while (n != 0 && !g_fail_copy.compare_exchange_weak(n, n - 1, std::memory_order_relaxed)) {
    }
    if (n == 1) return hipErrorUnknown;              // this is the armed copy: not issued
    return hipMemcpyAsync(dst, src, bytes, kind, st);
}

ss_status set_err(ss_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return st;
}
}  // namespace ss

namespace {

enum State { kIdle = 0, kPlanned = 1, kPacked = 2 };

struct TimedPair {
    hipEvent_t a = nullptr, b = nullptr;
    u64 bytes = 0;
};

}  // namespace

struct ss_pool {
    int device = 0;
    uint32_t N = 0;
    u64 U = 0;
    uint32_t P = 0;
    u64 unit_bytes = 0;
    uint32_t idbits = 1;
    uint32_t flags = 0;
    std::vector<u64> chunk_bytes;
    std::vector<uint32_t> s;
    std::vector<u64> host_off;
    char* host = nullptr;
    u64 host_bytes = 0;
    char* stage_out = nullptr;
    char* stage_in = nullptr;
    uint32_t ring = 1;
    u64 units_per_slot = 0;
    u64 slot_bytes = 0;
    u64 direct_bytes = 0;          // directions of at most this many bytes go direct
    char* host_dev = nullptr;      // device address of the host copies (direct mode)

    // device metadata
    unsigned* d_units = nullptr;
    u64* d_agent_off = nullptr;
    int* d_bt = nullptr;
    unsigned char* d_resident = nullptr;
    unsigned* d_occ = nullptr;
    unsigned occ_words = 0;
    PlanCounters* d_cnt = nullptr;
    unsigned* d_done = nullptr;
    u64 *d_listE = nullptr, *d_listC = nullptr, *d_listL = nullptr;
    u64 *d_sortE = nullptr, *d_sortC = nullptr, *d_sortL = nullptr;
    u64 *d_prefE = nullptr, *d_prefC = nullptr, *d_loff = nullptr;
    unsigned *d_victims = nullptr, *d_loads = nullptr;
    int *d_vunits = nullptr, *d_lunits = nullptr, *d_free_old = nullptr, *d_wunits = nullptr;
    unsigned char* d_vwritten = nullptr;
    u64* d_woff = nullptr;
    u64* d_host_off = nullptr;     // direct mode: [N] host-copy offsets
    u64 *d_whost = nullptr, *d_lhost = nullptr;   // direct mode: [U] per moved unit
    u64* d_rhost = nullptr;                       // direct mode: [U] per released position
    unsigned* d_wrel = nullptr;                   // direct mode: [U] per written-back position
    PlanResult* d_res = nullptr;
    BtArgs* d_btargs = nullptr;    // the block-table update's arguments (pool constants)
    // timing mode: two plans' phase stamps in mapped host memory (the kernel
    // writes them, the host reads them directly) and two plans' event pairs,
    // so a plan's timing is folded one step later, when it is long complete
    u64* h_phase = nullptr;        // [2][kPlanPhases]
    u64* h_phase_dev = nullptr;
    u64* d_hist_w = nullptr;
    unsigned* d_hist_e = nullptr;
    uint32_t smax = 1;             // largest agent size in units
    bool plan_pending[2] = {false, false};
    double us_per_tick = 0.01;     // device wall clock
    CopyItem* d_items = nullptr;
    unsigned n_items = 0;
    u64* d_plane_base = nullptr;
    u64* d_chunk_bytes = nullptr;

    // mapped pinned host mirrors of the plan
    unsigned* h_flag = nullptr;    // the plan kernel's last write: its sequence number
    unsigned* h_flag_dev = nullptr;
    unsigned plan_seq = 0;
    PlanResult* h_res = nullptr;
    unsigned* h_victims = nullptr;
    unsigned* h_loads = nullptr;
    unsigned char* h_vwritten = nullptr;
    PlanResult* h_res_dev = nullptr;
    unsigned* h_victims_dev = nullptr;
    unsigned* h_loads_dev = nullptr;
    unsigned char* h_vwritten_dev = nullptr;
    // mapped pinned mirrors of host-memory plan inputs (distances, mask, dirty
    // mask): the plan kernel reads them over the host link
    unsigned* h_in_dist = nullptr;
    unsigned char* h_in_act = nullptr;
    unsigned char* h_in_dirty = nullptr;
    unsigned* h_in_dist_dev = nullptr;
    unsigned char* h_in_act_dev = nullptr;
    unsigned char* h_in_dirty_dev = nullptr;

    hipStream_t st_out = nullptr, st_in = nullptr;
    hipEvent_t ev_planned = nullptr, ev_caller = nullptr,
               ev_out_done = nullptr, ev_in_done = nullptr;
    std::vector<hipEvent_t> ev_packed;            // per eviction slot index in the step
    unsigned n_pack_step = 0;                     // pack launches of the current step
    bool direct_out = false;                      // this step's eviction went direct
    bool inline_step = false;                     // this step runs on the caller's stream
    bool duplex_step = false;                     // this step's two directions were one launch
    hipStream_t bt_stream = nullptr;              // stream of the last plan's block-table update
    hipStream_t joined_stream = nullptr;          // caller stream that the last ss_prefetch_unpack
                                                  // made wait for the whole step
    bool joined_valid = false;

    // timing (SS_FLAG_TIMING): one pair per launch or per slot's copies
    std::vector<TimedPair> t_pack, t_unpack, t_d2h, t_h2d, t_dout, t_din, t_dup;
    size_t n_t_pack = 0, n_t_unpack = 0, n_t_d2h = 0, n_t_h2d = 0, n_t_dout = 0, n_t_din = 0,
           n_t_dup = 0;
    ss_stats stats{};

    // plan of the current step (host)
    ss_plan plan{};
    PlanResult res{};
    std::vector<u64> voff, loff, woff;
    std::vector<long long> last_written;   // per victim: last written-back victim <= i, or -1

    State state = kIdle;
    bool poisoned = false;
};

namespace {

// Per-device out/in stream pair, shared by the device's pools.
struct SharedStreams {
    hipStream_t out = nullptr, in = nullptr;
    int refs = 0;
};
std::mutex g_streams_mu;
std::map<int, SharedStreams> g_streams;

hipError_t acquire_streams(int device, hipStream_t* out, hipStream_t* in) {
    std::lock_guard<std::mutex> lk(g_streams_mu);
    SharedStreams& ss = g_streams[device];
    if (ss.refs == 0) {
        hipError_t e = hipStreamCreateWithFlags(&ss.out, hipStreamNonBlocking);
        if (e != hipSuccess) return e;
        e = hipStreamCreateWithFlags(&ss.in, hipStreamNonBlocking);
        if (e != hipSuccess) {
            (void)hipStreamDestroy(ss.out);
            ss.out = nullptr;
            return e;
        }
    }
    ss.refs++;
    *out = ss.out;
    *in = ss.in;
    return hipSuccess;
}

void release_streams(int device) {
    std::lock_guard<std::mutex> lk(g_streams_mu);
    auto it = g_streams.find(device);
    if (it == g_streams.end() || it->second.refs == 0) return;
    if (--it->second.refs == 0) {
        (void)hipStreamDestroy(it->second.out);
        (void)hipStreamDestroy(it->second.in);
        g_streams.erase(it);
    }
}

struct DeviceGuard {
    int prev = -1;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        if (prev != dev) (void)hipSetDevice(dev);
    }
    ~DeviceGuard() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

ss_status hip_fail(ss_pool* p, hipError_t e, const char* what, bool poison) {
    if (p && poison) p->poisoned = true;
    return set_err(SS_ERR_HIP, "%s failed: %s", what, hipGetErrorString(e));
}

#define TRY_HIP(pool, expr, poison)                                              \
    do {                                                                         \
        hipError_t _e = (expr);                                                  \
        if (_e != hipSuccess) return hip_fail((pool), _e, #expr, (poison));      \
    } while (0)

template <class T>
hipError_t dalloc(T** p, size_t n) {
    return hipMalloc(reinterpret_cast<void**>(p), std::max<size_t>(n, 1) * sizeof(T));
}

unsigned pow2ceil_u(unsigned n) {
    unsigned p = 1;
    while (p < n) p <<= 1;
    return p;
}

void free_pool(ss_pool* p) {
    if (!p) return;
    DeviceGuard g(p->device);
    hipStream_t sts[] = {p->st_out, p->st_in};
    for (hipStream_t s : sts)
        if (s) (void)hipStreamSynchronize(s);
    // work of steps that ran on a caller's stream
    for (hipEvent_t e : {p->ev_planned, p->ev_out_done, p->ev_in_done})
        if (e) (void)hipEventSynchronize(e);
    void* dptrs[] = {p->d_units, p->d_agent_off, p->d_bt, p->d_resident, p->d_occ, p->d_cnt,
                     p->d_listE, p->d_listC, p->d_listL, p->d_sortE, p->d_sortC, p->d_sortL,
                     p->d_prefE, p->d_prefC, p->d_loff, p->d_victims, p->d_loads, p->d_vunits,
                     p->d_lunits, p->d_free_old, p->d_res, p->d_hist_w, p->d_hist_e,
                     p->d_wunits, p->d_vwritten, p->d_woff, p->d_items, p->d_plane_base,
                     p->d_chunk_bytes, p->d_done, p->d_host_off, p->d_whost, p->d_lhost,
                     p->d_rhost, p->d_wrel, p->d_btargs};
    for (void* d : dptrs)
        if (d) (void)hipFree(d);
    void* hptrs[] = {p->h_flag, p->h_phase, p->h_res, p->h_victims, p->h_loads, p->h_vwritten,
                     p->h_in_dist, p->h_in_act, p->h_in_dirty};
    for (void* h : hptrs)
        if (h) (void)hipHostFree(h);
    if (p->st_out) release_streams(p->device);
    hipEvent_t evs[] = {p->ev_planned, p->ev_caller, p->ev_out_done, p->ev_in_done};
    for (hipEvent_t e : evs)
        if (e) (void)hipEventDestroy(e);
    for (hipEvent_t e : p->ev_packed)
        if (e) (void)hipEventDestroy(e);
    for (auto* v : {&p->t_pack, &p->t_unpack, &p->t_d2h, &p->t_h2d, &p->t_dout, &p->t_din,
                    &p->t_dup})
        for (auto& tp : *v) {
            if (tp.a) (void)hipEventDestroy(tp.a);
            if (tp.b) (void)hipEventDestroy(tp.b);
        }
    delete p;
}

hipError_t make_event(hipEvent_t* e, bool timing) {
    return hipEventCreateWithFlags(e, timing ? hipEventDefault : hipEventDisableTiming);
}

hipError_t timed_pair(std::vector<TimedPair>& v, size_t idx, TimedPair** out) {
    while (v.size() <= idx) {
        TimedPair tp;
        hipError_t e = make_event(&tp.a, true);
        if (e != hipSuccess) return e;
        e = make_event(&tp.b, true);
        if (e != hipSuccess) return e;
        v.push_back(tp);
    }
    *out = &v[idx];
    return hipSuccess;
}

// Fold the previous step's event times into the stats.  Called only when that
// step's work is known to have finished.
void collect_timing(ss_pool* p) {
    if (!(p->flags & SS_FLAG_TIMING)) return;
    auto fold = [](std::vector<TimedPair>& v, size_t n, double* ms_acc, uint64_t* bytes_acc,
                   uint64_t* count) {
        float ms = 0.f;
        for (size_t i = 0; i < n; ++i)
            if (hipEventElapsedTime(&ms, v[i].a, v[i].b) == hipSuccess) {
                *ms_acc += ms;
                *bytes_acc += v[i].bytes;
                if (count) (*count)++;
            }
    };
    fold(p->t_pack, p->n_t_pack, &p->stats.pack_ms, &p->stats.pack_bytes, &p->stats.pack_launches);
    fold(p->t_unpack, p->n_t_unpack, &p->stats.unpack_ms, &p->stats.unpack_bytes,
         &p->stats.unpack_launches);
    fold(p->t_d2h, p->n_t_d2h, &p->stats.d2h_ms, &p->stats.d2h_bytes, nullptr);
    fold(p->t_h2d, p->n_t_h2d, &p->stats.h2d_ms, &p->stats.h2d_bytes, nullptr);
    fold(p->t_dout, p->n_t_dout, &p->stats.direct_out_ms, &p->stats.direct_out_bytes,
         &p->stats.direct_out_launches);
    fold(p->t_din, p->n_t_din, &p->stats.direct_in_ms, &p->stats.direct_in_bytes,
         &p->stats.direct_in_launches);
    fold(p->t_dup, p->n_t_dup, &p->stats.duplex_ms, &p->stats.duplex_bytes,
         &p->stats.duplex_launches);
    p->n_t_pack = p->n_t_unpack = p->n_t_d2h = p->n_t_h2d = p->n_t_dout = p->n_t_din = 0;
    p->n_t_dup = 0;
}

// Fold plan slot k (its phase stamps: the kernel's wall clock at its entry,
// at each phase's end, and after its block-table tail) into the stats; its
// kernel must have completed.  No event pair brackets the plan kernel, so a
// timed plan call queues what an untimed one does.
void fold_plan(ss_pool* p, int k) {
    if (!p->plan_pending[k]) return;
    p->plan_pending[k] = false;
    const volatile u64* ph = p->h_phase + k * kPlanPhases;
    if (ph[8] >= ph[0]) p->stats.plan_gpu_ms += (double)(ph[8] - ph[0]) * p->us_per_tick * 1e-3;
    for (int i = 1; i < 8; ++i)
        if (ph[i] >= ph[i - 1])
            p->stats.plan_phase_us[i - 1] += (double)(ph[i] - ph[i - 1]) * p->us_per_tick;
}

}  // namespace

namespace {
// device_range_ok for a pointer whose attributes are already known.
bool device_range_attr_ok(const hipPointerAttribute_t& attr, const void* ptr, u64 bytes,
                          int device) {
    if (attr.type == hipMemoryTypeManaged) return true;
    if (attr.type != hipMemoryTypeDevice || attr.device != device) return false;
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, const_cast<void*>(ptr)) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    const u64 off = reinterpret_cast<uintptr_t>(ptr) - reinterpret_cast<uintptr_t>(base);
    return off <= size && bytes <= size - off;
}
}  // namespace

namespace ss {
// True if [ptr, ptr + bytes) lies inside one allocation of device memory on
// `device` (or managed memory).
bool device_range_ok(const void* ptr, u64 bytes, int device) {
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, ptr) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    return device_range_attr_ok(attr, ptr, bytes, device);
}

// True if host_ptr is pinned (page-locked) host memory; when the runtime
// reports the allocation's extent, [host_ptr, host_ptr + bytes) must fit in it.
bool pinned_range_ok(const void* ptr, u64 bytes) {
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, ptr) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    if (attr.type != hipMemoryTypeHost) return false;
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, const_cast<void*>(ptr)) != hipSuccess) {
        (void)hipGetLastError();
        return true;
    }
    const u64 off = reinterpret_cast<uintptr_t>(ptr) - reinterpret_cast<uintptr_t>(base);
    return off <= size && bytes <= size - off;
}
}  // namespace ss

namespace {

// Where a plan input of `bytes` bytes lives: device memory of `device`
// (kInDevice, read by the kernel in place), host memory (kInHost: pageable or
// pinned; copied into the pool's mapped mirror), or neither (kInBad: device
// memory of another device, or a device range that is too short).
enum InputKind { kInDevice, kInHost, kInBad };
InputKind input_kind(const void* ptr, u64 bytes, int device) {
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, ptr) != hipSuccess) {
        (void)hipGetLastError();
        return kInHost;                              // memory the runtime does not know: pageable
    }
    if (attr.type == hipMemoryTypeHost || attr.type == hipMemoryTypeUnregistered) return kInHost;
    return device_range_attr_ok(attr, ptr, bytes, device) ? kInDevice : kInBad;
}

// The host's unit offsets of the current plan's lists (victims and loads in
// unit order, the written-back victims' units, and per victim the last
// written-back victim at or before it), for the copies of ss_evict_pack and
// ss_prefetch_unpack.  Computed by ss_evict_pack rather than ss_plan_step, so
// the plan call returns the plan without this bookkeeping.
void host_offsets(ss_pool* p) {
    const PlanResult& r = p->res;
    p->voff.resize(r.n_victims + 1);
    p->loff.resize(r.n_loads + 1);
    p->voff[0] = 0;
    for (unsigned i = 0; i < r.n_victims; ++i) p->voff[i + 1] = p->voff[i] + p->s[p->h_victims[i]];
    p->loff[0] = 0;
    for (unsigned i = 0; i < r.n_loads; ++i) p->loff[i + 1] = p->loff[i] + p->s[p->h_loads[i]];
    p->woff.resize(r.n_victims + 1);
    p->last_written.resize(r.n_victims);
    p->woff[0] = 0;
    for (unsigned i = 0; i < r.n_victims; ++i) {
        const bool w = p->h_vwritten[i] != 0;
        p->woff[i + 1] = p->woff[i] + (w ? p->s[p->h_victims[i]] : 0);
        p->last_written[i] = w ? (long long)i : (i ? p->last_written[i - 1] : -1);
    }
}

ss_status check_usable(ss_pool* p) {
    if (!p) return set_err(SS_ERR_ARG, "pool is NULL");
    if (p->poisoned) return set_err(SS_ERR_POISONED, "pool is poisoned by an earlier HIP failure");
    return SS_OK;
}

// The pool's waits: blocking, or under SS_FLAG_POLL_WAIT a loop of queries
// (the thread stays busy and the runtime's state stays in its caches, so the
// launches of the next call cost their warm host time).  A query that finds
// the work pending leaves that status as the thread's last error: cleared.
template <class Query>
hipError_t poll_until_done(Query query) {
    hipError_t e;
    while ((e = query()) == hipErrorNotReady) __builtin_ia32_pause();
    (void)hipGetLastError();
    return e;
}

hipError_t wait_stream(const ss_pool* p, hipStream_t s) {
    if (!(p->flags & SS_FLAG_POLL_WAIT)) return hipStreamSynchronize(s);
    return poll_until_done([s] { return hipStreamQuery(s); });
}

hipError_t wait_event(const ss_pool* p, hipEvent_t ev) {
    if (!(p->flags & SS_FLAG_POLL_WAIT)) return hipEventSynchronize(ev);
    return poll_until_done([ev] { return hipEventQuery(ev); });
}

// Fold the previous step's copy events and the previous plan's event time and
// phase stamps into the stats (timing mode; called before this step's pack).
// The previous step's loads completed before this plan's kernel ran, and so
// did the previous plan; the previous evictions are waited for here.  This
// plan is folded at the next step, or by ss_get_stats.
ss_status collect_plan_timing(ss_pool* p) {
    if (!(p->flags & SS_FLAG_TIMING)) return SS_OK;
    TRY_HIP(p, wait_event(p, p->ev_out_done), true);
    collect_timing(p);
    fold_plan(p, (int)((p->plan_seq + 1) & 1));      // the previous plan's slot
    return SS_OK;
}

// Everything pending, the current plan included (its kernel is waited for).
ss_status collect_all_timing(ss_pool* p) {
    if (!(p->flags & SS_FLAG_TIMING)) return SS_OK;
    for (hipEvent_t e : {p->ev_planned, p->ev_out_done, p->ev_in_done})
        TRY_HIP(p, wait_event(p, e), true);
    collect_timing(p);
    fold_plan(p, 0);
    fold_plan(p, 1);
    return SS_OK;
}

// The event that follows the last plan's block-table update: the plan's own
// event (the plan kernel runs the update in its tail).
hipEvent_t bt_event(const ss_pool* p) { return p->ev_planned; }

// Arguments of the block-table update that follows each plan.
BtArgs bt_args(const ss_pool* p) {
    BtArgs B{};
    B.res = p->d_res;
    B.victims = p->d_victims;
    B.loads = p->d_loads;
    B.units = p->d_units;
    B.agent_off = p->d_agent_off;
    B.bt = p->d_bt;
    B.occ = p->d_occ;
    B.voff = p->d_prefE;
    B.loff = p->d_loff;
    B.free_old = p->d_free_old;
    B.vunits = p->d_vunits;
    B.lunits = p->d_lunits;
    B.capacity = p->U;
    B.vwritten = p->d_vwritten;
    B.woff = p->d_woff;
    B.wunits = p->d_wunits;
    B.host_off = p->d_host_off;
    B.unit_bytes = p->unit_bytes;
    B.whost = p->d_whost;
    B.lhost = p->d_lhost;
    B.rhost = p->d_rhost;
    B.wrel = p->d_wrel;
    return B;
}

}  // namespace

extern "C" {

const char* ss_last_error(void) { return g_err.c_str(); }

void ss_debug_fail_copy(uint32_t n) { g_fail_copy.store(n, std::memory_order_relaxed); }

ss_status ss_pool_create(const ss_pool_desc* d, ss_pool** out) {
    if (!d || !out) return set_err(SS_ERR_ARG, "desc and out must not be NULL");
    if (d->n_agents == 0 || d->n_agents >= (1u << 31))
        return set_err(SS_ERR_ARG, "n_agents must be in [1, 2^31)");
    if (d->capacity_units == 0 || d->capacity_units >= (1ull << 31))
        return set_err(SS_ERR_ARG, "capacity_units must be in [1, 2^31)");
    if (d->n_planes == 0 || !d->plane_base || !d->chunk_bytes || !d->agent_units)
        return set_err(SS_ERR_ARG, "n_planes, plane_base, chunk_bytes and agent_units are required");
    if (!d->host_backing) return set_err(SS_ERR_ARG, "host_backing is required");
    if (!d->dev_staging) return set_err(SS_ERR_ARG, "dev_staging is required");
    if (d->ring_slots == 0) return set_err(SS_ERR_ARG, "ring_slots must be >= 1");
    if (d->flags & ~(SS_FLAG_TIMING | SS_FLAG_POLL_WAIT)) return set_err(SS_ERR_ARG, "unknown flag bits");
    u64 unit_bytes = 0;
    for (uint32_t c = 0; c < d->n_planes; ++c) {
        const u64 cb = d->chunk_bytes[c];
        if (cb < 16 || cb % 16 != 0)
            return set_err(SS_ERR_ARG, "chunk_bytes[%u] = %llu is not a positive multiple of 16", c,
                           (unsigned long long)cb);
        if (!d->plane_base[c]) return set_err(SS_ERR_ARG, "plane_base[%u] is NULL", c);
        if (reinterpret_cast<uintptr_t>(d->plane_base[c]) % 16 != 0)
            return set_err(SS_ERR_ARG, "plane_base[%u] is not 16-byte aligned", c);
        unit_bytes += cb;
    }
    if (reinterpret_cast<uintptr_t>(d->dev_staging) % 16 != 0)
        return set_err(SS_ERR_ARG, "dev_staging is not 16-byte aligned");
    u64 total_units = 0;
    for (uint32_t a = 0; a < d->n_agents; ++a) {
        if (d->agent_units[a] == 0) return set_err(SS_ERR_ARG, "agent_units[%u] is 0", a);
        total_units += d->agent_units[a];
    }
    if (total_units >= (1ull << 40)) return set_err(SS_ERR_ARG, "too many agent units");
    const u64 half = (d->staging_bytes / 2) & ~15ull;    // second half 16-byte aligned
    const u64 ups = half / d->ring_slots / unit_bytes;
    if (ups == 0)
        return set_err(SS_ERR_ARG, "staging_bytes %llu too small: each of 2 x %u slots needs >= %llu",
                       (unsigned long long)d->staging_bytes, d->ring_slots,
                       (unsigned long long)unit_bytes);

    std::vector<u64> host_off(d->n_agents);
    u64 acc = 0;
    for (uint32_t a = 0; a < d->n_agents; ++a) {
        const u64 off = d->host_off ? d->host_off[a] : acc;
        const u64 len = (u64)d->agent_units[a] * unit_bytes;
        if (off > d->host_bytes || len > d->host_bytes - off)
            return set_err(SS_ERR_ARG, "host copy of agent %u [%llu, +%llu) exceeds host_bytes", a,
                           (unsigned long long)off, (unsigned long long)len);
        host_off[a] = off;
        acc += len;
    }
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || d->device < 0 || d->device >= ndev) {
        (void)hipGetLastError();
        return set_err(SS_ERR_ARG, "device %d not present", (int)d->device);
    }

    {
        DeviceGuard g(d->device);
        for (uint32_t c = 0; c < d->n_planes; ++c)
            if (!device_range_ok(d->plane_base[c], d->capacity_units * d->chunk_bytes[c], d->device))
                return set_err(SS_ERR_ARG, "plane %u: [plane_base, +capacity*chunk_bytes) is not "
                                           "device memory of device %d", c, (int)d->device);
        if (!device_range_ok(d->dev_staging, d->staging_bytes, d->device))
            return set_err(SS_ERR_ARG, "dev_staging [0, staging_bytes) is not device memory");
        if (!pinned_range_ok(d->host_backing, d->host_bytes))
            return set_err(SS_ERR_ARG, "host_backing [0, host_bytes) is not pinned host memory");
    }

    ss_pool* p = new (std::nothrow) ss_pool();
    if (!p) return set_err(SS_ERR_NOMEM, "out of host memory");
    p->device = d->device;
    p->N = d->n_agents;
    p->U = d->capacity_units;
    p->P = d->n_planes;
    p->unit_bytes = unit_bytes;
    p->flags = d->flags;
    p->chunk_bytes.assign(d->chunk_bytes, d->chunk_bytes + d->n_planes);
    p->s.assign(d->agent_units, d->agent_units + d->n_agents);
    p->host_off = std::move(host_off);
    p->host = static_cast<char*>(d->host_backing);
    p->host_bytes = d->host_bytes;
    p->direct_bytes = d->direct_bytes;
    p->ring = d->ring_slots;
    p->units_per_slot = ups;
    p->slot_bytes = ups * unit_bytes;
    p->stage_out = static_cast<char*>(d->dev_staging);
    p->stage_in = static_cast<char*>(d->dev_staging) + half;
    while ((1ull << p->idbits) < p->N) p->idbits++;

    DeviceGuard g(p->device);
    hipError_t e = hipSuccess;
#define CREATE_TRY(expr)                                          \
    do {                                                          \
        e = (expr);                                               \
        if (e != hipSuccess) {                                    \
            ss_status st = hip_fail(nullptr, e, #expr, false);    \
            free_pool(p);                                         \
            return st;                                            \
        }                                                         \
    } while (0)

    const u64 N = p->N, U = p->U;
    const unsigned npad = pow2ceil_u(p->N);
    p->occ_words = (unsigned)((U + 31) / 32);
    CREATE_TRY(dalloc(&p->d_units, N));
    CREATE_TRY(dalloc(&p->d_agent_off, N + 1));
    CREATE_TRY(dalloc(&p->d_bt, total_units));
    CREATE_TRY(dalloc(&p->d_resident, N));
    CREATE_TRY(dalloc(&p->d_occ, p->occ_words));
    CREATE_TRY(dalloc(&p->d_cnt, 1));
    CREATE_TRY(dalloc(&p->d_done, 1));
    CREATE_TRY(dalloc(&p->d_listE, N));
    CREATE_TRY(dalloc(&p->d_listC, N * kCandLists));
    CREATE_TRY(dalloc(&p->d_listL, N));
    CREATE_TRY(dalloc(&p->d_sortE, npad));
    CREATE_TRY(dalloc(&p->d_sortC, npad));
    CREATE_TRY(dalloc(&p->d_sortL, npad));
    CREATE_TRY(dalloc(&p->d_prefE, N + 1));
    CREATE_TRY(dalloc(&p->d_prefC, N + 1));
    CREATE_TRY(dalloc(&p->d_loff, N + 1));
    CREATE_TRY(dalloc(&p->d_victims, N));
    CREATE_TRY(dalloc(&p->d_loads, N));
    CREATE_TRY(dalloc(&p->d_vunits, U));
    CREATE_TRY(dalloc(&p->d_lunits, U));
    CREATE_TRY(dalloc(&p->d_free_old, U));
    CREATE_TRY(dalloc(&p->d_wunits, U));
    if (p->direct_bytes) {
        if (hipHostGetDevicePointer(reinterpret_cast<void**>(&p->host_dev), p->host, 0) !=
            hipSuccess) {
            (void)hipGetLastError();
            free_pool(p);
            return set_err(SS_ERR_ARG, "direct_bytes > 0 needs host_backing that the device can "
                                       "access (pinned, mapped)");
        }
        CREATE_TRY(dalloc(&p->d_host_off, N));
        CREATE_TRY(dalloc(&p->d_whost, U));
        CREATE_TRY(dalloc(&p->d_lhost, U));
        CREATE_TRY(dalloc(&p->d_rhost, U));
        CREATE_TRY(dalloc(&p->d_wrel, U));
        CREATE_TRY(hipMemcpy(p->d_host_off, p->host_off.data(), N * sizeof(u64),
                             hipMemcpyHostToDevice));
    }
    CREATE_TRY(dalloc(&p->d_vwritten, N));
    CREATE_TRY(dalloc(&p->d_woff, N + 1));
    CREATE_TRY(dalloc(&p->d_res, 1));
    CREATE_TRY(hipHostMalloc(reinterpret_cast<void**>(&p->h_phase), 2 * kPlanPhases * sizeof(u64),
                             hipHostMallocMapped));
    std::memset(p->h_phase, 0, 2 * kPlanPhases * sizeof(u64));
    CREATE_TRY(hipHostGetDevicePointer(reinterpret_cast<void**>(&p->h_phase_dev), p->h_phase, 0));
    CREATE_TRY(dalloc(&p->d_hist_w, kDistBuckets));
    CREATE_TRY(dalloc(&p->d_hist_e, kDistBuckets));
    for (uint32_t a = 0; a < p->N; ++a) p->smax = std::max(p->smax, p->s[a]);
    {
        int khz = 0;
        if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, p->device) == hipSuccess &&
            khz > 0)
            p->us_per_tick = 1000.0 / khz;
    }
    CREATE_TRY(hipHostMalloc(reinterpret_cast<void**>(&p->h_flag), 64, hipHostMallocMapped));
    *p->h_flag = 0;
    CREATE_TRY(hipHostGetDevicePointer(reinterpret_cast<void**>(&p->h_flag_dev), p->h_flag, 0));
    CREATE_TRY(hipHostMalloc(reinterpret_cast<void**>(&p->h_res), sizeof(PlanResult),
                             hipHostMallocMapped));
    CREATE_TRY(hipHostMalloc(reinterpret_cast<void**>(&p->h_victims), N * sizeof(unsigned),
                             hipHostMallocMapped));
    CREATE_TRY(hipHostMalloc(reinterpret_cast<void**>(&p->h_loads), N * sizeof(unsigned),
                             hipHostMallocMapped));
    CREATE_TRY(hipHostGetDevicePointer(reinterpret_cast<void**>(&p->h_res_dev), p->h_res, 0));
    CREATE_TRY(hipHostGetDevicePointer(reinterpret_cast<void**>(&p->h_victims_dev), p->h_victims, 0));
    CREATE_TRY(hipHostGetDevicePointer(reinterpret_cast<void**>(&p->h_loads_dev), p->h_loads, 0));
    CREATE_TRY(hipHostMalloc(reinterpret_cast<void**>(&p->h_vwritten), N, hipHostMallocMapped));
    CREATE_TRY(hipHostGetDevicePointer(reinterpret_cast<void**>(&p->h_vwritten_dev), p->h_vwritten, 0));
    CREATE_TRY(hipHostMalloc(reinterpret_cast<void**>(&p->h_in_dist), N * sizeof(unsigned),
                             hipHostMallocMapped));
    CREATE_TRY(hipHostGetDevicePointer(reinterpret_cast<void**>(&p->h_in_dist_dev), p->h_in_dist, 0));
    CREATE_TRY(hipHostMalloc(reinterpret_cast<void**>(&p->h_in_act), N, hipHostMallocMapped));
    CREATE_TRY(hipHostGetDevicePointer(reinterpret_cast<void**>(&p->h_in_act_dev), p->h_in_act, 0));
    CREATE_TRY(hipHostMalloc(reinterpret_cast<void**>(&p->h_in_dirty), N, hipHostMallocMapped));
    CREATE_TRY(hipHostGetDevicePointer(reinterpret_cast<void**>(&p->h_in_dirty_dev), p->h_in_dirty, 0));

    // copy items: pieces of at most kItemBytes, plane by plane
    std::vector<CopyItem> items;
    u64 plane_off = 0;
    for (uint32_t c = 0; c < p->P; ++c) {
        for (u64 off = 0; off < p->chunk_bytes[c]; off += kItemBytes) {
            CopyItem it;
            it.plane = c;
            it.len = (unsigned)std::min<u64>(kItemBytes, p->chunk_bytes[c] - off);
            it.chunk_off = off;
            it.unit_off = plane_off + off;
            items.push_back(it);
        }
        plane_off += p->chunk_bytes[c];
    }
    p->n_items = (unsigned)items.size();
    CREATE_TRY(dalloc(&p->d_items, items.size()));
    CREATE_TRY(dalloc(&p->d_plane_base, p->P));
    CREATE_TRY(dalloc(&p->d_chunk_bytes, p->P));

    std::vector<u64> agent_off(N + 1, 0);
    for (u64 a = 0; a < N; ++a) agent_off[a + 1] = agent_off[a] + p->s[a];
    std::vector<int> bt(total_units, -1);
    std::vector<unsigned> occ(p->occ_words, 0u);
    if (U % 32) occ.back() = ~((1u << (U % 32)) - 1u);       // units >= U never free
    std::vector<u64> bases(p->P);
    for (uint32_t c = 0; c < p->P; ++c) bases[c] = reinterpret_cast<u64>(d->plane_base[c]);
    std::vector<unsigned char> zeros_n(N, 0);
    PlanCounters zc{};
    CREATE_TRY(hipMemcpy(p->d_units, p->s.data(), N * sizeof(unsigned), hipMemcpyHostToDevice));
    CREATE_TRY(hipMemcpy(p->d_agent_off, agent_off.data(), (N + 1) * sizeof(u64),
                         hipMemcpyHostToDevice));
    CREATE_TRY(hipMemcpy(p->d_bt, bt.data(), total_units * sizeof(int), hipMemcpyHostToDevice));
    CREATE_TRY(hipMemcpy(p->d_occ, occ.data(), occ.size() * sizeof(unsigned), hipMemcpyHostToDevice));
    CREATE_TRY(hipMemcpy(p->d_resident, zeros_n.data(), N, hipMemcpyHostToDevice));
    CREATE_TRY(hipMemcpy(p->d_cnt, &zc, sizeof zc, hipMemcpyHostToDevice));
    {
        const unsigned zero = 0;
        CREATE_TRY(hipMemcpy(p->d_done, &zero, sizeof zero, hipMemcpyHostToDevice));
    }
    {
        std::vector<u64> zw(kDistBuckets, 0);
        CREATE_TRY(hipMemcpy(p->d_hist_w, zw.data(), kDistBuckets * sizeof(u64), hipMemcpyHostToDevice));
        CREATE_TRY(hipMemcpy(p->d_hist_e, zw.data(), kDistBuckets * sizeof(unsigned),
                             hipMemcpyHostToDevice));
    }
    CREATE_TRY(hipMemcpy(p->d_items, items.data(), items.size() * sizeof(CopyItem),
                         hipMemcpyHostToDevice));
    CREATE_TRY(hipMemcpy(p->d_plane_base, bases.data(), p->P * sizeof(u64), hipMemcpyHostToDevice));
    CREATE_TRY(hipMemcpy(p->d_chunk_bytes, p->chunk_bytes.data(), p->P * sizeof(u64),
                         hipMemcpyHostToDevice));

    CREATE_TRY(acquire_streams(p->device, &p->st_out, &p->st_in));
    for (hipEvent_t* ev : {&p->ev_planned, &p->ev_caller, &p->ev_out_done, &p->ev_in_done})
        CREATE_TRY(make_event(ev, false));
    {
        // every pointer the block-table update uses is fixed from here on
        const BtArgs B = bt_args(p);
        CREATE_TRY(dalloc(&p->d_btargs, 1));
        CREATE_TRY(hipMemcpy(p->d_btargs, &B, sizeof(BtArgs), hipMemcpyHostToDevice));
    }
    CREATE_TRY(hipEventRecord(p->ev_out_done, p->st_out));
    CREATE_TRY(hipEventRecord(p->ev_in_done, p->st_in));
    CREATE_TRY(hipStreamSynchronize(p->st_out));
    CREATE_TRY(hipStreamSynchronize(p->st_in));
#undef CREATE_TRY
    *out = p;
    return SS_OK;
}

void ss_pool_destroy(ss_pool* p) { free_pool(p); }

ss_status ss_plan_step(ss_pool* p, const uint32_t* distances, const uint8_t* active,
                       const ss_plan_params* params, ss_plan* out, void* stream) {
    ss_status st = check_usable(p);
    if (st) return st;
    if (!distances || !active || !params || !out)
        return set_err(SS_ERR_ARG, "distances, active, params and out are required");
    if (p->state != kIdle)
        return set_err(SS_ERR_ORDER, "previous step not finished: call ss_evict_pack and "
                                     "ss_prefetch_unpack before the next ss_plan_step");
    DeviceGuard g(p->device);
    const auto h0 = std::chrono::steady_clock::now();
    const InputKind kd = input_kind(distances, (u64)p->N * 4, p->device);
    const InputKind ka = input_kind(active, (u64)p->N, p->device);
    const InputKind kw = params->dirty ? input_kind(params->dirty, (u64)p->N, p->device) : kInDevice;
    if (kd == kInBad || ka == kInBad || kw == kInBad)
        return set_err(SS_ERR_ARG, "distances, active and dirty must be host memory or device "
                                   "memory of device %d holding N elements", p->device);
    // Host inputs go to the pool's mapped pinned mirrors, which the plan
    // kernel reads over the host link.  The previous plan's kernel read its
    // inputs before it published that plan, so the mirrors are free again.
    const unsigned* in_dist = distances;
    const unsigned char* in_act = active;
    const unsigned char* in_dirty = params->dirty;
    if (kd == kInHost) {
        std::memcpy(p->h_in_dist, distances, (size_t)p->N * 4);
        in_dist = p->h_in_dist_dev;
    }
    if (ka == kInHost) {
        std::memcpy(p->h_in_act, active, p->N);
        in_act = p->h_in_act_dev;
    }
    if (params->dirty && kw == kInHost) {
        std::memcpy(p->h_in_dirty, params->dirty, p->N);
        in_dirty = p->h_in_dirty_dev;
    }
    hipStream_t caller = static_cast<hipStream_t>(stream);
    const auto e0 = std::chrono::steady_clock::now();     // inputs checked (and copied)

    // The plan kernels run on the caller's stream, after the caller's earlier
    // work (which may produce the distances), after the previous step's loads
    // and evictions, and after the previous plan's block-table update (which
    // an overcommitted plan's successor on another stream must not overtake).
    // The evictions matter as much as the loads: this plan's block-table
    // update rewrites the unit lists the previous packs read, this step's
    // unpacks into pre-step free units may overwrite units the previous
    // step released before its packs read them, and this step's
    // host-to-device copies may read a host copy that the previous step's
    // device-to-host copies still write.  When the caller's stream is the one
    // the previous ss_prefetch_unpack made wait for the whole step, stream
    // order already gives all of this.  This plan's block-table update runs
    // after the plan on the same stream.
    if (!(p->joined_valid && p->joined_stream == caller)) {
        TRY_HIP(p, hipStreamWaitEvent(caller, p->ev_in_done, 0), true);
        TRY_HIP(p, hipStreamWaitEvent(caller, p->ev_out_done, 0), true);
    }
    TRY_HIP(p, hipStreamWaitEvent(caller, bt_event(p), 0), true);
    const auto e1 = std::chrono::steady_clock::now();     // stream waits queued

    PlanArgs A{};
    A.dist = in_dist;
    A.active = in_act;
    A.resident = p->d_resident;
    A.units = p->d_units;
    A.n = p->N;
    A.idbits = p->idbits;
    A.threshold = params->threshold;
    A.budget = params->budget_units;
    A.capacity = p->U;
    A.cnt = p->d_cnt;
    A.listE = p->d_listE;
    A.listC = p->d_listC;
    A.listL = p->d_listL;
    A.sortE = p->d_sortE;
    A.sortC = p->d_sortC;
    A.sortL = p->d_sortL;
    A.prefE = p->d_prefE;
    A.prefC = p->d_prefC;
    A.loff = p->d_loff;
    A.victims = p->d_victims;
    A.loads = p->d_loads;
    A.occ = p->d_occ;
    A.occ_words = p->occ_words;
    A.free_old = p->d_free_old;
    A.res = p->d_res;
    A.res_host = p->h_res_dev;
    A.victims_host = p->h_victims_dev;
    A.loads_host = p->h_loads_dev;
    A.fused = p->N <= kFuseAgents ? 1u : 0u;

    A.hist_w = p->d_hist_w;
    A.hist_e = p->d_hist_e;
    A.smax = p->smax;
    A.dirty = in_dirty;
    A.vwritten = p->d_vwritten;
    A.vwritten_host = p->h_vwritten_dev;
    A.woff = p->d_woff;
    A.done = p->d_done;
    A.bt = p->d_btargs;
    if (++p->plan_seq == 0) p->plan_seq = 1;
    A.flag_host = p->h_flag_dev;
    A.seq = p->plan_seq;
    const int tslot = (int)(p->plan_seq & 1);
    A.phase = (p->flags & SS_FLAG_TIMING) ? p->h_phase_dev + tslot * kPlanPhases : nullptr;

    const bool timing = p->flags & SS_FLAG_TIMING;
    if (timing) fold_plan(p, tslot);     // a plan two steps back that was never folded
    TRY_HIP(p, launch_plan(A, caller), true);
    TRY_HIP(p, hipEventRecord(p->ev_planned, caller), true);
    const auto e2 = std::chrono::steady_clock::now();     // plan kernel and its events queued
    // The block-table update runs in the plan kernel's own tail, after the
    // plan is published; it needs nothing from the host, and it changes
    // nothing after an overcommitted plan.
    p->bt_stream = caller;

    const auto h1 = std::chrono::steady_clock::now();
    // The kernel's last write is the sequence number into the mapped flag
    // word, after its results and lists are visible to the host: poll it for
    // up to kPlanPollUs, then wait on the plan's event (which also reports a
    // failed launch or kernel).
    {
        bool seen = false;
        for (;;) {
            if (__atomic_load_n(p->h_flag, __ATOMIC_ACQUIRE) == p->plan_seq) {
                seen = true;
                break;
            }
            if (std::chrono::steady_clock::now() - h1 > std::chrono::microseconds(kPlanPollUs)) break;
            __builtin_ia32_pause();
        }
        if (!seen) {
            TRY_HIP(p, hipEventSynchronize(p->ev_planned), true);
            if (__atomic_load_n(p->h_flag, __ATOMIC_ACQUIRE) != p->plan_seq) {
                p->poisoned = true;              // the device state is unknown
                return set_err(SS_ERR_HIP, "plan kernel finished without publishing its plan");
            }
        }
    }
    const auto h2 = std::chrono::steady_clock::now();
    // this plan's event time and phase stamps are folded into the stats one
    // step later (or by ss_get_stats), off the path that returns the plan
    if (timing) p->plan_pending[tslot] = true;

    const PlanResult r = *p->h_res;
    if (r.status == 1) {
        return set_err(SS_ERR_OVERCOMMIT, "active agents need more than %llu units",
                       (unsigned long long)p->U);
    }
    p->res = r;

    ss_plan& pl = p->plan;
    pl.n_victims = r.n_victims;
    pl.n_loads = r.n_loads;
    pl.n_demand = r.n_demand;
    pl.n_demand_victims = r.n_demand_victims;
    pl.victims = p->h_victims;
    pl.loads = p->h_loads;
    pl.units_out = r.units_out;
    pl.units_in = r.units_in;
    pl.bytes_out = r.units_written * p->unit_bytes;
    pl.bytes_in = r.units_in * p->unit_bytes;
    pl.units_written = r.units_written;
    pl.victim_written = p->h_vwritten;
    pl.d_victims = p->d_victims;
    pl.d_loads = p->d_loads;
    *out = pl;
    p->state = kPlanned;
    p->stats.steps++;
    if (timing) {
        const auto h3 = std::chrono::steady_clock::now();
        auto us = [](std::chrono::steady_clock::duration d) {
            return std::chrono::duration<double, std::micro>(d).count();
        };
        p->stats.plan_host_us[0] += us(h1 - h0);
        p->stats.plan_host_us[1] += us(h2 - h1);
        p->stats.plan_host_us[2] += us(h3 - h2);
        p->stats.plan_enqueue_us[0] += us(e0 - h0);
        p->stats.plan_enqueue_us[1] += us(e1 - e0);
        p->stats.plan_enqueue_us[2] += us(e2 - e1);
        p->stats.plan_enqueue_us[3] += us(h1 - e2);
    }
    return SS_OK;
}

ss_status ss_evict_pack(ss_pool* p, void* stream) {
    ss_status st = check_usable(p);
    if (st) return st;
    if (p->state != kPlanned) return set_err(SS_ERR_ORDER, "ss_evict_pack must follow ss_plan_step");
    DeviceGuard g(p->device);
    host_offsets(p);
    hipStream_t caller = static_cast<hipStream_t>(stream);
    const u64 total = p->res.units_written;
    const u64 ups = p->units_per_slot;
    const bool direct = p->direct_bytes && total && total * p->unit_bytes <= p->direct_bytes;
    // A step whose moves are all direct (or empty) runs on the caller's
    // stream: block-table update, pack and unpack queue behind the plan on one
    // hardware queue, without the cross-queue waits that cost more than such
    // a step's kernels.
    const u64 total_in = p->res.units_in;
    const bool direct_in = p->direct_bytes && total_in &&
                           total_in * p->unit_bytes <= p->direct_bytes;
    p->inline_step = p->direct_bytes && (total == 0 || direct) && (total_in == 0 || direct_in);
    // Both directions direct and non-empty: one launch moves both (k_duplex),
    // so the link carries them at once instead of one after the other (the
    // loads mostly reuse the units the victims release).
    p->duplex_step = p->inline_step && direct && direct_in && p->d_rhost;
    hipStream_t so = p->inline_step ? caller : p->st_out;
    st = collect_plan_timing(p);
    if (st) return st;
    const bool timing = p->flags & SS_FLAG_TIMING;
    if (!p->inline_step) {
        TRY_HIP(p, hipEventRecord(p->ev_caller, caller), true);
        TRY_HIP(p, hipStreamWaitEvent(p->st_out, p->ev_caller, 0), true);
    }
    // The packs read the unit lists the block-table update writes.  It was
    // queued on the plan's stream: when that is this call's stream, the packs
    // already follow it (on that stream, or behind ev_caller); otherwise they
    // wait for it.  (A wait on another stream's pending event costs the host
    // about 16 us.)
    if (caller != p->bt_stream) TRY_HIP(p, hipStreamWaitEvent(so, bt_event(p), 0), true);

    const u64 nslots = direct ? 1 : (total + ups - 1) / ups;
    while (p->ev_packed.size() < nslots) {
        hipEvent_t ev;
        TRY_HIP(p, make_event(&ev, false), true);
        p->ev_packed.push_back(ev);
    }
    p->n_pack_step = (unsigned)nslots;
    p->direct_out = direct;
    CopyArgs C{};
    C.units_list = p->d_wunits;
    C.items = p->d_items;
    C.n_items = p->n_items;
    C.item_groups = (p->n_items + kCopyWavesPerBlock - 1) / kCopyWavesPerBlock;
    C.run_order = p->n_items == p->P;
    C.plane_base = p->d_plane_base;
    C.chunk_bytes = p->d_chunk_bytes;
    C.unit_bytes = p->unit_bytes;
    C.capacity = p->U;
    if (p->duplex_step) {
        DuplexArgs D{};
        D.lunits = p->d_lunits;
        D.lhost = p->d_lhost;
        D.wunits = p->d_wunits;
        D.whost = p->d_whost;
        D.wrel = p->d_wrel;
        D.rhost = p->d_rhost;
        D.n_in = total_in;
        D.n_written = total;
        D.n_free = p->res.n_free_used;
        D.items = p->d_items;
        D.n_items = p->n_items;
        D.item_groups = C.item_groups;
        D.plane_base = p->d_plane_base;
        D.chunk_bytes = p->d_chunk_bytes;
        D.host = p->host_dev;
        D.capacity = p->U;
        TimedPair* tp = nullptr;
        if (timing) {
            TRY_HIP(p, timed_pair(p->t_dup, p->n_t_dup++, &tp), true);
            tp->bytes = (total + total_in) * p->unit_bytes;
            TRY_HIP(p, hipEventRecord(tp->a, so), true);
        }
        TRY_HIP(p, launch_duplex(D, so), true);
        if (timing) TRY_HIP(p, hipEventRecord(tp->b, so), true);
        TRY_HIP(p, hipEventRecord(p->ev_packed[0], so), true);
    } else if (direct) {
        // one launch gathers every written-back unit straight into its host copy
        C.first = 0;
        C.count = total;
        C.staging = p->host_dev;
        C.stage_off = p->d_whost;
        TimedPair* tp = nullptr;
        if (timing) {
            TRY_HIP(p, timed_pair(p->t_dout, p->n_t_dout++, &tp), true);
            tp->bytes = total * p->unit_bytes;
            TRY_HIP(p, hipEventRecord(tp->a, so), true);
        }
        TRY_HIP(p, launch_pack(C, so), true);
        if (timing) TRY_HIP(p, hipEventRecord(tp->b, so), true);
        TRY_HIP(p, hipEventRecord(p->ev_packed[0], so), true);
    }
    size_t vi = 0;
    for (u64 k = 0; !direct && k < nslots; ++k) {
        const u64 p0 = k * ups, p1 = std::min(total, p0 + ups);
        char* slot = p->stage_out + (k % p->ring) * p->slot_bytes;
        C.first = p0;
        C.count = p1 - p0;
        C.staging = slot;
        TimedPair* tp = nullptr;
        if (timing) {
            TRY_HIP(p, timed_pair(p->t_pack, p->n_t_pack++, &tp), true);
            tp->bytes = (p1 - p0) * p->unit_bytes;
            TRY_HIP(p, hipEventRecord(tp->a, p->st_out), true);
        }
        TRY_HIP(p, launch_pack(C, p->st_out), true);
        if (timing) TRY_HIP(p, hipEventRecord(tp->b, p->st_out), true);
        TRY_HIP(p, hipEventRecord(p->ev_packed[k], p->st_out), true);
        if (timing) {
            TRY_HIP(p, timed_pair(p->t_d2h, p->n_t_d2h++, &tp), true);
            tp->bytes = (p1 - p0) * p->unit_bytes;
            TRY_HIP(p, hipEventRecord(tp->a, p->st_out), true);
        }
        // each written-back victim's bytes inside [p0, p1) go to its host copy
        while (vi < p->res.n_victims && p->woff[vi + 1] <= p0) vi++;
        for (size_t i = vi; i < p->res.n_victims && p->woff[i] < p1; ++i) {
            if (p->woff[i + 1] == p->woff[i]) continue;              // clean victim
            const u64 lo = std::max(p0, p->woff[i]), hi = std::min(p1, p->woff[i + 1]);
            const unsigned v = p->h_victims[i];
            char* dst = p->host + p->host_off[v] + (lo - p->woff[i]) * p->unit_bytes;
            const char* src = slot + (lo - p0) * p->unit_bytes;
            TRY_HIP(p, copy_async(dst, src, (hi - lo) * p->unit_bytes, hipMemcpyDeviceToHost,
                                  p->st_out), true);
        }
        if (timing) TRY_HIP(p, hipEventRecord(tp->b, p->st_out), true);
    }
    TRY_HIP(p, hipEventRecord(p->ev_out_done, so), true);
    p->state = kPacked;
    return SS_OK;
}

ss_status ss_prefetch_unpack(ss_pool* p, void* stream) {
    ss_status st = check_usable(p);
    if (st) return st;
    if (p->state != kPacked)
        return set_err(SS_ERR_ORDER, "ss_prefetch_unpack must follow ss_evict_pack");
    DeviceGuard g(p->device);
    hipStream_t caller = static_cast<hipStream_t>(stream);
    const bool timing = p->flags & SS_FLAG_TIMING;
    hipStream_t si = p->inline_step ? caller : p->st_in;
    if (!p->inline_step) {
        TRY_HIP(p, hipEventRecord(p->ev_caller, caller), true);
        TRY_HIP(p, hipStreamWaitEvent(p->st_in, p->ev_caller, 0), true);
    }
    // the unpacks write units the block-table update assigns (as in
    // ss_evict_pack, the wait is implied when the plan ran on this stream)
    if (caller != p->bt_stream) TRY_HIP(p, hipStreamWaitEvent(si, bt_event(p), 0), true);

    const u64 total = p->res.units_in;
    const u64 ups = p->units_per_slot;
    const bool direct = p->direct_bytes && total && total * p->unit_bytes <= p->direct_bytes;
    const u64 nslots = direct ? 0 : (total + ups - 1) / ups;
    const u64 nF = p->res.n_free_used;
    CopyArgs C{};
    C.units_list = p->d_lunits;
    C.items = p->d_items;
    C.n_items = p->n_items;
    C.item_groups = (p->n_items + kCopyWavesPerBlock - 1) / kCopyWavesPerBlock;
    C.run_order = p->n_items == p->P;
    C.plane_base = p->d_plane_base;
    C.chunk_bytes = p->d_chunk_bytes;
    C.unit_bytes = p->unit_bytes;
    C.capacity = p->U;
    if (direct && !p->duplex_step) {
        // one launch scatters every load straight from its host copy; units
        // released this step are overwritten only after the packs read them
        // (a duplex step's loads moved with its write-backs)
        if (total > nF && p->n_pack_step)
            TRY_HIP(p, hipStreamWaitEvent(si, p->ev_packed[p->n_pack_step - 1], 0), true);
        C.first = 0;
        C.count = total;
        C.staging = p->host_dev;
        C.stage_off = p->d_lhost;
        TimedPair* tp = nullptr;
        if (timing) {
            TRY_HIP(p, timed_pair(p->t_din, p->n_t_din++, &tp), true);
            tp->bytes = total * p->unit_bytes;
            TRY_HIP(p, hipEventRecord(tp->a, si), true);
        }
        TRY_HIP(p, launch_unpack(C, si), true);
        if (timing) TRY_HIP(p, hipEventRecord(tp->b, si), true);
    }
    size_t li = 0, ri = 0;
    // host-to-device copies of slot k into the ring
    auto issue_h2d = [&](u64 k) -> ss_status {
        const u64 q0 = k * ups, q1 = std::min(total, q0 + ups);
        char* slot = p->stage_in + (k % p->ring) * p->slot_bytes;
        TimedPair* tp = nullptr;
        if (timing) {
            TRY_HIP(p, timed_pair(p->t_h2d, p->n_t_h2d++, &tp), true);
            tp->bytes = (q1 - q0) * p->unit_bytes;
            TRY_HIP(p, hipEventRecord(tp->a, p->st_in), true);
        }
        while (li < p->res.n_loads && p->loff[li + 1] <= q0) li++;
        for (size_t i = li; i < p->res.n_loads && p->loff[i] < q1; ++i) {
            const u64 lo = std::max(q0, p->loff[i]), hi = std::min(q1, p->loff[i + 1]);
            const unsigned a = p->h_loads[i];
            const char* src = p->host + p->host_off[a] + (lo - p->loff[i]) * p->unit_bytes;
            char* dst = slot + (lo - q0) * p->unit_bytes;
            TRY_HIP(p, copy_async(dst, src, (hi - lo) * p->unit_bytes, hipMemcpyHostToDevice,
                                  p->st_in), true);
        }
        if (timing) TRY_HIP(p, hipEventRecord(tp->b, p->st_in), true);
        return SS_OK;
    };
    // unpack of slot k
    auto issue_unpack = [&](u64 k) -> ss_status {
        const u64 q0 = k * ups, q1 = std::min(total, q0 + ups);
        char* slot = p->stage_in + (k % p->ring) * p->slot_bytes;
        // units released by victims are overwritten only after the pack read
        // them: released positions [r0, r1) of this slot; the last written-back
        // victim overlapping them gives the last pack slot to wait for
        if (q1 > nF) {
            const u64 r0 = q0 > nF ? q0 - nF : 0, r1 = q1 - nF;
            while (ri + 1 < p->res.n_victims && p->voff[ri + 1] < r1) ri++;
            const long long j = p->res.n_victims ? p->last_written[ri] : -1;
            if (j >= 0 && p->voff[j + 1] > r0) {
                const u64 maxpos = p->woff[j] + std::min(r1, p->voff[j + 1]) - p->voff[j] - 1;
                const u64 ps = p->direct_out ? 0 : maxpos / ups;     // a direct pack is one launch
                TRY_HIP(p, hipStreamWaitEvent(p->st_in, p->ev_packed[ps], 0), true);
            }
        }
        // the pack of slot k + 1 becomes ready (its ring slot's device-to-host
        // copy done) about when this slot's host-to-device copy lands: let it
        // finish first, so the two HBM-bound kernels do not share HBM
        if (!p->direct_out && k + 1 < p->n_pack_step)
            TRY_HIP(p, hipStreamWaitEvent(p->st_in, p->ev_packed[k + 1], 0), true);
        C.first = q0;
        C.count = q1 - q0;
        C.staging = slot;
        TimedPair* tp = nullptr;
        if (timing) {
            TRY_HIP(p, timed_pair(p->t_unpack, p->n_t_unpack++, &tp), true);
            tp->bytes = (q1 - q0) * p->unit_bytes;
            TRY_HIP(p, hipEventRecord(tp->a, p->st_in), true);
        }
        TRY_HIP(p, launch_unpack(C, p->st_in), true);
        if (timing) TRY_HIP(p, hipEventRecord(tp->b, p->st_in), true);
        return SS_OK;
    };
    // With two or more ring slots the copy of slot k + 1 is queued before the
    // unpack of slot k, so the copy engine never waits for an unpack (stream
    // order still refills a slot only after the unpack that read it, ring
    // slots earlier).  With one slot they alternate.
    for (u64 k = 0; k < nslots; ++k) {
        if (p->ring >= 2) {
            st = issue_h2d(k);
            if (!st && k >= 1) st = issue_unpack(k - 1);
        } else {
            st = issue_h2d(k);
            if (!st) st = issue_unpack(k);
        }
        if (st) return st;
    }
    if (p->ring >= 2 && nslots) {
        st = issue_unpack(nslots - 1);
        if (st) return st;
    }
    TRY_HIP(p, hipEventRecord(p->ev_in_done, si), true);
    if (!p->inline_step) {
        TRY_HIP(p, hipStreamWaitEvent(caller, p->ev_in_done, 0), true);
        TRY_HIP(p, hipStreamWaitEvent(caller, p->ev_out_done, 0), true);
    } else {
        // an eviction queued on another caller stream
        TRY_HIP(p, hipStreamWaitEvent(caller, p->ev_out_done, 0), true);
    }
    // `caller` now follows the whole step (both directions)
    p->joined_stream = caller;
    p->joined_valid = true;
    p->state = kIdle;
    return SS_OK;
}

ss_status ss_block_table(ss_pool* p, const int32_t** d_units, const uint64_t** d_agent_off) {
    if (!p || !d_units || !d_agent_off) return set_err(SS_ERR_ARG, "NULL argument");
    *d_units = p->d_bt;
    *d_agent_off = reinterpret_cast<const uint64_t*>(p->d_agent_off);
    return SS_OK;
}

ss_status ss_block_table_host(ss_pool* p, uint32_t agent, int32_t* out, uint32_t cap, uint32_t* n) {
    ss_status st = check_usable(p);
    if (st) return st;
    if (!out || !n || agent >= p->N) return set_err(SS_ERR_ARG, "bad agent or NULL output");
    const uint32_t s = p->s[agent];
    *n = s;
    if (cap < s) return set_err(SS_ERR_ARG, "cap %u < %u units", cap, s);
    DeviceGuard g(p->device);
    u64 off = 0;
    for (uint32_t a = 0; a < agent; ++a) off += p->s[a];
    TRY_HIP(p, hipStreamSynchronize(p->st_out), false);
    TRY_HIP(p, hipEventSynchronize(bt_event(p)), false);  // an update queued on a caller's stream
    TRY_HIP(p, hipMemcpy(out, p->d_bt + off, s * sizeof(int32_t), hipMemcpyDeviceToHost), false);
    return SS_OK;
}

ss_status ss_block_table_host_all(ss_pool* p, int32_t* out, uint64_t cap, uint64_t* n) {
    ss_status st = check_usable(p);
    if (st) return st;
    if (!out || !n) return set_err(SS_ERR_ARG, "NULL output");
    u64 total = 0;
    for (uint32_t a = 0; a < p->N; ++a) total += p->s[a];
    *n = total;
    if (cap < total) return set_err(SS_ERR_ARG, "cap %llu < %llu entries", (unsigned long long)cap,
                                    (unsigned long long)total);
    DeviceGuard g(p->device);
    TRY_HIP(p, hipStreamSynchronize(p->st_out), false);
    TRY_HIP(p, hipEventSynchronize(bt_event(p)), false);  // an update queued on a caller's stream
    TRY_HIP(p, hipMemcpy(out, p->d_bt, total * sizeof(int32_t), hipMemcpyDeviceToHost), false);
    return SS_OK;
}

ss_status ss_resident_host(ss_pool* p, uint8_t* out) {
    ss_status st = check_usable(p);
    if (st) return st;
    if (!out) return set_err(SS_ERR_ARG, "NULL output");
    DeviceGuard g(p->device);
    TRY_HIP(p, hipStreamSynchronize(p->st_out), false);
    TRY_HIP(p, hipEventSynchronize(bt_event(p)), false);  // an update queued on a caller's stream
    TRY_HIP(p, hipMemcpy(out, p->d_resident, p->N, hipMemcpyDeviceToHost), false);
    return SS_OK;
}

ss_status ss_get_stats(ss_pool* p, ss_stats* out) {
    if (!p || !out) return set_err(SS_ERR_ARG, "NULL argument");
    DeviceGuard g(p->device);
    for (hipStream_t s : {p->st_out, p->st_in})
        TRY_HIP(p, hipStreamSynchronize(s), false);
    ss_status st = collect_all_timing(p);
    if (st) return st;
    *out = p->stats;
    return SS_OK;
}

ss_status ss_reset_stats(ss_pool* p) {
    if (!p) return set_err(SS_ERR_ARG, "NULL pool");
    DeviceGuard g(p->device);
    for (hipStream_t s : {p->st_out, p->st_in})
        TRY_HIP(p, hipStreamSynchronize(s), false);
    ss_status st = collect_all_timing(p);
    if (st) return st;
    p->stats = ss_stats{};
    return SS_OK;
}

ss_status ss_sync(ss_pool* p) {
    ss_status st = check_usable(p);
    if (st) return st;
    DeviceGuard g(p->device);
    for (hipStream_t s : {p->st_out, p->st_in})
        TRY_HIP(p, wait_stream(p, s), true);
    // work of a step that ran on a caller's stream
    for (hipEvent_t e : {p->ev_planned, p->ev_out_done, p->ev_in_done})
        TRY_HIP(p, wait_event(p, e), true);
    return SS_OK;
}

ss_status ss_device_count(int32_t* n) {
    if (!n) return set_err(SS_ERR_ARG, "NULL output");
    int c = 0;
    if (hipGetDeviceCount(&c) != hipSuccess) {
        (void)hipGetLastError();
        c = 0;
    }
    *n = c;
    return SS_OK;
}

ss_status ss_device_alloc(int32_t device, uint64_t bytes, void** out) {
    if (!out || bytes == 0) return set_err(SS_ERR_ARG, "bad allocation arguments");
    *out = nullptr;
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || device < 0 || device >= ndev) {
        (void)hipGetLastError();
        return set_err(SS_ERR_ARG, "device %d not present", (int)device);
    }
    DeviceGuard g(device);
    hipError_t e = hipMalloc(out, bytes);
    if (e != hipSuccess) {
        *out = nullptr;
        return set_err(e == hipErrorOutOfMemory ? SS_ERR_NOMEM : SS_ERR_HIP,
                       "hipMalloc(%llu) failed: %s", (unsigned long long)bytes, hipGetErrorString(e));
    }
    return SS_OK;
}

ss_status ss_host_alloc(uint64_t bytes, void** out) {
    if (!out || bytes == 0) return set_err(SS_ERR_ARG, "bad allocation arguments");
    *out = nullptr;
    hipError_t e = hipHostMalloc(out, bytes, hipHostMallocDefault);
    if (e != hipSuccess) {
        *out = nullptr;
        return set_err(e == hipErrorOutOfMemory ? SS_ERR_NOMEM : SS_ERR_HIP,
                       "hipHostMalloc(%llu) failed: %s", (unsigned long long)bytes,
                       hipGetErrorString(e));
    }
    return SS_OK;
}

ss_status ss_device_free(void* ptr) {
    if (ptr) TRY_HIP(nullptr, hipFree(ptr), false);
    return SS_OK;
}

ss_status ss_host_free(void* ptr) {
    if (ptr) TRY_HIP(nullptr, hipHostFree(ptr), false);
    return SS_OK;
}

ss_status ss_copy(void* dst, const void* src, uint64_t bytes) {
    if (!dst || !src) return set_err(SS_ERR_ARG, "NULL pointer");
    if (bytes == 0) return SS_OK;
    TRY_HIP(nullptr, hipMemcpy(dst, src, bytes, hipMemcpyDefault), false);
    return SS_OK;
}

ss_status ss_stream_create(void** stream) {
    if (!stream) return set_err(SS_ERR_ARG, "NULL output");
    hipStream_t s = nullptr;
    TRY_HIP(nullptr, hipStreamCreateWithFlags(&s, hipStreamNonBlocking), false);
    *stream = s;
    return SS_OK;
}

ss_status ss_stream_destroy(void* stream) {
    if (stream) TRY_HIP(nullptr, hipStreamDestroy(static_cast<hipStream_t>(stream)), false);
    return SS_OK;
}

ss_status ss_stream_sync(void* stream) {
    TRY_HIP(nullptr, hipStreamSynchronize(static_cast<hipStream_t>(stream)), false);
    return SS_OK;
}

ss_status ss_event_create(void** event) {
    if (!event) return set_err(SS_ERR_ARG, "NULL output");
    hipEvent_t e = nullptr;
    TRY_HIP(nullptr, hipEventCreate(&e), false);
    *event = e;
    return SS_OK;
}

ss_status ss_event_destroy(void* event) {
    if (event) TRY_HIP(nullptr, hipEventDestroy(static_cast<hipEvent_t>(event)), false);
    return SS_OK;
}

ss_status ss_event_record(void* event, void* stream) {
    if (!event) return set_err(SS_ERR_ARG, "NULL event");
    TRY_HIP(nullptr, hipEventRecord(static_cast<hipEvent_t>(event), static_cast<hipStream_t>(stream)),
            false);
    return SS_OK;
}

ss_status ss_event_elapsed(void* start, void* end, float* ms) {
    if (!start || !end || !ms) return set_err(SS_ERR_ARG, "NULL argument");
    TRY_HIP(nullptr, hipEventSynchronize(static_cast<hipEvent_t>(end)), false);
    TRY_HIP(nullptr, hipEventElapsedTime(ms, static_cast<hipEvent_t>(start),
                                         static_cast<hipEvent_t>(end)), false);
    return SS_OK;
}

ss_status ss_probe_copy(void* dst, const void* src, uint64_t bytes, int iters, float* ms) {
    if (!dst || !src || !ms || iters < 1 || bytes == 0 || bytes % 16)
        return set_err(SS_ERR_ARG, "bad probe arguments");
    hipEvent_t a, b;
    TRY_HIP(nullptr, make_event(&a, true), false);
    TRY_HIP(nullptr, make_event(&b, true), false);
    hipStream_t s;
    TRY_HIP(nullptr, hipStreamCreateWithFlags(&s, hipStreamNonBlocking), false);
    hipError_t e = launch_probe_copy(dst, src, bytes, s);                 // warm-up
    if (e == hipSuccess) e = hipEventRecord(a, s);
    for (int i = 0; i < iters && e == hipSuccess; ++i) e = launch_probe_copy(dst, src, bytes, s);
    if (e == hipSuccess) e = hipEventRecord(b, s);
    if (e == hipSuccess) e = hipEventSynchronize(b);
    float t = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&t, a, b);
    (void)hipStreamDestroy(s);
    (void)hipEventDestroy(a);
    (void)hipEventDestroy(b);
    if (e != hipSuccess) return hip_fail(nullptr, e, "probe copy", false);
    *ms = t / iters;
    return SS_OK;
}

ss_status ss_probe_launch(int iters, float* us) {
    if (!us || iters < 1) return set_err(SS_ERR_ARG, "bad probe arguments");
    hipEvent_t ev;
    hipStream_t s;
    TRY_HIP(nullptr, make_event(&ev, false), false);
    TRY_HIP(nullptr, hipStreamCreateWithFlags(&s, hipStreamNonBlocking), false);
    std::vector<float> t;
    hipError_t e = launch_nop(s);                                        // warm-up
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    for (int i = 0; i < iters && e == hipSuccess; ++i) {
        const auto t0 = std::chrono::steady_clock::now();
        e = launch_nop(s);
        if (e == hipSuccess) e = hipEventRecord(ev, s);
        if (e == hipSuccess) e = hipEventSynchronize(ev);
        t.push_back(std::chrono::duration<float, std::micro>(std::chrono::steady_clock::now() - t0)
                        .count());
    }
    (void)hipStreamDestroy(s);
    (void)hipEventDestroy(ev);
    if (e != hipSuccess) return hip_fail(nullptr, e, "probe launch", false);
    std::sort(t.begin(), t.end());
    *us = t[t.size() / 2];
    return SS_OK;
}

ss_status ss_probe_link(void* host, void* dev, uint64_t bytes, int dir, int iters, float* ms) {
    if (!host || !dev || !ms || iters < 1 || bytes == 0 || dir < 0 || dir > 2)
        return set_err(SS_ERR_ARG, "bad probe arguments");
    hipEvent_t a, b, c;
    hipStream_t s1, s2;
    TRY_HIP(nullptr, make_event(&a, true), false);
    TRY_HIP(nullptr, make_event(&b, true), false);
    TRY_HIP(nullptr, make_event(&c, false), false);
    TRY_HIP(nullptr, hipStreamCreateWithFlags(&s1, hipStreamNonBlocking), false);
    TRY_HIP(nullptr, hipStreamCreateWithFlags(&s2, hipStreamNonBlocking), false);
    char* h = static_cast<char*>(host);
    char* d = static_cast<char*>(dev);
    hipError_t e = hipSuccess;
    auto issue = [&](hipStream_t st, int which) {
        if (which == 0) return hipMemcpyAsync(d, h, bytes, hipMemcpyHostToDevice, st);
        return hipMemcpyAsync(h + (dir == 2 ? bytes : 0), d + (dir == 2 ? bytes : 0), bytes,
                              hipMemcpyDeviceToHost, st);
    };
    for (int w = 0; w < 2 && e == hipSuccess; ++w) {               // warm-up, then timed
        if (e == hipSuccess) e = hipEventRecord(a, s1);
        if (e == hipSuccess) e = hipStreamWaitEvent(s2, a, 0);
        for (int i = 0; i < (w ? iters : 1) && e == hipSuccess; ++i) {
            if (dir == 0 || dir == 2) e = issue(s1, 0);
            if (e == hipSuccess && dir == 1) e = issue(s1, 1);
            if (e == hipSuccess && dir == 2) e = issue(s2, 1);
        }
        if (e == hipSuccess) e = hipEventRecord(c, s2);
        if (e == hipSuccess) e = hipStreamWaitEvent(s1, c, 0);
        if (e == hipSuccess) e = hipEventRecord(b, s1);
        if (e == hipSuccess) e = hipEventSynchronize(b);
    }
    float t = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&t, a, b);
    (void)hipStreamDestroy(s1);
    (void)hipStreamDestroy(s2);
    (void)hipEventDestroy(a);
    (void)hipEventDestroy(b);
    (void)hipEventDestroy(c);
    if (e != hipSuccess) return hip_fail(nullptr, e, "probe link", false);
    *ms = t / iters;
    return SS_OK;
}

}  // extern "C"
