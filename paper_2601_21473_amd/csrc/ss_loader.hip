// Load-task scheduler with preemption (Appendix A, "Load task scheduler" and
// "Preemption support"): the C ABI ss_loader_* declared in include/scalesim.h.
//
// One scheduler serves every registered memory module, so all CPU-to-GPU
// loads are ordered by one key, (distance, agent, module).  A task loads one
// agent's memory of one module into destination units the caller names (for
// instance the agent's block-table row) and runs as chunks of whole units:
// a hipMemcpyAsync of the chunk's bytes from the agent's pinned host copy
// into a staging slot of the module, then the pool's unpack kernel
// (k_copy<false>) scattering the slot into the destination units.
//
// The preemption signal is checked before every chunk: when a queued task
// has a strictly smaller distance than the running one, the running task
// goes back into the queue with its progress and the urgent task runs.  The
// host keeps at most `window` chunks in flight (the smallest ring of the
// modules) and takes each decision only after the chunk `window` places
// earlier has finished, so an urgent task submitted from another thread
// waits for at most `window` chunks.  Copies run in issue order on a copy
// stream and unpacks in issue order on a compute stream (both non-blocking,
// default priority): each unpack waits for its chunk's copy, and a copy into
// a staging slot waits for the unpack that last read the slot, so the copy
// engine moves the next chunk while the previous one is unpacked.
#include "scalesim.h"
#include "ss_internal.h"

#include <algorithm>
#include <map>
#include <mutex>
#include <new>
#include <set>
#include <tuple>
#include <vector>

using namespace ss;

namespace {

struct Module {
    u64 U = 0;
    unsigned P = 0;
    u64 unit_bytes = 0;
    std::vector<uint32_t> s;          // units per agent
    std::vector<u64> host_off;
    char* host = nullptr;
    char* staging = nullptr;
    u64 slot_bytes = 0;
    unsigned slots = 0, next_slot = 0;
    unsigned chunk_units = 0;
    std::vector<hipEvent_t> slot_free;  // recorded after the unpack that read each slot
    std::vector<bool> slot_used;
    CopyItem* d_items = nullptr;
    unsigned n_items = 0;
    u64* d_plane_base = nullptr;
    u64* d_chunk_bytes = nullptr;
};

struct Task {
    uint32_t dist = 0;
    uint32_t cursor = 0;              // units issued
    const int32_t* units = nullptr;   // device: destination unit of each logical unit
};

typedef std::tuple<uint32_t, uint32_t, uint32_t> Key;   // (distance, agent, module)
typedef std::pair<uint32_t, uint32_t> Id;                // (module, agent)

}  // namespace

struct ss_loader {
    std::vector<Module> mods;
    int device = 0;
    bool preempt = true;
    hipStream_t st = nullptr;         // unpacks
    hipStream_t cp = nullptr;         // host-to-device copies
    hipEvent_t copied = nullptr;      // recorded after each copy, waited on by its unpack
    std::vector<hipEvent_t> window;   // one per chunk in flight (after its unpack)
    u64 issued_total = 0;
    std::map<Id, Task> tasks;
    std::set<Key> queue;              // tasks not running
    bool running = false;
    Id run{0, 0};
    bool poisoned = false;
    ss_loader_stats stats{};
    std::mutex mu;
};

namespace {

ss_status hip_err(ss_loader* L, hipError_t e, const char* what) {
    if (L) L->poisoned = true;
    return set_err(SS_ERR_HIP, "%s failed: %s", what, hipGetErrorString(e));
}

#define L_TRY(L, expr)                                                 \
    do {                                                               \
        hipError_t _e = (expr);                                        \
        if (_e != hipSuccess) return hip_err((L), _e, #expr);          \
    } while (0)

struct DeviceScope {
    int prev = -1;
    explicit DeviceScope(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        if (prev != dev) (void)hipSetDevice(dev);
    }
    ~DeviceScope() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

void free_loader(ss_loader* L) {
    if (!L) return;
    if (L->cp) (void)hipStreamSynchronize(L->cp);
    if (L->st) (void)hipStreamSynchronize(L->st);
    for (Module& m : L->mods) {
        for (hipEvent_t e : m.slot_free)
            if (e) (void)hipEventDestroy(e);
        if (m.d_items) (void)hipFree(m.d_items);
        if (m.d_plane_base) (void)hipFree(m.d_plane_base);
        if (m.d_chunk_bytes) (void)hipFree(m.d_chunk_bytes);
    }
    for (hipEvent_t e : L->window)
        if (e) (void)hipEventDestroy(e);
    if (L->copied) (void)hipEventDestroy(L->copied);
    if (L->st) (void)hipStreamDestroy(L->st);
    if (L->cp) (void)hipStreamDestroy(L->cp);
    delete L;
}

ss_status check_module(const ss_pool_desc* d, uint32_t i) {
    if (!d->n_agents || d->n_agents >= (1u << 31))
        return set_err(SS_ERR_ARG, "module %u: n_agents must be in [1, 2^31)", i);
    if (!d->capacity_units || d->capacity_units >= (1ull << 31))
        return set_err(SS_ERR_ARG, "module %u: capacity_units must be in [1, 2^31)", i);
    if (!d->n_planes || !d->plane_base || !d->chunk_bytes || !d->agent_units)
        return set_err(SS_ERR_ARG, "module %u: planes, chunk sizes and agent units are required", i);
    if (!d->host_backing || !d->dev_staging || !d->ring_slots)
        return set_err(SS_ERR_ARG, "module %u: host_backing, dev_staging and ring_slots are required",
                       i);
    u64 ub = 0;
    for (uint32_t c = 0; c < d->n_planes; ++c) {
        if (!d->chunk_bytes[c] || d->chunk_bytes[c] % 16)
            return set_err(SS_ERR_ARG, "module %u: chunk_bytes[%u] is not a positive multiple of 16",
                           i, c);
        if (!d->plane_base[c] || reinterpret_cast<uintptr_t>(d->plane_base[c]) % 16)
            return set_err(SS_ERR_ARG, "module %u: plane_base[%u] is NULL or not 16-byte aligned", i,
                           c);
        ub += d->chunk_bytes[c];
    }
    if (reinterpret_cast<uintptr_t>(d->dev_staging) % 16)
        return set_err(SS_ERR_ARG, "module %u: dev_staging is not 16-byte aligned", i);
    const u64 slot = (d->staging_bytes / d->ring_slots) & ~15ull;
    if (slot < ub)
        return set_err(SS_ERR_ARG, "module %u: a staging slot (%llu bytes) holds no whole unit (%llu)",
                       i, (unsigned long long)slot, (unsigned long long)ub);
    u64 acc = 0;
    for (uint32_t a = 0; a < d->n_agents; ++a) {
        if (!d->agent_units[a]) return set_err(SS_ERR_ARG, "module %u: agent_units[%u] is 0", i, a);
        const u64 off = d->host_off ? d->host_off[a] : acc;
        const u64 len = (u64)d->agent_units[a] * ub;
        if (off > d->host_bytes || len > d->host_bytes - off)
            return set_err(SS_ERR_ARG, "module %u: host copy of agent %u exceeds host_bytes", i, a);
        acc += len;
    }
    return SS_OK;
}

}  // namespace

extern "C" {

ss_status ss_loader_create(const ss_pool_desc* modules, uint32_t n_modules, uint32_t flags,
                           ss_loader** out) {
    if (!modules || !n_modules || !out) return set_err(SS_ERR_ARG, "modules and out are required");
    if (flags & ~SS_LOADER_NO_PREEMPT) return set_err(SS_ERR_ARG, "unknown flag bits");
    const int dev = modules[0].device;
    for (uint32_t i = 0; i < n_modules; ++i) {
        ss_status st = check_module(&modules[i], i);
        if (st != SS_OK) return st;
        if (modules[i].device != dev)
            return set_err(SS_ERR_ARG, "all modules of a loader must be on one device");
    }
    int n_dev = 0;
    if (hipGetDeviceCount(&n_dev) != hipSuccess || dev < 0 || dev >= n_dev) {
        (void)hipGetLastError();
        return set_err(SS_ERR_ARG, "device %d not present", (int)dev);
    }
    DeviceScope g(dev);
    for (uint32_t i = 0; i < n_modules; ++i) {
        const ss_pool_desc& d = modules[i];
        for (uint32_t c = 0; c < d.n_planes; ++c)
            if (!device_range_ok(d.plane_base[c], d.capacity_units * d.chunk_bytes[c], dev))
                return set_err(SS_ERR_ARG, "module %u plane %u is not device memory of device %d", i,
                               c, dev);
        if (!device_range_ok(d.dev_staging, d.staging_bytes, dev))
            return set_err(SS_ERR_ARG, "module %u: dev_staging is not device memory", i);
        if (!pinned_range_ok(d.host_backing, d.host_bytes))
            return set_err(SS_ERR_ARG, "module %u: host_backing is not pinned host memory", i);
    }
    ss_loader* L = new (std::nothrow) ss_loader();
    if (!L) return set_err(SS_ERR_NOMEM, "out of host memory");
    L->device = dev;
    L->preempt = !(flags & SS_LOADER_NO_PREEMPT);
    L->mods.resize(n_modules);
    unsigned window = ~0u;
#define C_TRY(expr)                                                    \
    do {                                                               \
        hipError_t _e = (expr);                                        \
        if (_e != hipSuccess) {                                        \
            ss_status _s = hip_err(nullptr, _e, #expr);                \
            free_loader(L);                                            \
            return _s;                                                 \
        }                                                              \
    } while (0)
    for (uint32_t i = 0; i < n_modules; ++i) {
        const ss_pool_desc& d = modules[i];
        Module& m = L->mods[i];
        m.U = d.capacity_units;
        m.P = d.n_planes;
        m.s.assign(d.agent_units, d.agent_units + d.n_agents);
        std::vector<CopyItem> items;
        std::vector<u64> bases(m.P), cb(m.P);
        for (uint32_t c = 0; c < m.P; ++c) {
            for (u64 off = 0; off < d.chunk_bytes[c]; off += kItemBytes) {
                CopyItem it;
                it.plane = c;
                it.len = (unsigned)std::min<u64>(kItemBytes, d.chunk_bytes[c] - off);
                it.chunk_off = off;
                it.unit_off = m.unit_bytes + off;
                items.push_back(it);
            }
            m.unit_bytes += d.chunk_bytes[c];
            bases[c] = reinterpret_cast<u64>(d.plane_base[c]);
            cb[c] = d.chunk_bytes[c];
        }
        m.host_off.resize(d.n_agents);
        u64 acc = 0;
        for (uint32_t a = 0; a < d.n_agents; ++a) {
            m.host_off[a] = d.host_off ? d.host_off[a] : acc;
            acc += (u64)m.s[a] * m.unit_bytes;
        }
        m.host = static_cast<char*>(d.host_backing);
        m.staging = static_cast<char*>(d.dev_staging);
        m.slots = d.ring_slots;
        m.slot_bytes = (d.staging_bytes / d.ring_slots) & ~15ull;
        m.chunk_units = (unsigned)std::min<u64>(m.slot_bytes / m.unit_bytes, 1u << 30);
        m.n_items = (unsigned)items.size();
        C_TRY(hipMalloc(reinterpret_cast<void**>(&m.d_items), items.size() * sizeof(CopyItem)));
        C_TRY(hipMalloc(reinterpret_cast<void**>(&m.d_plane_base), m.P * sizeof(u64)));
        C_TRY(hipMalloc(reinterpret_cast<void**>(&m.d_chunk_bytes), m.P * sizeof(u64)));
        C_TRY(hipMemcpy(m.d_items, items.data(), items.size() * sizeof(CopyItem),
                        hipMemcpyHostToDevice));
        C_TRY(hipMemcpy(m.d_plane_base, bases.data(), m.P * sizeof(u64), hipMemcpyHostToDevice));
        C_TRY(hipMemcpy(m.d_chunk_bytes, cb.data(), m.P * sizeof(u64), hipMemcpyHostToDevice));
        window = std::min(window, m.slots);
        m.slot_free.assign(m.slots, nullptr);
        m.slot_used.assign(m.slots, false);
        for (auto& e : m.slot_free) C_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    }
    C_TRY(hipStreamCreateWithFlags(&L->st, hipStreamNonBlocking));
    C_TRY(hipStreamCreateWithFlags(&L->cp, hipStreamNonBlocking));
    C_TRY(hipEventCreateWithFlags(&L->copied, hipEventDisableTiming));
    L->window.assign(window, nullptr);
    for (auto& e : L->window) C_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
#undef C_TRY
    *out = L;
    return SS_OK;
}

void ss_loader_destroy(ss_loader* L) {
    if (!L) return;
    DeviceScope g(L->device);
    free_loader(L);
}

ss_status ss_loader_submit(ss_loader* L, const ss_load_task* tasks, uint32_t n) {
    if (!L) return set_err(SS_ERR_ARG, "loader is NULL");
    if (n && !tasks) return set_err(SS_ERR_ARG, "tasks is NULL");
    std::lock_guard<std::mutex> lk(L->mu);
    if (L->poisoned) return set_err(SS_ERR_POISONED, "loader is poisoned by an earlier HIP failure");
    DeviceScope g(L->device);
    // validate every task before changing anything
    for (uint32_t i = 0; i < n; ++i) {
        const ss_load_task& t = tasks[i];
        if (t.module >= L->mods.size())
            return set_err(SS_ERR_ARG, "task %u: module %u out of range", i, t.module);
        const Module& m = L->mods[t.module];
        if (t.agent >= m.s.size())
            return set_err(SS_ERR_ARG, "task %u: agent %u out of range", i, t.agent);
        if (L->tasks.count(Id(t.module, t.agent))) continue;       // distance update only
        if (!t.units || !device_range_ok(t.units, (u64)m.s[t.agent] * 4, L->device))
            return set_err(SS_ERR_ARG, "task %u: units must be device memory of %u entries", i,
                           m.s[t.agent]);
    }
    for (uint32_t i = 0; i < n; ++i) {
        const ss_load_task& t = tasks[i];
        const Id id(t.module, t.agent);
        auto it = L->tasks.find(id);
        if (it == L->tasks.end()) {
            Task T;
            T.dist = t.distance;
            T.units = t.units;
            L->tasks.emplace(id, T);
            L->queue.insert(Key(t.distance, t.agent, t.module));
            L->stats.submitted++;
            continue;
        }
        const bool is_running = L->running && L->run == id;
        if (!is_running) L->queue.erase(Key(it->second.dist, t.agent, t.module));
        it->second.dist = t.distance;
        if (!is_running) L->queue.insert(Key(t.distance, t.agent, t.module));
    }
    return SS_OK;
}

ss_status ss_loader_pump(ss_loader* L, uint32_t max_chunks, ss_load_log* log, uint32_t log_cap,
                         uint32_t* n_issued) {
    if (!L) return set_err(SS_ERR_ARG, "loader is NULL");
    if (log_cap && !log) return set_err(SS_ERR_ARG, "log is NULL");
    DeviceScope g(L->device);
    uint32_t issued = 0;
    if (n_issued) *n_issued = 0;
    while (issued < max_chunks) {
        // pace: the chunk `window` places back must have finished; the wait
        // runs without the lock so that submissions (the preemption signal)
        // can arrive meanwhile
        hipEvent_t ev;
        {
            std::lock_guard<std::mutex> lk(L->mu);
            if (L->poisoned) return set_err(SS_ERR_POISONED, "loader is poisoned");
            if (!L->running && L->queue.empty()) break;
            ev = L->issued_total >= L->window.size()
                     ? L->window[L->issued_total % L->window.size()] : nullptr;
        }
        if (ev) {
            hipError_t e = hipEventSynchronize(ev);
            if (e != hipSuccess) {
                std::lock_guard<std::mutex> lk(L->mu);
                return hip_err(L, e, "hipEventSynchronize");
            }
        }
        std::lock_guard<std::mutex> lk(L->mu);
        uint32_t flags = 0;
        if (!L->running) {
            if (L->queue.empty()) break;
            const Key k = *L->queue.begin();
            L->queue.erase(L->queue.begin());
            L->run = Id(std::get<2>(k), std::get<1>(k));
            L->running = true;
            flags |= SS_LOAD_START;
        } else if (L->preempt && !L->queue.empty() &&
                   std::get<0>(*L->queue.begin()) < L->tasks[L->run].dist) {
            L->queue.insert(Key(L->tasks[L->run].dist, L->run.second, L->run.first));
            const Key k = *L->queue.begin();
            L->queue.erase(L->queue.begin());
            L->run = Id(std::get<2>(k), std::get<1>(k));
            flags |= SS_LOAD_START | SS_LOAD_PREEMPT;
            L->stats.preemptions++;
        }
        Task& T = L->tasks[L->run];
        Module& m = L->mods[L->run.first];
        const uint32_t a = L->run.second;
        const uint32_t cnt = std::min<uint32_t>(m.chunk_units, m.s[a] - T.cursor);
        const unsigned slot = m.next_slot;
        m.next_slot = (slot + 1) % m.slots;
        char* stage = m.staging + (u64)slot * m.slot_bytes;
        // the copy refills the slot only after the unpack that last read it
        if (m.slot_used[slot]) L_TRY(L, hipStreamWaitEvent(L->cp, m.slot_free[slot], 0));
        L_TRY(L, copy_async(stage, m.host + m.host_off[a] + (u64)T.cursor * m.unit_bytes,
                            (u64)cnt * m.unit_bytes, hipMemcpyHostToDevice, L->cp));
        L_TRY(L, hipEventRecord(L->copied, L->cp));
        L_TRY(L, hipStreamWaitEvent(L->st, L->copied, 0));
        CopyArgs C{};
        C.units_list = T.units;
        C.first = T.cursor;
        C.count = cnt;
        C.items = m.d_items;
        C.n_items = m.n_items;
        C.item_groups = (m.n_items + kCopyWavesPerBlock - 1) / kCopyWavesPerBlock;
        C.run_order = m.n_items == m.P;
        C.plane_base = m.d_plane_base;
        C.chunk_bytes = m.d_chunk_bytes;
        C.staging = stage;
        C.unit_bytes = m.unit_bytes;
        C.capacity = m.U;
        L_TRY(L, launch_unpack(C, L->st));
        L_TRY(L, hipEventRecord(m.slot_free[slot], L->st));
        m.slot_used[slot] = true;
        L_TRY(L, hipEventRecord(L->window[L->issued_total % L->window.size()], L->st));
        L->issued_total++;
        const uint32_t first = T.cursor;
        T.cursor += cnt;
        L->stats.chunks++;
        L->stats.bytes += (u64)cnt * m.unit_bytes;
        if (T.cursor == m.s[a]) {
            flags |= SS_LOAD_DONE;
            L->tasks.erase(L->run);
            L->running = false;
            L->stats.completed++;
        }
        if (issued < log_cap) log[issued] = ss_load_log{L->run.first, a, first, cnt, flags, 0u};
        issued++;
        if (n_issued) *n_issued = issued;
    }
    return SS_OK;
}

ss_status ss_loader_pending(ss_loader* L, uint32_t* queued, uint32_t* running) {
    if (!L) return set_err(SS_ERR_ARG, "loader is NULL");
    std::lock_guard<std::mutex> lk(L->mu);
    if (queued) *queued = (uint32_t)L->queue.size();
    if (running) *running = L->running ? 1u : 0u;
    return SS_OK;
}

ss_status ss_loader_sync(ss_loader* L) {
    if (!L) return set_err(SS_ERR_ARG, "loader is NULL");
    DeviceScope g(L->device);
    L_TRY(L, hipStreamSynchronize(L->cp));
    L_TRY(L, hipStreamSynchronize(L->st));
    return SS_OK;
}

ss_status ss_loader_get_stats(ss_loader* L, ss_loader_stats* out) {
    if (!L || !out) return set_err(SS_ERR_ARG, "NULL argument");
    std::lock_guard<std::mutex> lk(L->mu);
    *out = L->stats;
    return SS_OK;
}

}  // extern "C"
