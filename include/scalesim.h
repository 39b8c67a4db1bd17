/*
 * scalesim.h -- C ABI of the per-step hot path of an invocation-distance
 * memory manager for agent-specific GPU memory (prefix KV pages, LoRA
 * adapter slots) on one AMD Instinct MI355X (gfx950).
 *
 * The operations follow the paper's memory-module interface (ScaleSim,
 * Appendix A, Table "agent-mem-interface"):
 *   HandleReq(req, agentID)            -> the per-step activation mask;
 *   Evict(size, agentDistances)        -> the demand half of ss_plan_step;
 *   DispatchLoadTasks(agentDistances, threshold, budget)
 *                                      -> the prefetch half of ss_plan_step;
 *   Load(memObj, agentIDs, ...)        -> ss_prefetch_unpack;
 * with eviction writing memory back to its host copy (Section 3.3,
 * "Future reuse-aware eviction") -> ss_evict_pack.  One ss_pool is one
 * registered memory module (Appendix A); several modules are several pools
 * planned with the same distances and mask.
 *
 * Data model.  A pool has `capacity_units` physical units.  A unit is made of
 * `n_planes` planes: the chunk of plane c of unit u lives at
 *     plane_base[c] + u * chunk_bytes[c]          (device memory).
 * Agent a owns agent_units[a] >= 1 units, logical units j = 0..s[a]-1, and
 * a host copy of them at host_backing + host_off[a]: unit j, then plane c,
 * each chunk contiguous (s[a] * unit_bytes bytes in all).
 *
 * Decision rules (each the reading of a passage; the CPU oracle applies the
 * same ones):
 *   d[a]   = 0 if a is active (Section 3.3, prefetch example), else the
 *            caller's distance estimate (Section 3.2; only order matters);
 *   key[a] = (d[a], a) compared lexicographically: ties go to the agent id;
 *   demand = active agents not resident, loaded in id order; when the free
 *            units cannot hold them, inactive residents are evicted largest
 *            key first, shortest prefix that frees enough (Section 3.3);
 *   prefetch = offloaded, inactive agents with distance < threshold, in
 *            increasing key; each is taken if it fits into free units or into
 *            units of further inactive residents with strictly larger
 *            distance, and the total stays within the budget; the first one
 *            that cannot be taken ends the prefetch (Section 3.3,
 *            "Distance-guided proactive prefetch"; Appendix A,
 *            DispatchLoadTasks);
 *   units  = loads receive the units free before the step in ascending index,
 *            then the units released by this step's victims in eviction
 *            order, in load order and logical-unit order.
 *
 * Threading and streams.  A pool is used by one host thread at a time.  The
 * library owns its internal HIP streams (all at the default priority).  Work
 * of a call starts after the work the caller has queued on `stream` before
 * the call; ss_prefetch_unpack makes `stream` wait for the whole step (both
 * directions of the copy) before the caller's later work on it, and the next
 * ss_plan_step's kernels start after the previous step's loads, evictions and
 * block-table update whatever stream each call is given.  A step whose moves
 * are all direct transfers (ss_pool_desc.direct_bytes) queues its kernels on
 * `stream` itself.
 *
 * Errors.  No C++ exception crosses this boundary.  Every call returns an
 * ss_status; ss_last_error() gives a message for the calling thread.
 * SS_ERR_ARG and SS_ERR_OVERCOMMIT leave the pool unchanged.  A HIP failure
 * while moving data poisons the pool: every later call returns
 * SS_ERR_POISONED (moves that were partly applied cannot be undone).
 */
#ifndef SCALESIM_H
#define SCALESIM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ss_pool ss_pool;     /* opaque; ss_pool_create / ss_pool_destroy */
typedef int32_t ss_status;

#define SS_OK               0
#define SS_ERR_ARG         (-1)     /* invalid argument; nothing changed            */
#define SS_ERR_OVERCOMMIT  (-2)     /* active agents need more units than the pool  */
#define SS_ERR_ORDER       (-3)     /* calls out of plan -> evict -> prefetch order */
#define SS_ERR_HIP         (-4)     /* a HIP runtime call failed                     */
#define SS_ERR_NOMEM       (-5)     /* the library could not allocate its metadata   */
#define SS_ERR_POISONED    (-6)     /* an earlier HIP failure left the pool unusable */

#define SS_NO_BUDGET       UINT64_MAX
#define SS_NO_DISTANCE     0xFFFFFFFFu  /* "never activated again"; never < threshold */

#define SS_FLAG_TIMING     1u       /* record HIP events around every copy launch   */
#define SS_FLAG_POLL_WAIT  2u       /* ss_sync and ss_get_stats poll the pool's
                                       streams and events instead of blocking: the
                                       calling thread spins while the device works,
                                       and the next call's launches cost their warm
                                       host time (after a blocking wait on long work
                                       a launch and its event record take 2-3 times
                                       as long)                                    */

typedef struct {
    uint32_t        n_agents;       /* N >= 1, N < 2^31                                    */
    uint64_t        capacity_units; /* U >= 1, U < 2^31                                    */
    uint32_t        n_planes;       /* P >= 1                                              */
    void* const*    plane_base;     /* [P] device pointers, plane c = U chunks (caller-owned) */
    const uint64_t* chunk_bytes;    /* [P] bytes per chunk, multiples of 16, >= 16         */
    const uint32_t* agent_units;    /* [N] units per agent, each >= 1 (copied)             */
    void*           host_backing;   /* pinned host memory from hipHostMalloc (caller-owned) */
    const uint64_t* host_off;       /* [N] byte offset of each agent's host copy (copied);
                                       NULL = packed, agent after agent. Offsets may alias
                                       (agents then share one host copy, as when one
                                       physical adapter serves many logical ones).       */
    uint64_t        host_bytes;     /* size of host_backing; every copy must fit           */
    void*           dev_staging;    /* device buffer (caller-owned): first half stages
                                       evictions, second half stages loads               */
    uint64_t        staging_bytes;  /* each half is cut into ring_slots slots of whole units */
    uint32_t        ring_slots;     /* >= 1 slots per direction                            */
    int32_t         device;         /* HIP device ordinal                                  */
    uint32_t        flags;          /* SS_FLAG_*                                           */
    uint64_t        direct_bytes;   /* a direction of a step that moves at most this many
                                       bytes runs as one kernel straight between the pool's
                                       units and the pinned host copies (no staging, no
                                       copy commands), which suits small steps where the
                                       latency of each copy dominates; larger steps use the
                                       staged pipeline.  When both directions of a step
                                       are direct and non-empty they run as one launch
                                       (each released unit written back, then loaded).
                                       0 = always staged.  host_backing must then be
                                       device-accessible pinned memory.  (The load
                                       scheduler ignores it.)                             */
} ss_pool_desc;

typedef struct {
    uint32_t threshold;             /* prefetch agents with distance < threshold (0 = off) */
    uint64_t budget_units;          /* max prefetched units per step; SS_NO_BUDGET = none  */
    const uint8_t* dirty;           /* [N] host or device, optional: 1 = the agent's memory changed
                                       since it was loaded, so an eviction writes it back;
                                       0 = its host copy is current and its units are
                                       released without a copy.  NULL = every eviction
                                       writes back (Section 3.3: evicted memory is restored
                                       from its host copy).                               */
} ss_plan_params;

typedef struct {
    uint32_t        n_victims;      /* agents evicted this step                         */
    uint32_t        n_loads;        /* agents loaded this step                          */
    uint32_t        n_demand;       /* leading loads that are demand loads              */
    uint32_t        n_demand_victims; /* leading victims evicted for demand             */
    const uint32_t* victims;        /* [n_victims] host, eviction order; pool-owned,
                                       valid until the next ss_plan_step               */
    const uint32_t* loads;          /* [n_loads] host: demand loads by id, then prefetches */
    uint64_t        units_out, units_in;   /* units released by victims / loaded    */
    uint64_t        bytes_out, bytes_in;   /* bytes written back / loaded           */
    uint64_t        units_written;         /* victims' units written back (<= units_out) */
    const uint8_t*  victim_written;        /* [n_victims] host: 1 = written back     */
    const uint32_t* d_victims;      /* [n_victims] DEVICE mirror of `victims`; pool-owned.
                                       Written by the plan kernel on the call's stream:
                                       work queued on that stream after the call (or any
                                       work after ss_sync) may read it until the next
                                       ss_plan_step's kernel rewrites it               */
    const uint32_t* d_loads;        /* [n_loads] DEVICE mirror of `loads`, same terms    */
} ss_plan;

typedef struct {                    /* cumulative since create or ss_reset_stats          */
    uint64_t steps;
    uint64_t pack_launches, unpack_launches;
    uint64_t pack_bytes, unpack_bytes;     /* bytes moved (each read once, written once) */
    double   pack_ms, unpack_ms;           /* sum of per-launch event durations         */
    uint64_t d2h_bytes, h2d_bytes;
    double   d2h_ms, h2d_ms;               /* per step: first to last copy on its stream */
    double   plan_gpu_ms;                  /* plan kernels, from the first workgroup's
                                              entry to the end of the block-table update,
                                              by the kernels' own wall-clock stamps       */
    double   plan_phase_us[7];             /* plan phases up to the published plan
                                              (classify; the histogram cuts and the sorts
                                              of the evictable, demand and candidate sets
                                              with their unit prefixes; demand victims;
                                              the acceptance's LDS copy of the evictable
                                              prefix; acceptance; lists; the result and
                                              its publication); classify runs
                                              from the plan kernel's entry (its first
                                              workgroup when N > 12288).  The free-unit
                                              pick and the block-table update follow in
                                              plan_gpu_ms only                             */
    double   plan_host_us[3];              /* ss_plan_step on the host: queueing the plan,
                                              waiting for it, reading it back              */
    uint64_t direct_out_launches, direct_in_launches;  /* directions moved by direct_bytes */
    uint64_t direct_out_bytes, direct_in_bytes;        /* (not counted in pack/unpack or
                                                          d2h/h2d above)                  */
    double   direct_out_ms, direct_in_ms;              /* event time of those launches    */
    double   plan_enqueue_us[4];           /* plan_host_us[0] in parts: checking (and
                                              copying) the inputs, queueing the stream
                                              waits, queueing the plan kernel and its
                                              events, the rest                             */
    uint64_t duplex_launches;              /* direct steps whose two directions moved in
                                              one launch (both non-empty, both within
                                              direct_bytes)                               */
    uint64_t duplex_bytes;                 /* their bytes, both directions (not counted
                                              in direct_out/in above)                     */
    double   duplex_ms;                    /* event time of those launches                */
} ss_stats;

/* Create a pool (Appendix A: register a memory module).  Validates every
 * descriptor field, copies the host arrays, allocates the library's device
 * metadata (block table, state, plan buffers; O(N + U + sum(s)) bytes) and its
 * streams.  The pool starts empty.  Returns SS_ERR_ARG (message in
 * ss_last_error) for an invalid descriptor, SS_ERR_HIP / SS_ERR_NOMEM on
 * runtime failures; *out is set only on SS_OK. */
ss_status ss_pool_create(const ss_pool_desc* desc, ss_pool** out);

/* Wait for the pool's queued work and free what the library allocated.
 * Caller-owned buffers are not touched.  NULL is ignored. */
void ss_pool_destroy(ss_pool* pool);

/* Plan one step (Section 3.3 and Appendix A, Evict + DispatchLoadTasks):
 * turns distances and the activation mask into victims and loads and updates
 * the block table.  `distances` [N] uint32 and `active` [N] uint8 (0/1), and
 * params->dirty [N] when given, are each either host memory (pageable or
 * pinned; the call copies them into pool-owned mapped pinned memory, which the
 * plan kernel reads over the host link, so the caller may reuse them once the
 * call returns) or device memory of the pool's device (read in place by the
 * call's kernels, which must not race with writers).  The kernels run on `stream`
 * after the work queued there before the call and after the previous step's
 * loads, evictions (packs and device-to-host copies) and block-table update
 * (when `stream` is the stream the previous ss_prefetch_unpack was given,
 * stream order already implies this and no wait is added; a stream handle is
 * identified by its value).  The call returns once the plan is known on
 * the host: the plan kernel writes its lists into mapped host memory and,
 * last, a sequence number that the call polls (for up to 2 ms, then it waits
 * on the kernel's completion event); by then the kernel has finished reading
 * its inputs, though it may still be ending on the device.  The
 * block-table update that the plan implies runs on `stream` after the plan is
 * published, in the plan kernel's own tail (after an overcommitted plan it
 * changes nothing); the copy kernels of ss_evict_pack and ss_prefetch_unpack
 * follow it whatever stream those calls are given.  Host inputs must hold N
 * readable elements; their copy into the mirrors is part of the call's host
 * time.  `out` receives the host lists and their device mirrors (ss_plan).
 * SS_ERR_OVERCOMMIT if the active agents need more than capacity_units
 * (pool unchanged).  SS_ERR_ARG (pool unchanged) if an input is device memory
 * of another device or a device range shorter than N elements.  SS_ERR_ORDER
 * if the previous step was not completed with ss_evict_pack and
 * ss_prefetch_unpack. */
ss_status ss_plan_step(ss_pool* pool, const uint32_t* distances, const uint8_t* active,
                       const ss_plan_params* params, ss_plan* out, void* stream);

/* Evict (Section 3.3: eviction writes the victims' memory back to host):
 * packs the written-back victims' units (victim, then logical unit, then
 * plane) into the eviction staging ring with the pack kernel and copies each
 * such victim's bytes to its host copy with hipMemcpyAsync, ring slot by ring
 * slot.  Clean victims (dirty mask) are not copied.  Returns once
 * queued.  SS_ERR_ORDER unless called right after ss_plan_step. */
ss_status ss_evict_pack(ss_pool* pool, void* stream);

/* Load (Appendix A, Load(memObj, agentIDs, ...)): copies every loaded agent's
 * host copy into the load staging ring with hipMemcpyAsync and scatters it
 * into the agent's new units with the unpack kernel on a side stream.  A slot
 * is unpacked only after the eviction has read every unit it overwrites, so
 * the two directions overlap.  `stream` then waits for the whole step.
 * SS_ERR_ORDER unless called right after ss_evict_pack. */
ss_status ss_prefetch_unpack(ss_pool* pool, void* stream);

/* The device block table in CSR form: agent a's logical unit j is physical
 * unit (*d_units)[(*d_agent_off)[a] + j], or -1 when a is not resident.
 * Pool-owned device memory, valid until ss_pool_destroy.  The table is
 * current once the update queued by the last ss_plan_step has run (for
 * instance after ss_sync). */
ss_status ss_block_table(ss_pool* pool, const int32_t** d_units, const uint64_t** d_agent_off);

/* Copy agent's block-table row to host (synchronous).  *n = agent's units;
 * SS_ERR_ARG if cap < *n or agent >= N. */
ss_status ss_block_table_host(ss_pool* pool, uint32_t agent, int32_t* out, uint32_t cap,
                              uint32_t* n);

/* Copy the whole block table (sum of agent_units entries, agent after agent,
 * -1 = not resident) to host (synchronous).  *n = entries; SS_ERR_ARG if
 * cap < *n. */
ss_status ss_block_table_host_all(ss_pool* pool, int32_t* out, uint64_t cap, uint64_t* n);

/* Resident flags [N] (0/1) to host (synchronous). */
ss_status ss_resident_host(ss_pool* pool, uint8_t* out);

/* Timing counters (SS_FLAG_TIMING); waits for the pool's queued work. */
ss_status ss_get_stats(ss_pool* pool, ss_stats* out);
ss_status ss_reset_stats(ss_pool* pool);

/* Measurement probes (not part of a step).  ss_probe_copy runs the library's
 * copy loop as a plain device-to-device copy of `bytes` (multiple of 16) and
 * returns its event time; ss_probe_link times `iters` hipMemcpyAsync copies of
 * `bytes` between pinned host memory and device memory: dir 0 = host to
 * device, 1 = device to host, 2 = both at once on two streams: host[0, bytes)
 * to dev[0, bytes) and dev[bytes, 2 bytes) to host[bytes, 2 bytes), so both
 * buffers must hold 2 * bytes; the time is for the pair. */
ss_status ss_probe_copy(void* dst, const void* src, uint64_t bytes, int iters, float* ms_per_iter);
/* Host round trip of one empty kernel launch on the current device: launch,
 * event record, wait for the event; *us_median = the median over `iters`
 * (>= 1) round trips, in microseconds.  A one-launch plan cannot return
 * faster than this (the plan's lists come back through mapped host memory,
 * without a copy). */
ss_status ss_probe_launch(int iters, float* us_median);
ss_status ss_probe_link(void* host, void* dev, uint64_t bytes, int dir, int iters,
                        float* ms_per_iter);

/* ---- Distance estimation (inputs of ss_plan_step) ------------------------
 *
 * Shared memory objects (Appendix A, "Fine-grained distance assignment"): an
 * object referenced by several agents, such as a node of a shared prefix
 * tree, gets the smallest distance of the agents that reference it, and is
 * needed now when any of them is active.  Planning a pool whose "agents" are
 * objects then uses obj_distances / obj_active as its distances and mask.
 *
 *   obj_off      [n_objects + 1] nondecreasing, obj_off[0] = 0,
 *                obj_off[n_objects] = n_refs: object o is referenced by
 *                obj_agents[obj_off[o] .. obj_off[o+1]).
 *   obj_agents   [n_refs] agent ids; ids >= n_agents are ignored.
 *   distances    [n_agents] agent distances, active [n_agents] 0/1.
 *   obj_distances [n_objects] out: min over the referencing agents of
 *                (0 if active else distance); 0xFFFFFFFF when no agent
 *                references the object.
 *   obj_active   [n_objects] out: 1 if any referencing agent is active.
 *   workspace    device memory of at least
 *                ss_object_distances_workspace(n_objects, n_refs, n_agents)
 *                bytes, 16-byte aligned, owned by the caller; its contents
 *                need no initialisation.
 * Every array is device memory of the current device, owned by the caller.
 * The work is queued on `stream` (a hipStream_t, NULL = the null stream) and
 * the call returns without waiting.  n_objects and n_refs must be below 2^31.
 * Offsets that break the rules above give unspecified output values but no
 * access outside the arrays.  SS_ERR_ARG for NULL, too small or non-device
 * arguments (nothing queued), SS_ERR_HIP if a launch fails. */
uint64_t ss_object_distances_workspace(uint32_t n_objects, uint32_t n_refs, uint32_t n_agents);
ss_status ss_object_distances(const uint32_t* obj_off, const uint32_t* obj_agents,
                              uint32_t n_objects, uint32_t n_refs, const uint32_t* distances,
                              const uint8_t* active, uint32_t n_agents, uint32_t* obj_distances,
                              uint8_t* obj_active, void* workspace, uint64_t workspace_bytes,
                              void* stream);

/* Measurement probe (not part of a step): runs ss_object_distances `iters`
 * times back to back on a private stream after one warm-up run and returns the
 * event time per run.  Same arguments and errors as ss_object_distances;
 * n_objects must be >= 1.  Synchronous. */
ss_status ss_probe_object_distances(const uint32_t* obj_off, const uint32_t* obj_agents,
                                    uint32_t n_objects, uint32_t n_refs,
                                    const uint32_t* distances, const uint8_t* active,
                                    uint32_t n_agents, uint32_t* obj_distances,
                                    uint8_t* obj_active, void* workspace,
                                    uint64_t workspace_bytes, int iters, float* ms_per_iter);

/* Hop counts (Section 3.2, "predefined activation paths": an agent's
 * distance is its hop count from the origin of the propagation).  A
 * breadth-first search along the directed edges of a CSR graph from the
 * sources (the agents holding the information now, hop 0):
 *   row_off  [n_vertices + 1] nondecreasing, row_off[n_vertices] = n_edges;
 *   col      [n_edges]: col[row_off[u] .. row_off[u+1]) are u's out-neighbours;
 *   sources  [n_sources] vertex ids (ids >= n_vertices are skipped,
 *            repeated ids count once);
 *   hops     [n_vertices] out: edges on a shortest path from the nearest
 *            source, or 0xFFFFFFFF if no source reaches the vertex within
 *            max_hops edges (0xFFFFFFFF = no horizon);
 *   workspace  ss_hop_distances_workspace(n_vertices) bytes of device memory,
 *            8-byte aligned, owned by the caller, no initialisation needed.
 * Every array is device memory of the current device, owned by the caller.
 * The search is queued on `stream` (two ordinary launches, then one
 * cooperative launch for the levels); the call returns without waiting.  The 32-bit word at workspace offset 20 is 1 after
 * the search if a grid barrier wait ever exceeded its bound (the hop counts
 * are then incomplete); it stays 0 otherwise.  n_vertices and n_edges must be
 * below 2^31; offsets that break the rules above give unspecified hop counts
 * but no access outside the arrays.  SS_ERR_ARG for NULL, too small or
 * non-device arguments, SS_ERR_HIP if the device has no cooperative launch or
 * a launch fails. */
uint64_t ss_hop_distances_workspace(uint32_t n_vertices);
ss_status ss_hop_distances(const uint32_t* row_off, const uint32_t* col, uint32_t n_vertices,
                           uint32_t n_edges, const uint32_t* sources, uint32_t n_sources,
                           uint32_t max_hops, uint32_t* hops, void* workspace,
                           uint64_t workspace_bytes, void* stream);

/* Interaction distances (Section 3.2, interaction-involved simulations:
 * D = min(D_action, D_interaction), D_interaction = physical distance /
 * velocity).  Per agent i:
 *   out[i] = min(d_action[i], floor(max(0, isqrt(d2_i) - radius) / velocity))
 * with d2_i the squared Euclidean distance to the nearest other agent, or
 * out[i] = d_action[i] when there is no other agent.
 *   pos_xy   [n_agents][2] int32 tile coordinates (x, y), each in [0, 32768);
 *            other values give unspecified results but no fault;
 *   d_action [n_agents] remaining steps of each agent's current action;
 *   velocity closing speed in tiles per step (>= 1); radius in tiles;
 *   out      [n_agents] out (may alias d_action);
 *   workspace  ss_interaction_distances_workspace(n_agents) bytes of device
 *            memory, owned by the caller, no initialisation needed.
 * Device memory of the current device, owned by the caller; queued on
 * `stream`, returns without waiting.  SS_ERR_ARG for NULL, too small or
 * non-device arguments or velocity 0, SS_ERR_HIP if a launch fails. */
uint64_t ss_interaction_distances_workspace(uint32_t n_agents);
ss_status ss_interaction_distances(const int32_t* pos_xy, const uint32_t* d_action,
                                   uint32_t n_agents, uint32_t velocity, uint32_t radius,
                                   uint32_t* out, void* workspace, uint64_t workspace_bytes,
                                   void* stream);

/* The same computation for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the partial minima live in a static device array of the
 * library instead of a workspace, so the call allocates nothing.  At most
 * 1,048,576 agents (SS_ERR_ARG beyond, nothing queued).  The array holds
 * 4 MiB on each device the library runs on until the process ends; its
 * device address is looked up on the first call on a device.  Every call on
 * one device shares that array and clears it on `stream` before use: calls
 * whose work overlaps on one device (other streams, other threads) race and
 * give unspecified results.  Other arguments, errors and results as
 * ss_interaction_distances. */
ss_status ss_interaction_distances_static(const int32_t* pos_xy, const uint32_t* d_action,
                                          uint32_t n_agents, uint32_t velocity, uint32_t radius,
                                          uint32_t* out, void* stream);

/* ---- Load-task scheduler (Appendix A, "Load task scheduler" and
 * "Preemption support") ------------------------------------------------------
 *
 * One centralized scheduler for every CPU-to-GPU load of its memory modules
 * (each described by an ss_pool_desc, the same data model as a pool: planes,
 * agent sizes, pinned host copies, a staging buffer cut into ring_slots
 * slots; the loader uses all of the staging buffer for loads).  Tasks are
 * ordered by (distance, agent, module), smallest first.  A task loads one
 * agent's memory of one module into the destination units it names and runs
 * as chunks of whole units (as many as fit in one staging slot): a copy of
 * the chunk from the agent's host copy into a slot, then a scatter into the
 * destination units on the device.  Before every chunk the scheduler checks
 * the preemption signal: if a queued task's distance is strictly smaller than
 * the running task's, the running task returns to the queue with its
 * progress (it later resumes at its next chunk) and the urgent task runs.
 * At most min(ring_slots) chunks are in flight, and each decision is taken
 * after the chunk that many places earlier has finished, so an urgent task
 * waits for at most that many chunks. */
typedef struct ss_loader ss_loader;

#define SS_LOADER_NO_PREEMPT 2u     /* tasks start in key order but always finish   */

#define SS_LOAD_START        1u     /* log flag: the task starts or resumes         */
#define SS_LOAD_PREEMPT      2u     /* log flag: it interrupted the running task    */
#define SS_LOAD_DONE         4u     /* log flag: the task's last chunk              */

typedef struct {
    uint32_t       module;          /* index into the loader's modules               */
    uint32_t       agent;           /* agent id within the module                    */
    uint32_t       distance;        /* invocation distance (0 = needed now)          */
    uint32_t       pad;
    const int32_t* units;           /* device: destination unit of each of the agent's
                                       agent_units[agent] logical units (caller-owned,
                                       valid until the task's last chunk has run);
                                       unit ids outside [0, capacity) are skipped  */
} ss_load_task;

typedef struct {
    uint32_t module, agent;
    uint32_t first;                 /* first logical unit of the chunk               */
    uint32_t count;                 /* units in the chunk                            */
    uint32_t flags;                 /* SS_LOAD_*                                     */
    uint32_t pad;
} ss_load_log;

typedef struct {
    uint64_t submitted, completed;  /* tasks                                         */
    uint64_t chunks, bytes;         /* chunks issued and their bytes                 */
    uint64_t preemptions;
} ss_loader_stats;

/* Create a scheduler over n_modules modules, all on one device (flags:
 * SS_LOADER_NO_PREEMPT or 0).  Every staging slot must hold at least one
 * unit.  SS_ERR_ARG for an invalid descriptor (message in ss_last_error). */
ss_status ss_loader_create(const ss_pool_desc* modules, uint32_t n_modules, uint32_t flags,
                           ss_loader** out);
/* Waits for issued chunks, then frees the scheduler (NULL is ignored). */
void ss_loader_destroy(ss_loader* loader);
/* DispatchLoadTasks: queue tasks.  A task whose (module, agent) is already
 * queued or running only takes the new distance (its units are kept); one
 * submitted after the agent's previous task completed is a new task.  All
 * tasks are checked before any is queued (SS_ERR_ARG: module or agent out of
 * range, units not device memory of the right size).  Thread-safe with
 * ss_loader_pump. */
ss_status ss_loader_submit(ss_loader* loader, const ss_load_task* tasks, uint32_t n);
/* Issue up to max_chunks chunks in priority order, checking the preemption
 * signal before each; blocks while the in-flight window is full.  Writes one
 * entry per issued chunk to log (up to log_cap; log may be NULL when log_cap
 * is 0) and the number issued to *n_issued.  Returns when max_chunks are
 * issued or no task is left.  One thread at a time. */
ss_status ss_loader_pump(ss_loader* loader, uint32_t max_chunks, ss_load_log* log,
                         uint32_t log_cap, uint32_t* n_issued);
/* Tasks waiting in the queue and whether one is running. */
ss_status ss_loader_pending(ss_loader* loader, uint32_t* queued, uint32_t* running);
/* Block until every issued chunk has landed in its destination units. */
ss_status ss_loader_sync(ss_loader* loader);
ss_status ss_loader_get_stats(ss_loader* loader, ss_loader_stats* out);

/* Wait until all work the pool has queued (plan, copies, kernels) is done
 * (blocking, or polling under SS_FLAG_POLL_WAIT). */
ss_status ss_sync(ss_pool* pool);

/* Plumbing for callers without a framework allocator: thin wrappers over the
 * HIP runtime this library is linked with.  Memory must be allocated by the
 * same runtime instance that runs the pool; a process that has loaded another
 * copy of the HIP runtime (for example one bundled with a Python framework)
 * must allocate through that one and must not mix the two.
 *   ss_device_count   number of visible devices (0 when none; not an error)
 *   ss_device_alloc   hipMalloc of `bytes` on `device`
 *   ss_host_alloc     pinned host memory (hipHostMalloc), device-accessible
 *   ss_device_free / ss_host_free   release them (NULL is ignored)
 *   ss_copy           synchronous copy of `bytes` between any two of them */
ss_status ss_device_count(int32_t* n);
ss_status ss_device_alloc(int32_t device, uint64_t bytes, void** out);
ss_status ss_host_alloc(uint64_t bytes, void** out);
ss_status ss_device_free(void* ptr);
ss_status ss_host_free(void* ptr);
ss_status ss_copy(void* dst, const void* src, uint64_t bytes);

/* Streams and events of the same runtime, for callers that time or order
 * the calls above without a framework:
 *   ss_stream_create   non-blocking stream at the default priority on the
 *                      current device; ss_stream_destroy / ss_stream_sync
 *                      (ss_stream_sync(NULL) waits for the null stream)
 *   ss_event_create    timing event; ss_event_record on a stream;
 *   ss_event_elapsed   waits for `end`, then milliseconds from start to end */
ss_status ss_stream_create(void** stream);
ss_status ss_stream_destroy(void* stream);
ss_status ss_stream_sync(void* stream);
ss_status ss_event_create(void** event);
ss_status ss_event_destroy(void* event);
ss_status ss_event_record(void* event, void* stream);
ss_status ss_event_elapsed(void* start, void* end, float* ms);

/* Message of the last failed call on this thread ("" if none). */
const char* ss_last_error(void);

/* Failure injection, for callers that test their handling of SS_ERR_HIP and
 * SS_ERR_POISONED (a failing HIP call cannot otherwise be provoked without
 * harming the device).  Counting from this call, the n-th copy command issued
 * by ss_evict_pack, ss_prefetch_unpack or ss_loader_pump, in any pool or
 * loader of the process, is not issued and fails as a HIP error would: that
 * call returns SS_ERR_HIP and its pool or loader is poisoned.  n = 0 disarms;
 * the hook disarms itself once it has fired.  Work queued before the failing
 * copy still runs, so ss_pool_destroy and ss_loader_destroy stay clean. */
void ss_debug_fail_copy(uint32_t n);

#ifdef __cplusplus
}
#endif
#endif /* SCALESIM_H */
