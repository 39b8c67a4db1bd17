"""Seeded synthetic agent traces and agent-memory contents.

This module only *generates inputs*: which agents are activated at each
simulation step, each agent's invocation-distance estimate, each agent's
memory footprint per memory module, and the byte contents of that memory.  It
holds none of the memory manager's arithmetic (no keys, no eviction or
prefetch decisions, no allocation), so the CPU oracle and the HIP path can
both consume it without sharing any of the method.

The workloads stand in for the paper's three application classes (Section 4.1,
"Benchmarks": independent simulation, interaction-involved simulation and
information diffusion over a social graph).  None of those simulators or their
data are used: every trace is drawn from a seeded ``numpy`` PCG64 generator
with the shapes listed in ``CONFIGS``.

Distances follow the invocation-distance abstraction (Section 3.2): a
*relative* estimate of how soon an agent will next call the LLM.  Here the
exact value is the number of steps until the agent's next activation, or
``SENTINEL`` when it is never activated again inside the trace; the noisy
variant adds rounded Gaussian noise (the estimate need only preserve relative
urgency, Section 3.2, "Independent simulation").
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

SENTINEL = 0xFFFFFFFF          # "no future activation inside the trace"
KIB = 1024
MIB = 1024 * 1024


@dataclass
class PoolSpec:
    """One memory module's device pool (Appendix A: one registered module).

    A pool has ``capacity_units`` physical units; every unit is made of
    ``len(chunk_bytes)`` planes, plane ``c`` holding a ``chunk_bytes[c]``-byte
    chunk of the unit.  Agent ``a`` owns ``agent_units[a]`` units.
    """
    name: str
    capacity_units: int
    chunk_bytes: list
    agent_units: np.ndarray          # uint32 [N], every entry >= 1

    @property
    def unit_bytes(self) -> int:
        return int(sum(self.chunk_bytes))

    @property
    def n_planes(self) -> int:
        return len(self.chunk_bytes)


@dataclass
class Trace:
    name: str
    n_agents: int
    n_steps: int
    pools: list                      # [PoolSpec]
    active: np.ndarray               # uint8 [T, N]   1 = agent issues an LLM call at step t
    dist: np.ndarray                 # uint32 [T, N]  distance estimate handed to the manager
    dist_true: np.ndarray            # uint32 [T, N]  exact steps to next activation (or SENTINEL)
    meta: dict = field(default_factory=dict)


# --------------------------------------------------------------------------
# distances from an activation schedule
# --------------------------------------------------------------------------

def exact_distances(active: np.ndarray) -> np.ndarray:
    """Steps from t to the first activation strictly after t, else SENTINEL."""
    T, N = active.shape
    out = np.empty((T, N), dtype=np.uint32)
    nxt = np.full(N, -1, dtype=np.int64)           # first activation index > t
    for t in range(T - 1, -1, -1):
        out[t] = np.where(nxt >= 0, nxt - t, SENTINEL).astype(np.uint32)
        nxt = np.where(active[t] != 0, t, nxt)
    return out


def noisy_distances(dist_true: np.ndarray, sd: float, rng: np.random.Generator) -> np.ndarray:
    """Rounded Gaussian noise on finite distances, clamped to >= 1."""
    noise = rng.normal(0.0, sd, size=dist_true.shape)
    finite = dist_true != SENTINEL
    est = np.maximum(1.0, np.rint(dist_true.astype(np.float64) + noise))
    est = np.minimum(est, float(SENTINEL - 1))
    return np.where(finite, est.astype(np.uint32), np.uint32(SENTINEL)).astype(np.uint32)


def _pages(tokens: np.ndarray, page_tokens: int = 16) -> np.ndarray:
    return ((tokens + page_tokens - 1) // page_tokens).astype(np.uint32)


def _lognormal_tokens(rng, n, mean, sigma, cap):
    mu = math.log(mean) - sigma * sigma / 2.0         # arithmetic mean == `mean`
    x = rng.lognormal(mu, sigma, size=n)
    return np.clip(np.rint(x), 1, cap).astype(np.int64)


def lora_chunk_bytes(layers, hidden, inter, kv_out, rank, dtype_bytes=2):
    """Per-plane byte sizes of a LoRA adapter: for each layer and each of
    q, k, v, o, gate, up, down, the A (rank x in) then the B (out x rank)
    matrix."""
    mods = [(hidden, hidden), (hidden, kv_out), (hidden, kv_out), (hidden, hidden),
            (hidden, inter), (hidden, inter), (inter, hidden)]
    out = []
    for _ in range(layers):
        for fin, fout in mods:
            out.append(rank * fin * dtype_bytes)
            out.append(fout * rank * dtype_bytes)
    return out


# --------------------------------------------------------------------------
# the five workloads
# --------------------------------------------------------------------------

def _tiny(seed: int) -> Trace:
    """64 agents, 2-layer x 2-KV-head x 64 fp16 KV (1 KiB/token), 256-token
    prefix = 16 pages of 16 KiB (4 planes of 4 KiB: layer x {K,V});
    pool of 256 units (16 agents); 6 of 64 agents uniformly per step; exact
    distances; 100 steps."""
    rng = np.random.default_rng(seed)
    N, T = 64, 100
    active = np.zeros((T, N), dtype=np.uint8)
    for t in range(T):
        active[t, rng.choice(N, 6, replace=False)] = 1
    units = np.full(N, 16, dtype=np.uint32)
    pool = PoolSpec("kv", 256, [4 * KIB] * 4, units)
    dt = exact_distances(active)
    return Trace("tiny", N, T, [pool], active, dt.copy(), dt, {"seed": seed})


def _roundrobin(seed: int) -> Trace:
    """1,000 agents, 32-layer x 8-KV-head x 128 bf16 KV (128 KiB/token),
    16-token pages = 2 MiB units of 64 planes x 32 KiB; prefix tokens
    uniform in [512, 2048]; 40 GB pool; round-robin activation with period
    20 and Poisson(2) jitter (~5% per step); exact distances; 200 steps."""
    rng = np.random.default_rng(seed)
    N, T, period = 1000, 200, 20
    tokens = rng.integers(512, 2049, size=N)
    units = _pages(tokens)
    active = np.zeros((T, N), dtype=np.uint8)
    nxt = np.arange(N) % period
    while True:
        live = nxt < T
        if not live.any():
            break
        active[nxt[live], np.flatnonzero(live)] = 1
        step = period + rng.poisson(2.0, size=N) - 2
        nxt = np.where(live, nxt + np.maximum(step, 1), nxt)
    cap = (40 * 10**9) // (2 * MIB)
    pool = PoolSpec("kv", cap, [32 * KIB] * 64, units)
    dt = exact_distances(active)
    return Trace("roundrobin", N, T, [pool], active, dt.copy(), dt, {"seed": seed})


def _bursty(seed: int) -> Trace:
    """10,000 agents, same KV unit as the round-robin workload; prefix tokens
    lognormal (mean 256, sigma 0.8, cap 4096); 120 GB pool; 100 clusters of
    100 agents; a wave centre random-walks over clusters (jumping uniformly
    with probability 0.05) and 100-300 agents of the centre and its two
    neighbour clusters fire per step; noisy distances (sd 2); 300 steps."""
    rng = np.random.default_rng(seed)
    N, T = 10_000, 300
    units = _pages(_lognormal_tokens(rng, N, 256, 0.8, 4096))
    perm = rng.permutation(N)
    clusters = perm.reshape(100, 100)
    centre = int(rng.integers(100))
    active = np.zeros((T, N), dtype=np.uint8)
    for t in range(T):
        if rng.random() < 0.05:
            centre = int(rng.integers(100))
        else:
            centre = (centre + (1 if rng.random() < 0.5 else -1)) % 100
        pool_agents = np.concatenate([clusters[(centre + k) % 100] for k in (-1, 0, 1)])
        k_t = int(rng.integers(100, 301))
        active[t, rng.choice(pool_agents, k_t, replace=False)] = 1
    cap = (120 * 10**9) // (2 * MIB)
    pool = PoolSpec("kv", cap, [32 * KIB] * 64, units)
    dt = exact_distances(active)
    nrng = np.random.default_rng([seed, 1])
    return Trace("bursty", N, T, [pool], active, noisy_distances(dt, 2.0, nrng), dt,
                 {"seed": seed})


def _zipf_lora(seed: int) -> Trace:
    """2,000 agents, each with a rank-16 bf16 LoRA adapter on q/k/v/o/gate/
    up/down of a 32-layer, hidden-4096, intermediate-14336 model (80 MiB, 448
    planes of 32-448 KiB, 256 slots) and a 512-token prefix in the 2 MiB KV
    unit (32 units, 30 GB pool); 80 agents per step drawn without replacement
    with probability proportional to rank^-1.1; exact distances; 200 steps."""
    rng = np.random.default_rng(seed)
    N, T, k = 2000, 200, 80
    rank = np.empty(N, dtype=np.int64)
    rank[rng.permutation(N)] = np.arange(N)
    w = (rank + 1.0) ** -1.1
    w /= w.sum()
    active = np.zeros((T, N), dtype=np.uint8)
    for t in range(T):
        active[t, rng.choice(N, k, replace=False, p=w)] = 1
    kv = PoolSpec("kv", (30 * 10**9) // (2 * MIB), [32 * KIB] * 64,
                  np.full(N, 32, dtype=np.uint32))
    lora = PoolSpec("lora", 256, lora_chunk_bytes(32, 4096, 14336, 1024, 16),
                    np.ones(N, dtype=np.uint32))
    dt = exact_distances(active)
    return Trace("zipf_lora", N, T, [kv, lora], active, dt.copy(), dt, {"seed": seed})


def _diffusion(seed: int) -> Trace:
    """50,000 agents in one unified pool of 512 KiB units (160 GB); each agent
    holds ceil(tokens/16) KV pages (16-layer x 8-head x 64 bf16, 32 KiB/token,
    tokens lognormal mean 128, sigma 0.8, cap 4096) plus a LoRA adapter of
    rank 8, 16 or 64 on a hidden-2048 / intermediate-8192 model padded to
    whole units (22, 43 or 172 units); activations spread over a random
    out-degree-8 graph: an active agent messages each out-neighbour with
    probability 0.1 and receivers fire one step later, plus spontaneous
    firing with probability 0.002 and 1% of agents seeded at step 0; noisy
    distances (sd 2); 500 steps."""
    rng = np.random.default_rng(seed)
    N, T = 50_000, 500
    pages = _pages(_lognormal_tokens(rng, N, 128, 0.8, 4096))
    ranks = rng.choice(np.array([8, 16, 64]), size=N)
    per_rank = {r: sum(lora_chunk_bytes(16, 2048, 8192, 512, r)) for r in (8, 16, 64)}
    unit = 512 * KIB
    lora_units = np.array([(per_rank[int(r)] + unit - 1) // unit for r in ranks], dtype=np.uint32)
    units = (pages + lora_units).astype(np.uint32)
    out = rng.integers(0, N - 1, size=(N, 8))
    out += out >= np.arange(N)[:, None]             # no self loops
    active = np.zeros((T, N), dtype=np.uint8)
    cur = rng.random(N) < 0.01
    for t in range(T):
        active[t] = cur
        send = rng.random((N, 8)) < 0.1
        send &= cur[:, None]
        nxt = np.zeros(N, dtype=bool)
        nxt[out[send]] = True
        nxt |= rng.random(N) < 0.002
        cur = nxt
    pool = PoolSpec("unified", (160 * 10**9) // unit, [unit], units)
    dt = exact_distances(active)
    nrng = np.random.default_rng([seed, 1])
    return Trace("diffusion", N, T, [pool], active, noisy_distances(dt, 2.0, nrng), dt,
                 {"seed": seed, "lora_rank": ranks, "out_neighbors": out})


CONFIGS = {
    "tiny": _tiny,
    "roundrobin": _roundrobin,
    "bursty": _bursty,
    "zipf_lora": _zipf_lora,
    "diffusion": _diffusion,
}


def make_trace(name: str, seed: int = 0) -> Trace:
    tr = CONFIGS[name](seed)
    for p in tr.pools:
        act_units = (tr.active.astype(np.int64) * p.agent_units.astype(np.int64)[None, :]).sum(1)
        assert act_units.max() <= p.capacity_units, "trace overcommits a pool"
        assert all(c % 16 == 0 for c in p.chunk_bytes)
    return tr


def shrink_planes(trace: Trace, chunk_bytes_fn) -> Trace:
    """Same schedule and unit counts, smaller chunk sizes (for byte tests whose
    full-size host backing would not fit): ``chunk_bytes_fn(pool)`` returns
    the new per-plane byte list."""
    pools = [PoolSpec(p.name, p.capacity_units, list(chunk_bytes_fn(p)), p.agent_units)
             for p in trace.pools]
    return Trace(trace.name + "_small", trace.n_agents, trace.n_steps, pools,
                 trace.active, trace.dist, trace.dist_true, dict(trace.meta))


def subsample_agents(trace: Trace, n_agents: int) -> Trace:
    """The first ``n_agents`` agents of a workload with every pool's capacity
    scaled by the same fraction (kept at least as large as the most units the
    kept agents ever need at once)."""
    act = trace.active[:, :n_agents]
    pools = []
    for p in trace.pools:
        units = p.agent_units[:n_agents]
        need = int((act.astype(np.int64) * units.astype(np.int64)[None, :]).sum(1).max())
        cap = max(need, int(round(p.capacity_units * n_agents / trace.n_agents)), 1)
        pools.append(PoolSpec(p.name, cap, list(p.chunk_bytes), units))
    return Trace(trace.name + "_sub%d" % n_agents, n_agents, trace.n_steps, pools, act,
                 trace.dist[:, :n_agents], trace.dist_true[:, :n_agents], dict(trace.meta))


def prefix_tree_objects(n_agents: int, branching: int, depth: int, seed: int,
                        node_pages=(1, 8)):
    """Memory objects of a shared prefix tree: a root shared by every agent,
    internal nodes shared by the agents below them, and one private leaf per
    agent; agents are spread uniformly over the tree's paths.  Returns the
    CSR map object -> referencing agents (``obj_off`` [M+1], ``obj_agents``)
    and each object's size in pages."""
    rng = np.random.default_rng(seed)
    paths = rng.integers(0, branching, size=(n_agents, depth))
    offs, lists = [np.zeros(1, np.int64)], []
    code = np.zeros(n_agents, dtype=np.int64)       # path prefix as a base-`branching` number
    total = 0
    for lvl in range(depth + 1):                    # nodes by depth, then by path
        if lvl:
            code = code * branching + paths[:, lvl - 1]
        order = np.argsort(code, kind="stable")     # members of a node in agent order
        _, counts = np.unique(code[order], return_counts=True)
        lists.append(order.astype(np.uint32))
        offs.append(total + np.cumsum(counts))
        total += n_agents
    lists.append(np.arange(n_agents, dtype=np.uint32))                # private leaves
    offs.append(total + np.arange(1, n_agents + 1))
    obj_off = np.concatenate(offs).astype(np.uint64)
    obj_agents = np.concatenate(lists)
    n_obj = len(obj_off) - 1
    sizes = rng.integers(node_pages[0], node_pages[1] + 1, size=n_obj).astype(np.uint32)
    return obj_off, obj_agents, sizes


def prefix_forest(n_trees: int, n_agents: int, branching: int, depth: int, seed: int):
    """``n_trees`` independent simulations of ``n_agents`` agents, each with a
    shared prefix tree (``prefix_tree_objects``): the trees' objects one after
    another, agent ids of tree k offset by k * n_agents."""
    off, agents, sizes = prefix_tree_objects(n_agents, branching, depth, seed)
    R = np.uint64(off[-1])
    offs = [off[:1]] + [off[1:] + np.uint64(k) * R for k in range(n_trees)]
    ags = [agents + np.uint32(k * n_agents) for k in range(n_trees)]
    return (np.concatenate(offs).astype(np.uint64), np.concatenate(ags),
            np.tile(sizes, n_trees))


def random_tiny_trace(rng: np.random.Generator, n_agents: int, n_steps: int,
                      max_active: int, capacity_agents: int, units=None):
    """A small random request trace for brute-force checks."""
    active = np.zeros((n_steps, n_agents), dtype=np.uint8)
    for t in range(n_steps):
        k = int(rng.integers(0, max_active + 1))
        if k:
            active[t, rng.choice(n_agents, k, replace=False)] = 1
    if units is None:
        units = np.ones(n_agents, dtype=np.uint32)
    pool = PoolSpec("tiny", capacity_agents * int(units.max()), [16], np.asarray(units, np.uint32))
    dt = exact_distances(active)
    return Trace("random_tiny", n_agents, n_steps, [pool], active, dt.copy(), dt, {})


# --------------------------------------------------------------------------
# agent memory contents
# --------------------------------------------------------------------------

_M64 = (1 << 64) - 1


def splitmix64(x: np.ndarray) -> np.ndarray:
    """SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014) on uint64."""
    with np.errstate(over="ignore"):
        z = (x.astype(np.uint64) + np.uint64(0x9E3779B97F4A7C15))
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


class Content:
    """Deterministic bytes of every (agent, logical unit, plane) chunk.

    64-bit word ``w`` of chunk ``(a, j, c)`` is ``pattern_c[w] XOR
    splitmix64((a << 32) | (j << 12) | c)``: a wrong agent, unit, plane or
    offset all produce different bytes."""

    def __init__(self, pool: PoolSpec, seed: int = 0, pool_index: int = 0):
        rng = np.random.default_rng([seed, 7, pool_index])
        self.pool = pool
        self.patterns = [rng.integers(0, 1 << 63, size=cb // 8, dtype=np.uint64)
                         | (rng.integers(0, 2, size=cb // 8, dtype=np.uint64) << np.uint64(63))
                         for cb in pool.chunk_bytes]
        self.plane_off = np.concatenate([[0], np.cumsum(pool.chunk_bytes)]).astype(np.int64)

    def tag(self, a, j, c) -> np.ndarray:
        a = np.asarray(a, dtype=np.uint64)
        j = np.asarray(j, dtype=np.uint64)
        c = np.asarray(c, dtype=np.uint64)
        return splitmix64((a << np.uint64(32)) | (j << np.uint64(12)) | c)

    def chunk(self, a: int, j: int, c: int) -> np.ndarray:
        """uint8 bytes of one chunk."""
        return (self.patterns[c] ^ self.tag(a, j, c)).view(np.uint8)

    def agent_bytes(self, a: int, n_units: int | None = None) -> np.ndarray:
        """The agent's serialised memory: unit j = 0.. in order, each unit the
        concatenation of its planes' chunks."""
        s = int(self.pool.agent_units[a]) if n_units is None else n_units
        W = self.pool.unit_bytes // 8
        out = np.empty((s, W), dtype=np.uint64)
        j = np.arange(s, dtype=np.uint64)
        for c, pat in enumerate(self.patterns):
            lo, hi = self.plane_off[c] // 8, self.plane_off[c + 1] // 8
            out[:, lo:hi] = pat[None, :] ^ self.tag(a, j, c)[:, None]
        return out.reshape(-1).view(np.uint8)

    def units_bytes(self, a: np.ndarray, j: np.ndarray) -> np.ndarray:
        """Bytes of units (a[k], j[k]) for arrays of agents and logical units:
        uint8 [K, unit_bytes], planes concatenated in order."""
        a = np.asarray(a, dtype=np.uint64)
        j = np.asarray(j, dtype=np.uint64)
        W = self.pool.unit_bytes // 8
        out = np.empty((len(a), W), dtype=np.uint64)
        for c, pat in enumerate(self.patterns):
            lo, hi = self.plane_off[c] // 8, self.plane_off[c + 1] // 8
            out[:, lo:hi] = pat[None, :] ^ self.tag(a, j, c)[:, None]
        return out.view(np.uint8)

    def unit_chunk_words0(self, a: np.ndarray, j: np.ndarray, c: int) -> np.ndarray:
        """First 64-bit word of chunk (a, j, c) for arrays of (a, j): a cheap
        fingerprint for checks at full size."""
        return self.patterns[c][0] ^ self.tag(a, j, c)
