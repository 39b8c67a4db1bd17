"""The prefetch loop against an independent closed form.

Candidates are taken in increasing key; candidate i (cumulative prefetched
units S_i, distance d_i) is accepted iff every earlier one was and
    S_i <= budget  and  S_i <= free' + G(d_i),
where free' is the free space left after demand loads and demand victims and
G(x) is the number of units held by the remaining inactive residents whose
distance is strictly larger than x (Section 3.3: room comes from free space
or from inactive agents with larger distance).  Because S_i grows and G(d_i)
shrinks along the candidate order, the accepted candidates are exactly the
leading run of indices that satisfy it.  The victims are then the demand
victims plus the shortest further prefix of the eviction order that covers
S - free'."""
import numpy as np

from oracle import OraclePool

S = 0xFFFFFFFF


def closed_form(pool, D, active, theta, budget):
    s = pool.s
    act = active.astype(bool)
    res = pool.resident.copy()
    d = np.where(act, 0, D.astype(np.int64))
    ids = np.arange(pool.N)
    L = ids[act & ~res]
    free = pool.U - s[res].sum()
    need = s[L].sum() - free
    E = ids[res & ~act]
    E = E[np.lexsort((E, d[E]))][::-1]                 # key descending
    cs = np.concatenate([[0], np.cumsum(s[E])])
    n_d = 0 if need <= 0 else int(np.searchsorted(cs, need, side="left"))
    free1 = free + cs[n_d] - s[L].sum()
    C = ids[~res & ~act & (D.astype(np.int64) < theta)]
    C = C[np.lexsort((C, d[C]))]                        # key ascending
    Si = np.cumsum(s[C])
    rest = E[n_d:]
    G = np.array([s[rest][d[rest] > d[c]].sum() for c in C], dtype=np.int64)
    lim = free1 + G
    ok = Si <= lim
    if budget is not None:
        ok &= Si <= budget
    n_p = int(np.argmin(ok)) if not ok.all() else len(C)
    if n_p == 0 or Si[n_p - 1] <= free1:
        n_v = n_d
    else:
        cr = np.cumsum(s[rest])
        n_v = n_d + int(np.searchsorted(cr, Si[n_p - 1] - free1, side="left")) + 1
    return list(E[:n_v]), list(L) + list(C[:n_p])


def test_prefetch_loop_matches_closed_form():
    rng = np.random.default_rng(7)
    checked = 0
    for it in range(300):
        N = int(rng.integers(4, 40))
        s = rng.integers(1, 6, size=N)
        U = int(rng.integers(s.max(), s.sum() + 1))
        pool = OraclePool(U, s)
        theta = int(rng.choice([0, 1, 3, 6, 10, S]))
        budget = None if rng.random() < 0.5 else int(rng.integers(0, U + 1))
        for t in range(6):
            active = np.zeros(N, np.uint8)
            order = rng.permutation(N)
            tot = 0
            for a in order[: int(rng.integers(0, N // 2 + 1))]:
                if tot + s[a] <= U:
                    active[a] = 1
                    tot += s[a]
            D = rng.integers(1, 12, size=N).astype(np.uint32)
            D[rng.random(N) < 0.1] = S
            exp_v, exp_l = closed_form(pool, D, active, theta, budget)
            plan = pool.plan_step(D, active, theta, budget)
            assert plan.victims.tolist() == [int(x) for x in exp_v], (it, t)
            assert plan.loads.tolist() == [int(x) for x in exp_l], (it, t)
            checked += 1
    assert checked == 1800
