"""The descending threshold sweep run as two chains visits the same optimum (CPU).

The stage-DP kernel splits a class's descending sweep between two chains of
passes (each covering part of the threshold range, an idle chain taking the
lower half of the other's range).  This checks the argument on the oracle's
segment-cost tensors with a small model of the sweep: a pass at threshold t is
the least stage sum with every stage <= t and the largest stage of its
partition (ties: smallest split point), and an incumbent per B is replaced by a
lower objective, or an equal one with a lower largest stage.  For every
(candidate, group of B values) both forms must end with the same incumbents,
and the two chains must not need more rounds of passes than one chain."""
import numpy as np

from oracle import oracle as orc
from paper_2609_39350_amd import workloads

BIG = np.iinfo(np.int64).max // 4


def make_pass(cost, n):
    """Threshold pass over cost[s][a][b] (entries >= BIG: no segment)."""
    pp = cost.shape[0]
    c = np.minimum(cost, BIG)

    def run(t):
        f = np.full(n + 1, BIG, dtype=np.int64)
        f[0] = 0
        args = []
        for s in range(pp):
            m = np.where(c[s] <= t, c[s], BIG)
            tot = np.minimum(f[:, None] + m, BIG)
            a = np.argmin(tot, axis=0)   # first minimum: the smallest split point
            f = tot[a, np.arange(n + 1)]
            args.append(a)
        if f[n] >= BIG:
            return None
        b, mx = n, 0
        for s in range(pp - 1, -1, -1):
            a = args[s][b]
            mx = max(mx, int(c[s][a][b]))
            b = a
        return int(f[n]), mx
    return run


def sweep(run, bms, chains):
    """Incumbents (objective, largest stage) per B - 1 in bms and the number of
    rounds of passes; chains = 1 or 2."""
    first = run(BIG - 1)
    if first is None:
        return None, 1
    f1, m1 = first
    tbot, t = m1, m1 - 1   # the min-max value: the lowest largest stage reachable
    while (r := run(t)) is not None:
        tbot, t = r[1], r[1] - 1
    inc = [(f1 + bm * m1, m1) for bm in bms]

    def take(f, m):
        for i, bm in enumerate(bms):
            sc = f + bm * m
            if sc < inc[i][0] or (sc == inc[i][0] and m < inc[i][1]):
                inc[i] = (sc, m)

    def need(ch):   # the largest threshold a B still needs from the chain, or -1
        best = -1
        for (sc, m), bm in zip(inc, bms):
            if (m == tbot and sc == f1 + bm * tbot) or ch["F"] + bm * tbot > sc:
                continue
            lim = (sc - ch["F"]) // bm if bm > 0 else BIG
            best = max(best, min(lim, ch["t"]))
        return best if best > max(ch["stop"], tbot) else -1

    rounds = 1
    chs = [dict(F=f1, t=m1 - 1 if chains == 1 else -1, stop=tbot)]
    if chains == 2:
        chs.append(dict(F=f1, t=m1 - 1, stop=tbot))
    pending_bot = tbot < m1
    while True:
        ts = [need(ch) for ch in chs]
        jobs = []
        if pending_bot:   # the pass at t_bot, beside the top chain's first pass
            jobs.append((None, tbot))
            pending_bot = False
            if chains == 1:
                rounds += 1
                take(*run(tbot))
                continue
        elif chains == 2 and (ts[0] >= 0) != (ts[1] >= 0):
            x = 0 if ts[0] >= 0 else 1
            y = 1 - x
            lower = max(chs[x]["stop"], tbot)
            if ts[x] - lower >= 2:
                mid = lower + (ts[x] - lower) // 2
                chs[y] = dict(F=chs[x]["F"], t=mid, stop=chs[x]["stop"])
                chs[x]["stop"] = mid
                ts[y] = mid
        jobs += [(i, t) for i, t in enumerate(ts) if t >= 0]
        if not jobs:
            break
        rounds += 1
        for i, t in jobs:
            r = run(t)
            take(*r)
            if i is not None:
                chs[i]["F"], chs[i]["t"] = r[0], r[1] - 1
    return inc, rounds


def _check(problem, candidates):
    o = orc.Oracle(problem)
    micro = [int(b) for b in problem["space"]["micro"]]
    nm = len(micro)
    one = two = n = 0
    for idx in candidates:
        key = idx // nm
        pp = o.configs()[key // o.n_orders()][0]
        groups = {}
        for j, b in enumerate(micro):
            groups.setdefault(min(b, pp), []).append(j)
        for js in groups.values():
            cost, _ = o.segment_costs(key * nm + js[0])
            run = make_pass(cost, problem["model"]["n_layers"])
            bms = [micro[j] - 1 for j in js]
            r1, k1 = sweep(run, bms, 1)
            r2, k2 = sweep(run, bms, 2)
            assert r1 == r2, (idx, r1, r2)
            one, two, n = one + k1, two + k2, n + 1
    return one, two, n


def test_two_chains_reach_the_same_incumbents():
    one = two = n = 0
    probs = [workloads.random_tiny(s) for s in range(12)] + [workloads.config(1)]
    for p in probs:
        nc = orc.Oracle(p).n_instances()
        a, b, k = _check(p, range(0, nc, max(1, nc // 40)))
        one, two, n = one + a, two + b, n + k
    assert n > 100
    assert two <= one


def test_two_chains_save_rounds_on_deep_pipelines():
    p = workloads.config(2)
    o = orc.Oracle(p)
    nm = len(p["space"]["micro"])
    deep = [k * nm for k in range(o.n_instances() // nm)
            if o.configs()[k // o.n_orders()][0] == max(c[0] for c in o.configs())]
    one, two, n = _check(p, deep[:: max(1, len(deep) // 12)])
    assert n >= 10 and two < one
