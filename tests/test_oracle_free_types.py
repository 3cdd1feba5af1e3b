"""Free per-stage device types (the DP state m of Section 3.4 lets every stage
take its own device type): pins of the oracle's sequence enumeration and
of the stage layout it builds from a sequence.

In this mode a pipeline of PP stages with group size g = G / PP is a sequence
of pure stages, k_h = m_h / g of type h, and the candidate's "order" index
walks the distinct sequences in lexicographic order."""
import itertools
import math

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2609_39350_amd import workloads
from tests.problems import variant


def free(p):
    return variant(p, **{"space.stage_types": 1})


def multinomial(ks):
    n = math.factorial(sum(ks))
    for k in ks:
        n //= math.factorial(k)
    return n


def test_sequences_are_the_sorted_distinct_arrangements():
    # brute force: every distinct permutation of the stage-type multiset, sorted
    p = free(workloads.config(2))
    o = orc.Oracle(p)
    counts = [int(x) for x in p["cluster"]["count"]]
    G = sum(counts)
    pps = sorted({c[0] for c in o.configs()})
    assert pps, "no configuration left"
    most = 1
    for pp in pps:
        g = G // pp
        ks = [m // g for m in counts]
        multiset = [h for h, k in enumerate(ks) for _ in range(k)]
        want = sorted(set(itertools.permutations(multiset)))
        got = []
        while True:
            s = o.sequence(pp, len(got))
            if s is None:
                break
            got.append(tuple(s))
        assert got == want, pp
        assert len(got) == multinomial(ks)
        most = max(most, len(got))
    assert o.n_orders() == most


def test_configurations_need_whole_groups_of_one_type():
    for seed, p in ((0, workloads.config(1)), (1, workloads.config(2)),
                    (2, workloads.random_tiny(77, n_types=3))):
        ob, of = orc.Oracle(p), orc.Oracle(free(p))
        counts = [int(x) for x in p["cluster"]["count"]]
        G = sum(counts)
        want = [c for c in ob.configs() if all(m % (G // c[0]) == 0 for m in counts)]
        assert of.configs() == want, seed


def _block_sequence(o, perm, pp):
    counts = [int(x) for x in o.problem["cluster"]["count"]]
    g = sum(counts) // pp
    return [h for h in perm for _ in range(counts[h] // g)]


def _find_sequence(o, pp, seq):
    i = 0
    while True:
        s = o.sequence(pp, i)
        assert s is not None, (pp, seq)
        if s == seq:
            return i
        i += 1


def test_pure_block_ordering_equals_its_sequence():
    # where every type fills whole groups, a block ordering lays out pure stages;
    # the free mode's candidate with that very sequence must be the same candidate
    # (same stages, windows, constants and DP result)
    p = workloads.config(2)
    ob, of = orc.Oracle(p), orc.Oracle(free(p))
    nB = len(p["space"]["micro"])
    cfg_b, cfg_f = ob.configs(), of.configs()
    per_b, per_f = ob.n_orders() * nB, of.n_orders() * nB
    checked = 0
    for ci, cfg in enumerate(cfg_f):
        if ci % 7:
            continue
        bi = cfg_b.index(cfg)
        for ob_o in range(ob.n_orders()):
            seq = _block_sequence(ob, ob.order(ob_o), cfg[0])
            fo = _find_sequence(of, cfg[0], seq)
            assert of.dp_const(cfg, fo) == ob.dp_const(cfg, ob_o)
            for j, B in enumerate(p["space"]["micro"]):
                assert of.stages(cfg, fo, B) == ob.stages(cfg, ob_o, B)
                rb = ob.solve(bi * per_b + ob_o * nB + j)
                rf = of.solve(ci * per_f + fo * nB + j)
                assert rf == rb, (cfg, ob_o, fo, B)
                checked += 1
    assert checked > 100


def test_single_type_is_block_mode():
    # one device type: one sequence, every stage pure; both modes agree everywhere
    for s in range(4):
        p = workloads.random_tiny(300 + s, n_types=1)
        ob, of = orc.Oracle(p), orc.Oracle(free(p))
        assert of.n_orders() == 1 and ob.configs() == of.configs()
        n = ob.n_instances()
        assert of.n_instances() == n
        assert ob.solve_many(range(n)) == of.solve_many(range(n))
        assert [ob.solve_exact(i) for i in range(n)] == [of.solve_exact(i) for i in range(n)]


def test_free_layouts_solve_like_brute_force():
    # the DP over free layouts (mixed neighbours, every type boundary) against
    # enumeration of all partitions, for both objectives
    checked = 0
    for s in range(10):
        p = free(workloads.random_tiny(600 + s, n_types=2 + s % 2, n_layers=4 + s % 5))
        o = orc.Oracle(p)
        for i in range(o.n_instances()):
            a, b = o.solve(i), o.solve_brute(i)
            assert a["status"] == b["status"], (s, i)
            if a["status"] == 0:
                assert (a["opt"], a["sum"], a["tmax"]) == (b["opt"], b["sum"], b["tmax"]), (s, i)
                checked += 1
            e, f = o.solve_exact(i), o.solve_exact_brute(i)
            assert e["status"] == f["status"] and e["opt"] == f["opt"], (s, i)
    assert checked > 50


def test_empty_slots_are_infeasible():
    # a pipeline with fewer sequences than the most has empty order slots
    p = free(workloads.config(2))
    o = orc.Oracle(p)
    nB, no = len(p["space"]["micro"]), o.n_orders()
    cfgs = o.configs()
    counts = [int(x) for x in p["cluster"]["count"]]
    seen = 0
    for ci, cfg in enumerate(cfgs):
        g = sum(counts) // cfg[0]
        n_seq = multinomial([m // g for m in counts])
        if n_seq == no:
            continue
        for oi in (n_seq, no - 1):
            assert o.sequence(cfg[0], oi) is None
            assert o.dp_const(cfg, oi) == 0
            r = o.solve((ci * no + oi) * nB)
            assert r["status"] == 1 and r["opt"] == np.iinfo(np.int64).max
            assert r["stage_mask"] == [0] * cfg[0]
            seen += 1
        r = o.solve((ci * no + n_seq - 1) * nB)
        assert all(m in (1, 2, 4, 8) for m in r["stage_mask"])   # last sequence: pure stages
    assert seen > 0


def test_stage_types_field_is_checked():
    with pytest.raises(ValueError):
        orc.Oracle(variant(workloads.config(1), **{"space.stage_types": 4}))


# ---------------------------------------------------------------------------
# stage_types = 2: the DP over device counts (Section 3.4's state m) picks the
# stage types itself; one order slot per configuration.
def count_dp(p):
    return variant(p, **{"space.stage_types": 2})


def _key(r):
    return (r["status"], r["opt"], r["sum"], r["tmax"], r["layers"], r["types"])


def test_count_dp_core_matches_brute_force():
    # explicit cost tensors with many ties and holes: the DP and the enumeration of
    # every (sequence, composition) agree on the value and on the canonical choice
    rng = np.random.default_rng(11)
    INF = np.iinfo(np.int64).max
    checked = feasible = 0
    while checked < 250:
        T = int(rng.integers(1, 4))
        k = [int(x) for x in rng.integers(0, 3, size=T)]
        if sum(k) == 0:
            k[int(rng.integers(0, T))] = 1
        pp = sum(k)
        if pp > 5:
            continue
        n = int(rng.integers(pp, pp + 4))
        cost = rng.integers(1, int(rng.choice([4, 30, 1000])), size=(pp, T, T + 1, n + 1, n + 1)).astype(np.int64)
        cost[rng.random(cost.shape) < rng.uniform(0.0, 0.5)] = INF
        B = int(rng.integers(1, 6))
        a, b = orc.dp_types(k, n, B, cost), orc.brute_types(k, n, B, cost)
        assert _key(a) == _key(b), (k, n, B, a, b)
        checked += 1
        feasible += a["status"] == 0
    assert feasible > 100


def test_count_dp_is_the_best_stage_type_sequence():
    # on whole problems: the least objective over every sequence of the
    # sequence-enumeration mode, its smallest threshold, and a chosen sequence
    # whose own optimum is that value; brute force agrees in every field
    done = 0
    for seed in range(900, 940):
        base = workloads.random_tiny(seed, n_types=2 + seed % 2)
        o1, o2 = orc.Oracle(free(base)), orc.Oracle(count_dp(base))
        if o1.n_instances() == 0:
            continue
        nB, no = len(base["space"]["micro"]), o1.n_orders()
        assert o2.n_orders() == 1 and o2.configs() == o1.configs()
        assert o2.n_instances() == len(o1.configs()) * nB
        for ci, cfg in enumerate(o1.configs()):
            for j in range(nB):
                rs = o1.solve_many([(ci * no + o) * nB + j for o in range(no)])
                r2, rb = o2.solve(ci * nB + j), o2.solve_brute(ci * nB + j)
                assert {k: r2[k] for k in r2 if k != "thresholds"} == {k: rb[k] for k in rb if k != "thresholds"}
                feas = [r for r in rs if r["status"] == 0]
                if not feas:
                    assert r2["status"] == 1
                    continue
                assert (r2["opt"], r2["tmax"]) == min((r["opt"], r["tmax"]) for r in feas)
                seq = [m.bit_length() - 1 for m in r2["stage_mask"]]
                own = rs[_find_sequence(o1, cfg[0], seq)]
                assert (own["opt"], own["tmax"], own["sum"]) == (r2["opt"], r2["tmax"], r2["sum"])
                assert r2["dp_const"] == o1.dp_const(cfg, 0)
                done += 1
    assert done > 60


def test_count_dp_one_type_is_block_mode():
    for s in range(4):
        p = workloads.random_tiny(300 + s, n_types=1)
        ob, oc = orc.Oracle(p), orc.Oracle(count_dp(p))
        n = ob.n_instances()
        assert oc.n_instances() == n
        for a, b in zip(ob.solve_many(range(n)), oc.solve_many(range(n))):
            skip = ("thresholds",) if a["status"] == 0 else ("thresholds", "stage_mask")   # no chosen types
            assert {k: a[k] for k in a if k not in skip} == {k: b[k] for k in b if k not in skip}


def test_count_dp_config2_against_sequences():
    # 3 device types, pipelines of 4 and 8 stages: a stride sample
    p = workloads.config(2)
    o1, o2 = orc.Oracle(free(p)), orc.Oracle(count_dp(p))
    nB, no = len(p["space"]["micro"]), o1.n_orders()
    cfgs = o1.configs()
    for ci in range(0, len(cfgs), 47):
        for j in range(nB):
            r2 = o2.solve(ci * nB + j)
            rs = [r for r in o1.solve_many([(ci * no + o) * nB + j for o in range(no)]) if r["status"] == 0]
            if not rs:
                assert r2["status"] == 1
                continue
            assert (r2["opt"], r2["tmax"]) == min((r["opt"], r["tmax"]) for r in rs), (ci, j)


def test_count_dp_1f1b_core_matches_brute_force():
    # the 1F1B re-scoring over the device-count frontier: the DP's frontier walk
    # against every (sequence, composition), Pareto filter and canonical choice
    rng = np.random.default_rng(5)
    INF = np.iinfo(np.int64).max
    checked = feasible = 0
    while checked < 250:
        T = int(rng.integers(1, 4))
        k = [int(x) for x in rng.integers(0, 3, size=T)]
        if sum(k) == 0:
            k[0] = 1
        pp = sum(k)
        if pp > 5:
            continue
        n = int(rng.integers(pp, pp + 4))
        cost = rng.integers(1, int(rng.choice([4, 30, 1000])), size=(pp, T, T + 1, n + 1, n + 1)).astype(np.int64)
        cost[rng.random(cost.shape) < rng.uniform(0.0, 0.5)] = INF
        B = int(rng.integers(1, 8))
        a, b = orc.dp_types_exact(k, n, B, cost), orc.brute_types_exact(k, n, B, cost)
        assert _key(a) + (a["thresholds"],) == _key(b) + (b["thresholds"],), (k, n, B, a, b)
        checked += 1
        feasible += a["status"] == 0
    assert feasible > 100


def test_count_dp_1f1b_problems():
    # whole problems: brute force agrees in every field; the chosen plan's latency
    # recomputed from the oracle's cost tensor; one device type is block mode
    done = 0
    for seed in range(900, 930):
        p = count_dp(workloads.random_tiny(seed, n_types=2 + seed % 2))
        o = orc.Oracle(p)
        for i in range(o.n_instances()):
            e, f = o.solve_exact(i), o.solve_exact_brute(i)
            assert {x: e[x] for x in e if x != "thresholds"} == {x: f[x] for x in f if x != "thresholds"}
            if e["status"] != 0:
                continue
            cost, _ = o.type_costs(i)
            types = [m.bit_length() - 1 for m in e["stage_mask"]]
            a, cs = 0, []
            for s, n_i in enumerate(e["layers"]):
                hn = types[s + 1] if s + 1 < len(types) else p["cluster"]["n_types"]
                cs.append(int(cost[s, types[s], hn, a, a + n_i]))
                a += n_i
            B = p["space"]["micro"][i % len(p["space"]["micro"])]
            assert e["opt"] == orc.latency_1f1b(cs, B) + e["dp_const"]
            assert (e["sum"], e["tmax"]) == (sum(cs), max(cs))
            done += 1
    assert done > 30
    for s in range(3):
        p = workloads.random_tiny(300 + s, n_types=1)
        ob, oc = orc.Oracle(p), orc.Oracle(count_dp(p))
        for i in range(ob.n_instances()):
            a, b = ob.solve_exact(i), oc.solve_exact(i)
            if a["status"] == 0:
                assert {x: a[x] for x in a if x != "thresholds"} == {x: b[x] for x in b if x != "thresholds"}
            else:
                assert b["status"] == 1
