"""Pins of the oracle's 1F1B re-scoring of the (max, sum) Pareto frontier.

Hand-worked tensors (tests/golden/exact_1f1b.json), brute force over every
composition, a closed form for uniform layers and invariants -- none of them
re-types the oracle's code.
"""
import json
import os

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2609_39350_amd import workloads

INF = orc.INF
GOLD = os.path.join(os.path.dirname(__file__), "golden", "exact_1f1b.json")


def tensor(pp, n, entries):
    c = np.full((pp, n + 1, n + 1), INF, dtype=np.int64)
    for i, a, b, v in entries:
        c[i, a, b] = v
    return c


def cases():
    with open(GOLD) as f:
        for case in json.load(f)["cases"]:
            for e in case["expect"]:
                yield case, e


@pytest.mark.parametrize("case,e", list(cases()), ids=lambda x: x["name"] if "name" in x else f"B{x['B']}")
def test_hand_worked(case, e):
    c = tensor(case["pp"], case["n"], case["costs"])
    for solver in (orc.dp_exact, orc.brute_exact):
        r = solver(case["pp"], case["n"], e["B"], c)
        assert r["status"] == 0
        assert (r["opt"], r["sum"], r["tmax"], r["layers"], r["thresholds"]) == \
               (e["opt"], e["sum"], e["tmax"], e["layers"], e["points"]), solver.__name__


def random_tensor(rng, pp, n, p_inf, additive):
    c = np.full((pp, n + 1, n + 1), INF, dtype=np.int64)
    w = rng.integers(1, 20, size=n)
    for i in range(pp):
        for a in range(n):
            for b in range(a + 1, n + 1):
                if rng.random() < p_inf:
                    continue
                v = int(w[a:b].sum()) if additive else int(rng.integers(1, 60))
                c[i, a, b] = v + (int(rng.integers(0, 3)) if additive else 0)
    return c


def test_dp_exact_matches_brute_force():
    rng = np.random.default_rng(7)
    n_feasible = 0
    for trial in range(600):
        pp = int(rng.integers(1, 5))
        n = int(rng.integers(pp, 10))
        c = random_tensor(rng, pp, n, float(rng.choice([0.0, 0.2, 0.5])), bool(trial % 2))
        B = int(rng.integers(1, 12))
        d, b = orc.dp_exact(pp, n, B, c), orc.brute_exact(pp, n, B, c)
        assert d["status"] == b["status"]
        if d["status"] == 0:
            n_feasible += 1
            assert (d["opt"], d["sum"], d["tmax"], d["layers"], d["thresholds"]) == \
                   (b["opt"], b["sum"], b["tmax"], b["layers"], b["thresholds"]), trial
    assert n_feasible > 300


def test_uniform_layers_closed_form():
    # additive equal layer costs u, N = PP * k: every partition sums to N*u, the
    # least largest stage is k*u and only the uniform partition reaches it, so the
    # frontier is one point; its first stage is the bottleneck
    for pp, k, u, B in ((1, 5, 7, 4), (2, 3, 5, 1), (3, 2, 11, 9), (4, 3, 4, 2)):
        n = pp * k
        c = np.full((pp, n + 1, n + 1), INF, dtype=np.int64)
        for i in range(pp):
            for a in range(n):
                for b in range(a + 1, n + 1):
                    c[i, a, b] = (b - a) * u
        r = orc.dp_exact(pp, n, B, c)
        expect = n * u + -(-(k * u) // 3) + max(0, B - 2) * k * u
        assert (r["opt"], r["sum"], r["tmax"], r["layers"], r["thresholds"]) == (expect, n * u, k * u, [k] * pp, 1)


def test_invariants_on_tensors():
    rng = np.random.default_rng(11)
    for trial in range(200):
        pp = int(rng.integers(1, 5))
        n = int(rng.integers(pp, 11))
        c = random_tensor(rng, pp, n, 0.2, bool(trial % 2))
        prev = None
        for B in range(1, 10):
            e, t = orc.dp_exact(pp, n, B, c), orc.dp(pp, n, B, c)
            assert e["status"] == t["status"]
            if e["status"]:
                continue
            # the threshold objective's partition is on the frontier, so the
            # re-scored optimum is at most its latency
            a, cs = 0, []
            for i, ln in enumerate(t["layers"]):
                cs.append(int(c[i, a, a + ln]))
                a += ln
            assert e["opt"] <= orc.latency_1f1b(cs, B)
            # the latency of every partition grows with B
            if prev is not None:
                assert e["opt"] >= prev
            prev = e["opt"]
            # the chosen partition's own latency and its (max, sum)
            a, cs = 0, []
            for i, ln in enumerate(e["layers"]):
                cs.append(int(c[i, a, a + ln]))
                a += ln
            assert (sum(cs), max(cs), orc.latency_1f1b(cs, B)) == (e["sum"], e["tmax"], e["opt"])
            assert e["thresholds"] >= 1


def test_full_problems_match_brute_force():
    checked = 0
    for s in range(10):
        p = workloads.random_tiny(300 + s, n_layers=int(6 + s % 4))
        o = orc.Oracle(p)
        for i in range(o.n_instances()):
            d, b = o.solve_exact(i), o.solve_exact_brute(i)
            assert d["status"] == b["status"]
            if d["status"] == 0:
                checked += 1
                assert (d["opt"], d["sum"], d["tmax"], d["layers"], d["recompute"]) == \
                       (b["opt"], b["sum"], b["tmax"], b["layers"], b["recompute"]), (s, i)
                # the constant C is added as on the main path
                micro = p["space"]["micro"][i % len(p["space"]["micro"])]
                assert d["opt"] - d["dp_const"] == orc.latency_1f1b(_stage_costs(o, i, d), micro)
    assert checked > 50


def _stage_costs(o, i, r):
    cost, _ = o.segment_costs(i)
    a, cs = 0, []
    for k, ln in enumerate(r["layers"]):
        cs.append(int(cost[k, a, a + ln]))
        a += ln
    return cs
