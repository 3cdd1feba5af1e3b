"""Pins of the oracle's per-stage data-parallel widths (stage_types = 3): the
width-scaled terms worked by hand on W2 (tests/golden/worked_widths.json), the
reduction to the pinned uniform model at width 2, brute force over every width
sequence and composition, and invariants."""
import copy

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2609_39350_amd import workloads
from tests.problems import load_golden, variant, worked_problem_w2

G = load_golden("worked_widths.json")
INF = orc.INF


def widths(p, **kw):
    q = copy.deepcopy(p)
    q["space"]["stage_types"] = 3
    for k, v in kw.items():
        q["params"][k] = v
    return q


@pytest.fixture(scope="module")
def w2w():
    return orc.Oracle(widths(worked_problem_w2()))


def test_configurations(w2w):
    assert w2w.configs() == [tuple(c) for c in G["configs"]["list"]]


def test_hand_worked_width_terms(w2w):
    pi = tuple(G["pi"])
    g = G["width1_layer1"]
    t = w2w.width_terms(pi, 1, 1, 1)
    assert [[x["q_comp"], x["q_expert"]] for x in t["type"]] == g["type"]
    for k, v in g["set1"].items():
        assert t["mask"][k] == v, k
    assert [t["mem"]["q_w"], t["mem"]["q_a0"], t["mem"]["q_a1"]] == g["mem"]
    assert t["x_bytes"] == g["x_bytes"]
    g3 = G["width3_layer1"]
    t = w2w.width_terms(pi, 1, 1, 3)
    assert [t["type"][0]["q_comp"], t["type"][0]["q_expert"]] == g3["typeA"]
    assert [t["mem"]["q_w"], t["mem"]["q_a0"]] == g3["mem_w_a0"] and t["x_bytes"] == g3["x_bytes"]
    st = G["stages"]
    for key, (s, u, w) in (("s0_u0_w1", (0, 0, 1)), ("s3_u5_w3", (3, 5, 3))):
        x = w2w.width_stage(pi, 0, s, u, w, 3)
        for k, v in st[key].items():
            assert x[k] == v, (key, k)


@pytest.mark.parametrize("n", [1, 2])
def test_width_two_is_the_uniform_model(n):
    """Every stage at its nominal group (w = 2 at half-group 2s) costs what the
    uniform block layout's stage s costs, windows aside (no windows here)."""
    base = variant(workloads.config(n), **{"params.prune_window": 0})
    ou, ow = orc.Oracle(base), orc.Oracle(widths(base))
    cu, cw = ou.configs(), ow.configs()
    per_u, per_w = ou.n_orders() * len(base["space"]["micro"]), ow.n_orders() * len(base["space"]["micro"])
    for k in range(0, len(cw), max(1, len(cw) // 25)):
        iw = k * per_w + (k % per_w)
        iu = cu.index(cw[k]) * per_u + (k % per_w)
        cost_u, rf_u = ou.segment_costs(iu)
        cost_w, rf_w = ow.width_costs(iw)
        for s in range(cw[k][0]):
            assert np.array_equal(cost_w[s, 2 * s, 1], cost_u[s]), (k, s)
            assert np.array_equal(rf_w[s, 2 * s, 1], rf_u[s]), (k, s)


def _random_width_tensor(rng, pp, n, p_inf):
    U = 2 * pp
    c = np.full((pp, U + 1, 3, n + 1, n + 1), INF, dtype=np.int64)
    lw = rng.integers(1, 12, size=n)
    for s in range(pp):
        for u in range(U + 1):
            for w in range(1, 4):
                if u + w > U:
                    continue
                for a in range(n):
                    for b in range(a + 1, n + 1):
                        if rng.random() < p_inf:
                            continue
                        c[s, u, w - 1, a, b] = int(lw[a:b].sum()) * (4 - w) + int(rng.integers(0, 3))
    return c


def test_dp_matches_brute_force_on_tensors():
    rng = np.random.default_rng(21)
    feasible = 0
    for trial in range(250):
        pp = int(rng.integers(1, 4))
        n = int(rng.integers(pp, 8))
        c = _random_width_tensor(rng, pp, n, float(rng.choice([0.0, 0.3, 0.6])))
        B = int(rng.integers(1, 10))
        d, b = orc.dp_widths(pp, n, B, c), orc.brute_widths(pp, n, B, c)
        assert d["status"] == b["status"], trial
        if d["status"] == 0:
            feasible += 1
            assert (d["opt"], d["sum"], d["tmax"], d["layers"], d["width"]) == \
                   (b["opt"], b["sum"], b["tmax"], b["layers"], b["width"]), trial
            assert sum(d["width"]) == 2 * pp
    assert feasible > 120


def test_full_problems_match_brute_force():
    checked = 0
    for s in range(12):
        p = widths(workloads.random_tiny(700 + s, n_layers=int(4 + s % 4), max_pp=4))
        try:
            o = orc.Oracle(p)
        except ValueError:
            continue
        for i in range(o.n_instances()):
            d, b = o.solve(i), o.solve_brute(i)
            assert d == dict(b, thresholds=d["thresholds"]), (s, i)
            checked += d["status"] == 0
    assert checked > 30


@pytest.mark.parametrize("n", [1, 2])
def test_never_worse_than_uniform_without_windows(n):
    """Without windows, width 2 everywhere is one of the width plans, so the
    width optimum is at most the uniform one (same configuration, ordering, B);
    on the heterogeneous clusters it is lower for some candidates."""
    base = variant(workloads.config(n), **{"params.prune_window": 0})
    ou, ow = orc.Oracle(base), orc.Oracle(widths(base))
    cu, cw = ou.configs(), ow.configs()
    nb = len(base["space"]["micro"])
    per_u, per_w = ou.n_orders() * nb, ow.n_orders() * nb
    lower = 0
    for k in range(0, len(cw), max(1, len(cw) // 12)):
        for j in range(per_w):
            d, u = ow.solve(k * per_w + j), ou.solve(cu.index(cw[k]) * per_u + j)
            assert (d["status"] == 0) >= (u["status"] == 0)
            if u["status"] == 0:
                assert d["opt"] <= u["opt"]
                lower += d["opt"] < u["opt"]
    assert lower > 0


def test_more_memory_never_worse():
    p = widths(workloads.config(1))
    big = variant(p, **{"cluster.mem_bytes": p["cluster"]["mem_bytes"] * 2})
    o, ob = orc.Oracle(p), orc.Oracle(big)
    for i in range(o.n_instances()):
        a, b = o.solve(i), ob.solve(i)
        if a["status"] == 0:
            assert b["status"] == 0 and b["opt"] <= a["opt"]
