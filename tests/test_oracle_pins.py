"""Pins of the CPU oracle against values the paper's formulas fix by hand,
closed forms, library routines and brute force (no GPU needed)."""
import itertools
import math

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2609_39350_amd import workloads
from tests.problems import load_golden, variant, worked_problem

G = load_golden("worked_w1.json")
INF = orc.INF


@pytest.fixture(scope="module")
def w1():
    return orc.Oracle(worked_problem())


# ---------------------------------------------------------------- enumeration
def test_enumeration_hand_counts(w1):
    e = G["enumeration"]
    cfgs = w1.configs()
    assert len(cfgs) == e["n_configs"]
    assert cfgs[e["pi1_index"]] == tuple(e["pi1"])
    assert cfgs[e["pi2_index"]] == tuple(e["pi2"])
    assert w1.n_orders() == e["n_orders"]


def test_enumeration_config1_hand_counts():
    # PP=1: 10 (TP,CP) pairs with TP*CP | 8 times 10 (EP,TPE) pairs = 100;
    # PP=2: 6 x 6 = 36; PP=4: 3 x 3 = 9  -> 145.
    assert len(orc.Oracle(workloads.config(1)).configs()) == 145
    # literal product: exponent 4-tuples (TP,CP,EP,TPE) with sum <= 3, 2, 1
    # for PP = 1, 2, 4: C(7,4) + C(6,4) + C(5,4) = 35 + 15 + 5 = 55.
    assert len(orc.Oracle(workloads.config(1, mode=1)).configs()) == 55


def _set_builder(p):
    """The candidate set written as a set-builder expression over all tuples."""
    m, c, sp = p["model"], p["cluster"], p["space"]
    G_ = int(sum(c["count"]))
    E = m["n_experts"]
    pows = [1, 2, 4, 8]
    eps = [e for e in (2 ** i for i in range(10)) if E and e <= sp["ep_max"] and E % e == 0] or [1]
    out = []
    for PP, TP, CP, EP, TPE in itertools.product(range(1, G_ + 1), pows, pows, eps, pows):
        if G_ % PP or PP > sp["pp_max"] or PP > m["n_layers"]:
            continue
        g = G_ // PP
        ok = (sp["tp_mask"] >> pows.index(TP)) & 1 and (sp["cp_mask"] >> pows.index(CP)) & 1
        ok = ok and g % TP == 0 and m["hidden"] % TP == 0 and m["seq_len"] % CP == 0
        ok = ok and ((sp["tpe_mask"] >> pows.index(TPE)) & 1 if E else TPE == 1)
        if not ok:
            continue
        if sp["mode"] == 0:
            if g % (TP * CP) or g % (EP * TPE):
                continue
            DP = g // (TP * CP)
        else:
            if g % (TP * CP * EP * TPE):
                continue
            DP = g // (TP * CP * EP * TPE)
        out.append((PP, TP, CP, DP, EP, TPE))
    return sorted(out, key=lambda t: (t[0], t[1], t[2], t[4], t[5]))


@pytest.mark.parametrize("n", [1, 2, 3, 4])
def test_enumeration_matches_set_builder(n):
    p = workloads.config(n)
    assert orc.Oracle(p).configs() == _set_builder(p)


def test_enumeration_random_tiny_matches_set_builder():
    for s in range(40):
        p = workloads.random_tiny(s)
        assert orc.Oracle(p).configs() == _set_builder(p)


def test_orders_are_lexicographic_permutations():
    for T in (1, 2, 3, 4):
        p = workloads.random_tiny(0, n_types=T) if T < 4 else workloads.config(3)
        o = orc.Oracle(p)
        assert [tuple(o.order(i)) for i in range(o.n_orders())] == list(itertools.permutations(range(T)))


# ------------------------------------------------------------- cost model
def test_skew_and_type_terms_eq2(w1):
    pi1 = G["enumeration"]["pi1"]
    t = G["type_terms_pi1"]
    for layer in (0, 1):
        for h in (0, 1):
            r = w1.type_terms(pi1, layer, h)
            assert [r["q_comp"], r["q_expert"]] == t[f"layer{layer}"][f"h{h}"]
    assert w1.type_terms(pi1, 1, 0)["expert"] == t["layer1_fp64"]["h0_expert"]
    assert w1.type_terms(pi1, 1, 1)["expert"] == t["layer1_fp64"]["h1_expert"]


def test_mask_terms_eq3_and_collectives(w1):
    pi1 = G["enumeration"]["pi1"]
    g = G["mask_terms_pi1"]
    for key, (mask, layer) in {"mask1_layer0": (1, 0), "mask1_layer1": (1, 1), "mask2_layer0": (2, 0),
                               "mask2_layer1": (2, 1), "mask3_layer1": (3, 1)}.items():
        r = w1.mask_terms(pi1, layer, mask)
        for field, val in g[key].items():
            assert r[field] == val, (key, field)


def test_primitive_selection_allgather():
    o = orc.Oracle(variant(worked_problem(), **{"model.top_k": 4}))
    assert o.mask_terms([2, 2, 1, 1, 2, 1], 1, 1)["q_a2a"] == G["allgather_selection"]["q_a2a"]


def test_cp_ring_term(w1):
    g = G["cp_term"]
    assert w1.mask_terms(g["pi"], 0, 1)["q_cp"] == g["mask1"]
    assert w1.mask_terms(g["pi"], 0, 3)["q_cp"] == g["mask3"]


def test_memory_terms(w1):
    pi1 = G["enumeration"]["pi1"]
    g = G["memory_pi1"]
    for layer in (0, 1):
        r = w1.mem_terms(pi1, layer)
        assert [r["q_w"], r["q_a0"], r["q_a1"]] == g[f"layer{layer}"]
    assert w1.pi_terms(pi1)["x_bytes"] == g["x_bytes"]


def test_constants(w1):
    e, g = G["enumeration"], G["constants_pi1"]
    pi1, pi2 = e["pi1"], e["pi2"]
    assert w1.p2p(pi1, 0, 1) == g["p2p_01"] and w1.p2p(pi1, 1, 0) == g["p2p_01"]
    assert w1.p2p(pi1, 0, 0) == g["p2p_00"]
    assert w1.pi_terms(pi1)["tbar"] == g["tbar"]
    assert w1.dp_const(pi1, 0) == g["dp_const"] and w1.dp_const(pi1, 1) == g["dp_const"]
    assert w1.dp_const(pi2, 0) == g["pi2_dp_const"]


def test_windows(w1):
    pi1 = G["enumeration"]["pi1"]
    for o in (0, 1):
        st = w1.stages(pi1, o, 4)
        assert [[s["lo"], s["hi"]] for s in st] == G["windows_pi1"][f"order{o}"]
        assert [s["m_store"] for s in st] == [2, 1]


def test_worked_instances(w1):
    for key, exp in G["instances"].items():
        if not key.startswith("idx"):
            continue
        r = w1.solve(int(key[3:]))
        assert r["status"] == 0
        for f, v in exp.items():
            assert r[f] == v, (key, f)


def test_recompute_and_memory_boundary():
    g = G["recompute"]
    o = orc.Oracle(variant(worked_problem(), **{"cluster.mem_bytes": np.array([60_000_000, 20 * 10**9])}))
    for key, exp in g["cap0_60e6"].items():
        r = o.solve(int(key[3:]))
        assert r["status"] == 0 and r["opt"] == exp["opt"] and r["recompute"] == exp["recompute"]
    at = orc.Oracle(variant(worked_problem(), **{"cluster.mem_bytes": np.array([49_000_000, 20 * 10**9])}))
    below = orc.Oracle(variant(worked_problem(), **{"cluster.mem_bytes": np.array([48_999_999, 20 * 10**9])}))
    assert (at.solve(88)["status"] == 0) == g["cap0_49e6_idx88_feasible"]
    assert (below.solve(88)["status"] == 0) == g["cap0_48999999_idx88_feasible"]
    norc = orc.Oracle(variant(worked_problem(), **{"cluster.mem_bytes": np.array([60_000_000, 20 * 10**9]),
                                                   "params.allow_recompute": 0}))
    assert norc.solve(89)["status"] == 1


def test_hetero_pruning():
    o = orc.Oracle(variant(worked_problem(), **{"params.eta_prune": 0}))
    assert o.solve(88)["status"] == 1 and o.solve(89)["status"] == 1
    off = orc.Oracle(variant(worked_problem(), **{"params.eta_prune": 0, "params.prune_hetero": 0}))
    assert off.solve(88)["status"] == 0


def test_cost_model_special_cases():
    p = workloads.config(2)
    o = orc.Oracle(p)
    for cfg in o.configs()[::37]:
        for layer in (0, 5):
            for mask in (1, 2, 4, 7):
                r = o.mask_terms(cfg, layer, mask)
                if cfg[4] == 1:                      # EP = 1: no dispatch/combine
                    assert r["a2a"] == 0.0
                if cfg[1] == 1 and cfg[5] == 1:      # TP = TPE = 1: no TP collectives
                    assert r["tp"] == 0.0
                if cfg[2] == 1:
                    assert r["cp"] == 0.0
                assert r["t_r1"] >= r["t_r0"] >= r["comm"] >= 0


def test_eq2_paper_literal_form():
    # mult = 2, eta = 1, EP = TPE = 1, gamma = 0: comp + expert = t_base + t_ffn + t_route
    p = variant(worked_problem(), **{"params.gamma": 0.0, "cluster.eff": np.array([1.0, 1.0])})
    o = orc.Oracle(p)
    r = o.type_terms([1, 1, 1, 4, 1, 1], 1, 0)
    # td = 160000, tf = 80000 at TP = CP = 1; route = 0.001 * 1024 * 512 = 524.288
    assert r["q_comp"] + r["q_expert"] == 160000 + 80000 + 525


def test_skew_uniform_and_onehot():
    base = worked_problem()
    uni = variant(base, **{"model.expert_tokens": np.array([[0] * 4, [512] * 4], dtype=np.int64)})
    one = variant(base, **{"model.expert_tokens": np.array([[0] * 4, [2048, 0, 0, 0]], dtype=np.int64)})
    cfg = [1, 1, 1, 4, 2, 1]
    r0 = orc.Oracle(variant(uni, **{"params.gamma": 0.0})).mask_terms(cfg, 1, 1)["a2a"]
    r1 = orc.Oracle(variant(uni, **{"params.gamma": 1.0})).mask_terms(cfg, 1, 1)["a2a"]
    assert r0 == r1                                  # rho = 1 for uniform routing
    h0 = orc.Oracle(variant(one, **{"params.gamma": 0.0})).mask_terms(cfg, 1, 1)["a2a"]
    h1 = orc.Oracle(variant(one, **{"params.gamma": 1.0})).mask_terms(cfg, 1, 1)["a2a"]
    assert h1 == 4 * h0                              # rho = E = 4 for one-hot routing


def test_monotone_in_bandwidth_and_ep():
    p = workloads.config(2)
    fast = variant(p, **{"cluster.bw": p["cluster"]["bw"] * 2.0})
    o, f = orc.Oracle(p), orc.Oracle(fast)
    cfgs = o.configs()
    for cfg in cfgs[::53]:
        for mask in (1, 3, 7):
            assert f.mask_terms(cfg, 3, mask)["comm"] <= o.mask_terms(cfg, 3, mask)["comm"]
    by_ep = {}
    for cfg in cfgs:
        by_ep.setdefault((cfg[0], cfg[1], cfg[2], cfg[5]), []).append(cfg)
    for grp in by_ep.values():
        grp.sort(key=lambda c: c[4])
        vals = [o.type_terms(c, 3, 0)["expert"] for c in grp]
        assert all(a >= b for a, b in zip(vals, vals[1:]))


# ------------------------------------------------------------------ the DP
def _random_costs(rng, pp, n, p_inf):
    c = rng.integers(1, 60, size=(pp, n + 1, n + 1)).astype(np.int64)
    c[rng.random(c.shape) < p_inf] = INF
    for i in range(pp):
        for a in range(n + 1):
            c[i, a, : a + 1] = INF
    return c


def _check_partition(res, cost, micro):
    pp, n = cost.shape[0], cost.shape[1] - 1
    assert sum(res["layers"]) == n and min(res["layers"]) >= 1
    a, costs = 0, []
    for i, k in enumerate(res["layers"]):
        costs.append(int(cost[i, a, a + k]))
        a += k
    assert INF not in costs
    assert res["sum"] == sum(costs)
    assert res["tmax"] == max(costs)
    assert res["opt"] == res["sum"] + (micro - 1) * res["tmax"]


def test_dp_equals_brute_force_random_costs():
    rng = np.random.default_rng(7)
    for trial in range(600):
        pp = int(rng.integers(1, 5))
        n = int(rng.integers(pp, 11))
        micro = int(rng.choice([1, 2, 3, 8, 64]))
        cost = _random_costs(rng, pp, n, float(rng.choice([0.0, 0.3, 0.6])))
        d, b = orc.dp(pp, n, micro, cost), orc.brute(pp, n, micro, cost)
        assert d["status"] == b["status"]
        if b["status"] == 0:
            for k in ("opt", "sum", "tmax", "layers"):
                assert d[k] == b[k], (trial, k)
            _check_partition(d, cost, micro)


def test_dp_ties_low_values():
    # many equal costs: exercises the canonical tie rule
    rng = np.random.default_rng(11)
    for _ in range(300):
        pp = int(rng.integers(1, 5))
        n = int(rng.integers(pp, 10))
        micro = int(rng.choice([1, 2, 5]))
        cost = rng.integers(1, 3, size=(pp, n + 1, n + 1)).astype(np.int64)
        for i in range(pp):
            for a in range(n + 1):
                cost[i, a, : a + 1] = INF
        d, b = orc.dp(pp, n, micro, cost), orc.brute(pp, n, micro, cost)
        assert (d["opt"], d["tmax"], d["layers"]) == (b["opt"], b["tmax"], b["layers"])


def _uniform(pp, n, u):
    c = np.full((pp, n + 1, n + 1), INF, dtype=np.int64)
    for a in range(n + 1):
        for b in range(a + 1, n + 1):
            c[:, a, b] = u * (b - a)
    return c


def test_dp_closed_forms():
    # one stage: OPT = B * c(0, N)
    for n in (1, 5, 12):
        for micro in (1, 4):
            r = orc.dp(1, n, micro, _uniform(1, n, 7))
            assert r["opt"] == micro * 7 * n and r["layers"] == [n]
    # uniform per-layer cost u: OPT = N u + (B-1) u ceil(N/PP); the last stages take ceil(N/PP)
    r = orc.dp(4, 10, 5, _uniform(4, 10, 3))
    assert r["opt"] == 10 * 3 + 4 * 3 * 3 and r["layers"] == [1, 3, 3, 3]
    # PP = N: the unique partition
    r = orc.dp(6, 6, 3, _uniform(6, 6, 2))
    assert r["layers"] == [1] * 6 and r["opt"] == 12 + 2 * 2
    # every stage infeasible
    c = np.full((2, 5, 5), INF, dtype=np.int64)
    assert orc.dp(2, 4, 3, c)["status"] == 1


def _painter(weights, k):
    """Textbook linear partition: least possible largest part, by binary search + greedy."""
    lo, hi = max(weights), sum(weights)
    while lo < hi:
        mid = (lo + hi) // 2
        parts, cur = 1, 0
        for w in weights:
            if cur + w > mid:
                parts, cur = parts + 1, 0
            cur += w
        if parts <= k:
            hi = mid
        else:
            lo = mid + 1
    return lo


def test_dp_reduces_to_linear_partition():
    # identical stages, no windows/memory/P2P, large B: the max term dominates and the
    # optimum is the painter's-partition bottleneck with sum = total
    rng = np.random.default_rng(3)
    for _ in range(200):
        n = int(rng.integers(2, 14))
        pp = int(rng.integers(1, min(n, 6) + 1))
        w = rng.integers(1, 100, size=n)
        pre = np.concatenate([[0], np.cumsum(w)])
        c = np.full((pp, n + 1, n + 1), INF, dtype=np.int64)
        for a in range(n + 1):
            for b in range(a + 1, n + 1):
                c[:, a, b] = pre[b] - pre[a]
        r = orc.dp(pp, n, 10**6, c)
        assert r["tmax"] == _painter(list(w), pp)
        assert r["sum"] == int(pre[-1])


def test_full_pipeline_equals_brute_force_random_tiny():
    checked = 0
    for s in range(60):
        p = workloads.random_tiny(s)
        o = orc.Oracle(p)
        n = o.n_instances()
        for idx in range(0, n, max(1, n // 12)):
            d, b = o.solve(idx), o.solve_brute(idx)
            assert d["status"] == b["status"], (s, idx)
            if d["status"] == 0:
                assert (d["opt"], d["tmax"], d["layers"], d["recompute"]) == \
                       (b["opt"], b["tmax"], b["layers"], b["recompute"]), (s, idx)
                checked += 1
    assert checked > 50


def test_invariants_memory_and_micro():
    for s in range(25):
        p = workloads.random_tiny(s, micro=[2])
        big = variant(p, **{"cluster.mem_bytes": p["cluster"]["mem_bytes"] * 2})
        o, ob = orc.Oracle(p), orc.Oracle(big)
        for idx in range(0, o.n_instances(), 3):
            a, b = o.solve(idx), ob.solve(idx)
            if a["status"] == 0:
                assert b["status"] == 0 and b["opt"] <= a["opt"]
    for s in range(25):
        p = workloads.random_tiny(s, micro=[1, 2, 4, 9])
        o = orc.Oracle(p)
        for base in range(0, o.n_instances(), 4 * 5):
            opts = [o.solve(base + j)["opt"] for j in range(4)]
            assert all(x <= y for x, y in zip(opts, opts[1:]))


def test_config1_chosen_partition_is_feasible_and_consistent():
    p = workloads.config(1)
    o = orc.Oracle(p)
    for idx in range(o.n_instances()):
        r = o.solve(idx)
        if r["status"]:
            continue
        cost, rflag = o.segment_costs(idx)
        _check_partition({**r, "opt": r["opt"] - r["dp_const"]}, cost, p["space"]["micro"][idx % 1])
        a = 0
        for i, k in enumerate(r["layers"]):
            assert rflag[i, a, a + k] == r["recompute"][i]
            a += k


def test_segment_costs_monotone_in_length():
    # a longer segment never costs less, and memory feasibility shrinks with length
    p = workloads.config(2)
    o = orc.Oracle(p)
    for idx in range(5, o.n_instances(), 997):
        cost, _ = o.segment_costs(idx)
        pp, W = cost.shape[0], cost.shape[1]
        for i in range(pp):
            for b in range(W):
                row = [int(cost[i, a, b]) for a in range(b)]
                fin = [a for a in range(b) if row[a] != INF]
                if fin:
                    assert fin == list(range(fin[0], fin[-1] + 1))
                    vals = [row[a] for a in fin]
                    assert all(x >= y for x, y in zip(vals, vals[1:]))


@pytest.mark.parametrize("n,n_configs,n_candidates", [(1, 145, 290), (2, 904, 16272), (3, 1636, 117792),
                                                      (4, 2510, 3855360), (5, 1636, 117792)])
def test_enumeration_pinned_counts(n, n_configs, n_candidates):
    """Configuration and candidate counts of the five workloads, counted
    independently of both enumerators from the loop rules (PP | G, TP | group and
    hidden, CP | sequence, EP | experts, EP * TPE | group) times the orderings
    and micro-batch counts."""
    o = orc.Oracle(workloads.config(n))
    assert len(o.configs()) == n_configs
    assert o.n_instances() == n_candidates
