"""Pins of the CPU oracle on problem W2 (tests/golden/worked_w2.json), worked by
hand: the branches that W1 reaches only at their neutral values -- TP and CP both
2, TPE = 4 (not TP), EP = 2, DP = 2 -- and a four-stage pipeline whose third stage
straddles two device types."""
import numpy as np
import pytest

from oracle import oracle as orc
from tests.problems import load_golden, variant, worked_problem_w2

G = load_golden("worked_w2.json")
PI = tuple(G["enumeration"]["pi"])


@pytest.fixture(scope="module")
def w2():
    return orc.Oracle(worked_problem_w2())


def test_enumeration(w2):
    e = G["enumeration"]
    assert w2.configs() == [tuple(c) for c in e["configs"]]
    assert w2.configs()[e["pi_index"]] == PI
    assert w2.n_orders() == e["n_orders"] and w2.n_instances() == e["n_instances"]


def test_eq2_expert_divisor_uses_tpe(w2):
    t = G["type_terms"]
    for layer in range(4):
        for h in range(2):
            r = w2.type_terms(PI, layer, h)
            assert [r["q_comp"], r["q_expert"]] == t[f"layer{layer}"][f"h{h}"], (layer, h)
            assert r["expert"] == float(t[f"layer{layer}"][f"h{h}"][1])


def test_collectives_tp_tpe_cp_and_mixed_sets(w2):
    g = G["mask_terms"]
    for key, want in g.items():
        if not key.startswith("set"):
            continue
        mask, layer = int(key[3]), int(key[-1])
        r = w2.mask_terms(PI, layer, mask)
        for field, val in want.items():
            assert r[field] == val, (key, field, r[field], val)
    f = g["fp64"]
    assert abs(w2.mask_terms(PI, 1, 1)["tp"] - f["set1_layer1_tp"]) <= 1e-12 * f["set1_layer1_tp"]
    assert abs(w2.mask_terms(PI, 2, 3)["cp"] - f["set3_layer2_cp"]) <= 1e-12 * f["set3_layer2_cp"]
    assert abs(w2.mask_terms(PI, 3, 2)["a2a"] - f["set2_layer3_a2a"]) <= 1e-12 * f["set2_layer3_a2a"]


def test_memory_sharding_and_optimizer_state_over_dp(w2):
    m = G["memory"]
    for layer, key in ((0, "layer0"), (1, "layer1"), (2, "layer1"), (3, "layer1")):
        r = w2.mem_terms(PI, layer)
        assert [r["q_w"], r["q_a0"], r["q_a1"]] == m[key], layer
    assert w2.pi_terms(PI)["x_bytes"] == m["x_bytes"]


def test_constants(w2):
    c = G["constants"]
    assert w2.p2p(PI, 0, 0) == c["p2p_AA"] and w2.p2p(PI, 1, 1) == c["p2p_BB"]
    assert w2.p2p(PI, 0, 1) == c["p2p_AB"] and w2.p2p(PI, 1, 0) == c["p2p_AB"]
    pt = w2.pi_terms(PI)
    assert pt["tbar"] == c["tbar"] and pt["p_avg"] == c["p_avg"]
    assert w2.dp_const(PI, 0) == c["dp_const"] and w2.dp_const(PI, 1) == c["dp_const"]


@pytest.mark.parametrize("order", [0, 1])
def test_straddling_stage_layout_and_windows(w2, order):
    want = G["stages"][f"order{order}"]
    got = w2.stages(PI, order, 3)
    assert len(got) == 4
    for s, (g, x) in enumerate(zip(got, want)):
        for field, val in x.items():
            assert g[field] == val, (order, s, field, g[field], val)
    mixed = [s for s, x in enumerate(want) if x["mask"] == 3]
    assert [s for s, g in enumerate(got) if g["mixed"]] == mixed


def test_instances(w2):
    for key, idx in (("idx10", 10), ("idx11", 11)):
        r = w2.solve(idx)
        want = G["instances"][key]
        assert r["status"] == 0
        for field, val in want.items():
            assert r[field] == val, (key, field, r[field], val)
        assert r["dp_const"] == G["constants"]["dp_const"]
        assert w2.solve_brute(idx)["opt"] == want["opt"]


def test_pruning3_on_the_straddling_stage():
    h = G["hetero_pruning"]
    o = orc.Oracle(variant(worked_problem_w2(), **{"params.eta_prune": 1}))
    assert (o.solve(10)["status"] == 0) == h["eta1_idx10_feasible"]
    assert (o.solve(11)["status"] == 0) == h["eta1_idx11_feasible"]


def test_pruning3_removes_nothing_without_cross_type_traffic():
    """Section 3.4 pruning 3 targets cross-type communication: on one device
    type no stage has any, so even eta = 0 prunes nothing (the test is strict)."""
    p = worked_problem_w2()
    one = variant(p, **{"cluster.n_types": 1, "cluster.count": np.array([32], dtype=np.int32),
                        "cluster.speed": np.array([100], dtype=np.int32),
                        "cluster.mem_bytes": np.array([36_000_000], dtype=np.int64),
                        "cluster.eff": np.array([1.0]), "cluster.route_coef": np.array([2.0 ** -10]),
                        "cluster.bw": np.array([[400.0]]), "cluster.alpha": np.array([[1000.0]]),
                        "cluster.t_dense": p["cluster"]["t_dense"][:1], "cluster.t_ffn": p["cluster"]["t_ffn"][:1],
                        "params.eta_prune": 0})
    on, off = orc.Oracle(one), orc.Oracle(variant(one, **{"params.prune_hetero": 0}))
    res = [on.solve(i) for i in range(on.n_instances())]
    assert res == [off.solve(i) for i in range(off.n_instances())]
    assert any(r["status"] == 0 for r in res)
