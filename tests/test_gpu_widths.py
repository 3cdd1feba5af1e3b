"""Per-stage data-parallel widths on the GPU (hapmoe_stage_dp_widths) against
the oracle, through the C ABI: status, objective, stage sum, largest stage,
recomputation mask, stage lengths, stage type sets and widths bit-exact."""
import copy

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2609_39350_amd import binding, workloads
from tests import parity_digest
from tests.problems import worked_problem_w2

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def widths(p, **kw):
    q = copy.deepcopy(p)
    q["space"]["stage_types"] = 3
    for k, v in kw.items():
        q["params"][k] = v
    return q


def compare(problem, pl, idx, ref=None):
    res, types, wd = pl.results(), pl.stage_types(), pl.widths()
    if ref is None:
        o = orc.Oracle(problem)
        ref = [o.solve(int(i)) for i in idx]
    bad, feasible = [], 0
    for i, r in zip(idx, ref):
        g = res[i]
        if int(g["status"]) != r["status"]:
            bad.append((int(i), "status", int(g["status"]), r["status"]))
            continue
        if r["status"]:
            assert not types[i].any() and not wd[i].any()
            continue
        feasible += 1
        pp = r["pp"]
        got = (int(g["objective"]), int(g["stage_sum"]), int(g["t_max"]), list(g["layers"][:pp]),
               [(int(g["recompute_mask"]) >> s) & 1 for s in range(pp)], [int(x) for x in types[i][:pp]],
               [int(x) for x in wd[i][:pp]])
        exp = (r["opt"], r["sum"], r["tmax"], r["layers"], r["recompute"], r["stage_mask"], r["width"])
        if got != exp:
            bad.append((int(i), got, exp))
    assert not bad, f"{len(bad)} mismatches, first: {bad[:3]}"
    return feasible


def _run(p):
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run()
    return pl, plan


def test_worked_problem_and_config1_every_candidate(torch):
    for p in (widths(worked_problem_w2()), widths(workloads.config(1))):
        print(f"widths: {p['name']}", flush=True)
        pl, plan = _run(p)
        assert compare(p, pl, range(pl.n)) > 0
        res = pl.results()
        obj = np.where(res["status"] == 0, res["objective"], np.iinfo(np.int64).max)
        assert plan["instance"] == int(np.argmin(obj)) and plan["objective"] == int(obj.min())
        assert sum(plan["widths"]) == 2 * plan["config"][0]


def test_random_tiny_every_candidate(torch):
    total = 0
    for s in range(16):
        p = widths(workloads.random_tiny(700 + s, n_layers=int(4 + s % 6), max_pp=4))
        try:
            orc.Oracle(p)
        except ValueError:
            continue
        print(f"widths: {p['name']}", flush=True)
        pl = binding.Planner(p, "cuda:0")
        pl.eval_cost_tables()
        pl.stage_dp()
        total += compare(p, pl, range(pl.n))
    assert total > 30


@pytest.mark.parametrize("window", [1, 0])
def test_config2_sampled(torch, window):
    p = widths(workloads.config(2), prune_window=window)
    print(f"widths: config 2, windows {window}", flush=True)
    pl, plan = _run(p)
    idx = sorted(set(list(range(3, pl.n, max(1, pl.n // 160))) + [plan["instance"]]))
    from tests.test_gpu_parity import oracle_many
    assert compare(p, pl, idx, ref=oracle_many(p, idx, pool=True)) > 0


def test_config2_every_candidate(torch):
    """Every candidate of configuration 2 (10,584, one launch) against stored
    oracle digests of status, objective, stage sum, largest stage,
    recomputation mask, stage lengths, stage type sets and widths
    (tests/golden/parity_refs.npz, written from oracle/ alone)."""
    import os
    refs_path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "parity_refs.npz")
    with np.load(refs_path) as f:
        if "cfg2_widths" not in f.files:
            pytest.skip("no per-stage widths references in parity_refs.npz")
        idx, ref = f["cfg2_widths_idx"], f["cfg2_widths"]
    p = widths(workloads.config(2))
    print("widths: config 2, every candidate against stored oracle digests", flush=True)
    pl, plan = _run(p)
    assert len(idx) == pl.n
    got = parity_digest.of_gpu(pl.results(), idx, pl.stage_types(), pl.widths())
    bad = np.nonzero(got != ref)[0]
    assert len(bad) == 0, f"{len(bad)} of {len(idx)} differ, first: {idx[bad][:5]}"
    assert (pl.results()["status"] == 0).sum() > 1000


def test_config2_sub_ranges_equal_one_launch(torch):
    p = widths(workloads.config(2))
    pl, _ = _run(p)
    whole = (pl.results().copy(), pl.stage_types().copy(), pl.widths().copy())
    pl.d_res.zero_()
    pl.d_types.zero_()
    pl.d_widths.zero_()
    cuts = [0, 1, 2500, 2500, 7001, pl.n]
    for a, b in zip(cuts[:-1], cuts[1:]):
        pl.stage_dp(first=a, count=b - a)
    assert np.array_equal(pl.results(), whole[0])
    assert np.array_equal(pl.stage_types(), whole[1]) and np.array_equal(pl.widths(), whole[2])


def test_config3_launch_and_shallow_sample(torch):
    """The 61-layer workload in width mode (93,888 candidates, one launch); the
    oracle on a sample of the pipelines of up to 4 stages, and the properties of
    every result."""
    p = widths(workloads.config(3))
    print("widths: config 3", flush=True)
    pl, plan = _run(p)
    res, wd = pl.results(), pl.widths()
    ok = res["status"] == 0
    pp = pl.cand_host["pp"]
    assert (wd[ok].astype(int).sum(axis=1) == 2 * pp[ok]).all()
    assert (res["layers"][ok].astype(int).sum(axis=1) == p["model"]["n_layers"]).all()
    shallow = np.nonzero(pp <= 4)[0]
    idx = sorted(set(shallow[:: max(1, len(shallow) // 120)].tolist()))
    from tests.test_gpu_parity import oracle_many
    assert compare(p, pl, idx, ref=oracle_many(p, idx, pool=True)) > 0
