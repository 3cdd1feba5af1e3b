"""GPU path vs the CPU oracle, through the C ABI (needs an MI355X).

The bar (integer/index work): bit-exact objective, stage sum, t*, partition,
recomputation choice and status for every compared candidate; fp64 terms
before rounding within 1e-12 relative.  Small problems are compared in full;
the large configurations on a fixed stride sample plus the chosen best plan.
"""
import copy
import multiprocessing as mp
import os

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2609_39350_amd import binding, workloads
from tests.problems import variant, worked_problem, worked_problem_w2

pytestmark = pytest.mark.gpu

_POOL = None


def _pool():
    """Oracle worker processes (spawned: they never touch the GPU)."""
    global _POOL
    if _POOL is None:
        n = max(1, min(16, os.cpu_count() or 1))
        _POOL = mp.get_context("spawn").Pool(n)
    return _POOL


def oracle_many(problem, idx, objective="threshold", pool=None):
    """The oracle on candidates idx: in worker processes for long lists (or when
    pool is True: few candidates that take seconds each)."""
    idx = [int(i) for i in idx]
    if not pool and len(idx) < 64:
        o = orc.Oracle(problem)
        return o.solve_many(idx) if objective == "threshold" else o.solve_exact_many(idx)
    n = _pool()._processes
    parts = [idx[k::n] for k in range(n)]
    mode = "main" if objective == "threshold" else "exact"
    outs = _pool().map(orc.solve_worker, [(problem, part, mode) for part in parts])
    res = [None] * len(idx)
    for k, out in enumerate(outs):
        for j, r in enumerate(out):
            res[k + j * n] = r
    return res


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def compare(problem, planner, idx, res=None, objective="threshold", ref=None):
    """Element-by-element parity of the DP results at candidate indices idx
    (ref: the oracle's results there, if already computed)."""
    res = planner.results() if res is None else res
    ref = oracle_many(problem, idx, objective) if ref is None else ref
    bad = []
    for i, r in zip(idx, ref):
        g = res[i]
        st = int(g["status"])
        if st != r["status"]:
            bad.append((int(i), "status", st, r["status"]))
            continue
        if st != 0:
            assert int(g["objective"]) == np.iinfo(np.int64).max
            continue
        pp = r["pp"]
        got = (int(g["objective"]), int(g["stage_sum"]), int(g["t_max"]), list(g["layers"][:pp]),
               [(int(g["recompute_mask"]) >> s) & 1 for s in range(pp)])
        exp = (r["opt"], r["sum"], r["tmax"], r["layers"], r["recompute"])
        if got != exp:
            bad.append((int(i), got, exp))
        assert all(v == 0 for v in g["layers"][pp:])
    assert not bad, f"{len(bad)} mismatches, first: {bad[:3]}"
    return sum(r["status"] == 0 for r in ref)


# --------------------------------------------------------------- cost tables
def _check_tables(problem, planner, cfg_sample):
    t = binding.decode_tables(problem, planner.tables())
    dbg = planner.debug()
    DL = binding.debug_layout(problem)
    o = orc.Oracle(problem)
    cfgs = o.configs()
    N, T = problem["model"]["n_layers"], problem["cluster"]["n_types"]
    micro0 = problem["space"]["micro"][0]
    for k in cfg_sample:
        cfg = cfgs[k]
        pi = t["pi"][k]
        assert int(pi["status"]) == 0
        pt = o.pi_terms(cfg)
        assert int(pi["x_bytes"]) == pt["x_bytes"] and int(pi["tbar"]) == pt["tbar"]
        for h in range(T):
            for g in range(T):
                assert int(pi["p2p"][h * 4 + g]) == o.p2p(cfg, h, g)
        d = dbg[k * DL["per_cfg"]:(k + 1) * DL["per_cfg"]]
        mem = t["mem"][k]
        for layer in range(N):
            mt = o.mem_terms(cfg, layer)
            assert [int(mem[f, layer + 1] - mem[f, layer]) for f in range(3)] == \
                   [mt["q_w"], mt["q_a0"], mt["q_a1"]]
            assert int(mem[3, layer + 1] - mem[3, layer]) == int(problem["model"]["is_moe"][layer])
            for v, ref in ((d[DL["off_mem"] + 2 * layer], mt["w"]), (d[DL["off_mem"] + 2 * layer + 1], mt["a0"])):
                assert abs(v - ref) <= 1e-12 * abs(ref)
            for h in range(T):
                tt = o.type_terms(cfg, layer, h)
                for j, f in enumerate(("comp", "expert")):
                    v = d[DL["off_type"] + (layer * T + h) * 2 + j]
                    assert abs(v - tt[f]) <= 1e-12 * abs(tt[f]), (k, layer, h, f)
        used = int(pi["used_masks"])
        masks = [m for m in range(1, 2 ** T) if (used >> (m - 1)) & 1]
        for m in masks:
            tm = t["time"][k, m - 1]
            for layer in range(N):
                mt = o.mask_terms(cfg, layer, m)
                got = [int(tm[f, layer + 1] - tm[f, layer]) for f in range(3)]
                assert got == [mt["t_r0"], mt["t_r1"], mt["comm"]], (k, m, layer)
                for j, f in enumerate(("a2a", "tp", "cp")):
                    v = d[DL["off_mask"] + ((m - 1) * N + layer) * 3 + j]
                    assert abs(v - mt[f]) <= 1e-12 * abs(mt[f]), (k, m, layer, f)
        free = problem["space"].get("stage_types", 0)
        for oi in range(o.n_orders()):
            key = t["key"][k, oi]
            if free and o.sequence(cfg[0], oi) is None:   # an empty slot: nothing can fit
                assert int(key["dp_const"]) == 0 and not key["hi"][:cfg[0]].any()
                continue
            st = o.stages(cfg, oi, micro0)
            assert int(key["dp_const"]) == o.dp_const(cfg, oi)
            for s, x in enumerate(st):
                assert (int(key["mask"][s]), int(key["lo"][s]), int(key["hi"][s])) == (x["mask"], x["lo"], x["hi"])
                if s + 1 < len(st):
                    assert int(key["bpair"][s]) == (x["last_type"] << 2) | st[s + 1]["first_type"]
                assert (used >> (x["mask"] - 1)) & 1


@pytest.mark.parametrize("which", ["w1", "w2", "cfg1", "cfg2", "cfg3", "cfg4", "cfg5", "tiny"])
def test_cost_tables_match_oracle(torch, which):
    if which == "w1":
        probs = [worked_problem()]
    elif which == "w2":
        probs = [worked_problem_w2()]
    elif which == "tiny":
        probs = [workloads.random_tiny(s) for s in range(12)]
    else:
        probs = [workloads.config(int(which[-1]))]
    for p in probs:
        print(f"cost tables: {p['name']}", flush=True)
        pl = binding.Planner(p, "cuda:0", debug=True)
        pl.eval_cost_tables()
        ncfg = pl.n_configs
        n_sample = 24 if which == "cfg4" else 60   # the 96-layer model: 24 configurations
        sample = range(ncfg) if ncfg <= 200 else sorted(set(np.linspace(0, ncfg - 1, n_sample).astype(int)))
        _check_tables(p, pl, sample)


def test_cost_tables_sub_ranges_equal_one_call(torch):
    """hapmoe_eval_cost_tables over candidate sub-ranges (boundaries inside
    configurations, one empty range) fills the same buffer as one call."""
    p = workloads.config(3)
    pl = binding.Planner(p, "cuda:0", debug=True)
    pl.d_tables.zero_()
    pl.d_debug.zero_()
    pl.eval_cost_tables()
    whole, whole_dbg = pl.tables().copy(), pl.debug().copy()
    pl.d_tables.zero_()
    pl.d_debug.zero_()
    cuts = [0, 1, pl.n // 7 + 5, pl.n // 7 + 5, pl.n // 2 + 3, pl.n - 1, pl.n]
    for a, b in zip(cuts[:-1], cuts[1:]):
        pl.eval_cost_tables(first=a, count=b - a)
    assert np.array_equal(pl.tables(), whole)
    assert np.array_equal(pl.debug().view(np.int64), whole_dbg.view(np.int64))
    with pytest.raises(binding.HapmoeError) as e:
        pl.eval_cost_tables(first=pl.n - 1, count=2)
    assert e.value.code == -7


# ----------------------------------------------------------------- stage DP
def test_worked_example_w2_on_gpu(torch):
    """The hand-worked straddling-stage problem: both orderings' objectives."""
    from tests.problems import load_golden
    g = load_golden("worked_w2.json")["instances"]
    p = worked_problem_w2()
    pl = binding.Planner(p, "cuda:0")
    pl.run()
    res = pl.results()
    for key, idx in (("idx10", 10), ("idx11", 11)):
        r = res[idx]
        assert (int(r["objective"]), int(r["stage_sum"]), int(r["t_max"]), list(r["layers"][:4])) == \
               (g[key]["opt"], g[key]["sum"], g[key]["tmax"], g[key]["layers"])
        assert [(int(r["recompute_mask"]) >> s) & 1 for s in range(4)] == g[key]["recompute"]
    compare(p, pl, range(pl.n))


def test_worked_example_on_gpu(torch):
    p = worked_problem()
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run()
    res = pl.results()
    assert int(res[88]["objective"]) == 2030366 and int(res[89]["objective"]) == 1316910
    compare(p, pl, range(pl.n))
    assert plan["objective"] == min(int(r["objective"]) for r in res)


@pytest.mark.parametrize("n", [1, 2])
def test_small_configs_every_candidate(torch, n):
    p = workloads.config(n)
    print(f"config {n}: all candidates", flush=True)
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run()
    feas = compare(p, pl, range(pl.n))
    assert feas > 0
    res = pl.results()
    obj = np.where(res["status"] == 0, res["objective"], np.iinfo(np.int64).max)
    assert plan["instance"] == int(np.argmin(obj)) and plan["objective"] == int(obj.min())
    # per-configuration segmented minimum
    per = pl.n // pl.n_configs
    cb = pl.config_best()
    for k in range(pl.n_configs):
        seg = obj[k * per:(k + 1) * per]
        exp = -1 if seg.min() == np.iinfo(np.int64).max else k * per + int(np.argmin(seg))
        assert cb[k] == exp


def test_config1_literal_mode(torch):
    p = workloads.config(1, mode=1)
    pl = binding.Planner(p, "cuda:0")
    pl.run()
    compare(p, pl, range(pl.n))


@pytest.mark.parametrize("n,scale,stride", [(2, 0.35, 1), (3, 0.5, 97)])
def test_tight_memory_many_micro_counts(torch, n, scale, stride):
    """Memory binds at many stored micro-batch counts and B runs over 1..32, so
    the micro-batch groups of a key split into several classes of identical
    feasible windows (and merge inside each): every result must still be the
    oracle's."""
    p = workloads.config(n)
    p = variant(p, **{"cluster.mem_bytes": (p["cluster"]["mem_bytes"] * scale).astype(np.int64),
                      "space.micro": np.arange(1, 33, dtype=np.int32)})
    print(f"config {n}: memory x{scale}, B = 1..32, stride {stride}", flush=True)
    pl = binding.Planner(p, "cuda:0")
    pl.eval_cost_tables()
    pl.stage_dp()
    idx = list(range(0, pl.n, stride)) + [pl.n - 1]
    assert compare(p, pl, sorted(set(idx))) > 0


def _uniform_layers(problem):
    """Every layer a copy of layer 0: stage costs become multiples of one layer's
    cost, so equal objectives (ties in sum + (B-1) max) are everywhere."""
    q = variant(problem)
    m, c = q["model"], q["cluster"]
    for key in ("is_moe", "params_dense", "params_expert", "act_bytes"):
        m[key][:] = m[key][0]
    m["expert_tokens"][:] = m["expert_tokens"][0]
    for key in ("t_dense", "t_ffn"):
        c[key][...] = c[key][..., :1]
    return q


@pytest.mark.parametrize("n,micro", [(1, None), (2, list(range(1, 17)))])
def test_tied_objectives_every_candidate(torch, n, micro):
    p = _uniform_layers(workloads.config(n))
    if micro is not None:
        p["space"]["micro"] = np.array(micro, dtype=np.int32)
    print(f"config {n}: uniform layers", flush=True)
    pl = binding.Planner(p, "cuda:0")
    pl.eval_cost_tables()
    pl.stage_dp()
    assert compare(p, pl, range(pl.n)) > 0


def test_random_tiny_every_candidate(torch):
    total = 0
    for s in range(40):
        p = workloads.random_tiny(s)
        pl = binding.Planner(p, "cuda:0")
        pl.eval_cost_tables()
        pl.stage_dp()
        total += compare(p, pl, range(pl.n))
    assert total > 100


def _seven_sets(seed):
    """Four device types of 3, 4, 4 and 3 devices: the 2-device stages of the
    7-stage pipelines straddle every type boundary, so a key uses 7 device-type
    sets (4 single-type, 3 mixed) -- more than the kernel loads ahead."""
    p = copy.deepcopy(workloads.random_tiny(seed, n_layers=10, n_types=4, max_pp=8))
    p["cluster"]["count"] = np.array([3, 4, 4, 3], dtype=np.int32)
    p["name"] = f"seven-sets-{seed}"
    return p


def test_seven_device_type_sets_every_candidate(torch):
    total = 0
    for s in range(3):
        p = _seven_sets(s)
        print(p["name"], flush=True)
        o = orc.Oracle(p)
        assert max(len({st["mask"] for st in o.stages(c, od, 1)})
                   for c in o.configs() for od in range(o.n_orders())) == 7
        pl = binding.Planner(p, "cuda:0")
        pl.eval_cost_tables()
        pl.stage_dp()
        total += compare(p, pl, range(pl.n))
        pl.stage_dp(objective="1f1b")
        compare(p, pl, range(pl.n), objective="1f1b")
    assert total > 50


def test_subranges_and_repeat_are_identical(torch):
    p = workloads.config(2)
    pl = binding.Planner(p, "cuda:0")
    pl.eval_cost_tables()
    pl.stage_dp()
    full = pl.results().copy()
    pl.d_res.fill_(0)
    step = 1777   # ragged chunks
    for first in range(0, pl.n, step):
        pl.stage_dp(first=first, count=min(step, pl.n - first))
    assert np.array_equal(full.view(np.uint8), pl.results().view(np.uint8))


def test_stats_count_passes(torch):
    p = workloads.config(2)
    pl = binding.Planner(p, "cuda:0")
    pl.eval_cost_tables()
    pl.stage_dp(stats=True)
    st = pl.stats()
    res = pl.results()
    ok = res["status"] == 0
    assert st.shape == (pl.n, 4)
    assert (st[ok, 0] >= 1).all() and (st[~ok, 0] <= 1).all()
    assert (st[:, 1] >= 0).all() and st[ok, 1].sum() > 0 and st[:, 2].sum() > 0
    # lane slots of the relaxation loops bound the relaxations, group by group
    assert (st[:, 3] >= st[:, 1]).all() and st[:, 3].sum() > st[:, 1].sum()
    # shared sweeps are counted once per (pi, ordering, min(B, PP)) group
    per_key = len(p["space"]["micro"])
    assert (st[:, 1].reshape(-1, per_key) > 0).sum(axis=1).max() <= per_key


def test_all_infeasible_reports_infeasible(torch):
    p = variant(workloads.config(1), **{"cluster.mem_bytes": np.array([10**6, 10**6], dtype=np.int64)})
    pl = binding.Planner(p, "cuda:0")
    with pytest.raises(binding.HapmoeError) as e:
        pl.run()
    assert e.value.code == -6
    res = pl.results()
    assert (res["status"] == 1).all()


def test_degenerate_shapes(torch):
    # N = PP (one layer per stage), B = 1, dense model, single device type
    for s in range(6):
        p = workloads.random_tiny(100 + s, n_layers=4, max_pp=4, micro=[1, 5],
                                  flags={"prune_window": 0, "prune_hetero": 0, "allow_recompute": 1})
        pl = binding.Planner(p, "cuda:0")
        pl.eval_cost_tables()
        pl.stage_dp()
        compare(p, pl, range(pl.n))
    p = workloads.random_tiny(7, n_types=1)
    p["model"]["n_experts"] = 0
    p["model"]["is_moe"][:] = 0
    p["model"]["expert_tokens"] = np.zeros((p["model"]["n_layers"], 0), dtype=np.int64)
    p["model"]["params_expert"][:] = 0
    pl = binding.Planner(p, "cuda:0")
    pl.eval_cost_tables()
    pl.stage_dp()
    compare(p, pl, range(pl.n))


def test_config4_full_launch_sampled(torch):
    """The bench workload (3.86 M candidates, one launch): sampled parity + properties."""
    p = workloads.config(4)
    print("config 4: full launch, stride sample", flush=True)
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run()
    res = pl.results()
    ok = res["status"] == 0
    N = p["model"]["n_layers"]
    cand = pl.cand_host
    sums = res["layers"].astype(np.int64).sum(axis=1)
    assert (sums[ok] == N).all()
    pp = cand["pp"]
    assert all((res["layers"][ok][:, :] > 0).sum(axis=1) == pp[ok])
    obj = np.where(ok, res["objective"], np.iinfo(np.int64).max)
    assert plan["instance"] == int(np.argmin(obj))
    # a stride sample (every pipeline depth, ordering and B) plus the first and
    # last candidate of each depth and the winner
    idx = list(range(11, pl.n, 3967)) + [plan["instance"]]
    for d in np.unique(pp):
        at = np.nonzero(pp == d)[0]
        idx += [int(at[0]), int(at[-1])]
    compare(p, pl, sorted(set(idx)), res)
    # the per-configuration minima agree with the results
    per = pl.n // pl.n_configs
    cb = pl.config_best()
    seg = obj.reshape(pl.n_configs, per)
    exp = np.where(seg.min(axis=1) == np.iinfo(np.int64).max, -1,
                   np.arange(pl.n_configs) * per + seg.argmin(axis=1))
    assert (cb == exp).all()


# ------------------------------------------------- 1F1B re-scoring objective
@pytest.mark.parametrize("n", [1, 2])
def test_1f1b_small_configs_every_candidate(torch, n):
    p = workloads.config(n)
    print(f"1f1b config {n}: all candidates", flush=True)
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run(objective="1f1b")
    assert compare(p, pl, range(pl.n), objective="1f1b") > 0
    res = pl.results()
    obj = np.where(res["status"] == 0, res["objective"], np.iinfo(np.int64).max)
    assert plan["instance"] == int(np.argmin(obj)) and plan["objective"] == int(obj.min())


def test_1f1b_random_and_tied_every_candidate(torch):
    probs = [workloads.random_tiny(s) for s in range(20)]
    probs += [_uniform_layers(workloads.config(1))]
    q = _uniform_layers(workloads.config(2))
    q["space"]["micro"] = np.arange(1, 17, dtype=np.int32)
    probs.append(q)
    total = 0
    for p in probs:
        print(f"1f1b {p.get('name', '')}", flush=True)
        pl = binding.Planner(p, "cuda:0")
        pl.eval_cost_tables()
        pl.stage_dp(objective="1f1b")
        total += compare(p, pl, range(pl.n), objective="1f1b")
    assert total > 100


@pytest.mark.parametrize("n,gbs", [(1, 16), (4, 2048)])
def test_fixed_global_batch_arg_min(torch, n, gbs):
    """With the training batch fixed at gbs sequences, the arg-min takes only the
    candidates with B * DP * mbs = gbs (per configuration and global); the stage
    DP results do not change."""
    p = workloads.config(n)
    pl = binding.Planner(p, "cuda:0")
    pl.run()
    free = pl.results().copy()
    q = variant(p, **{"space.global_batch": gbs})
    ql = binding.Planner(q, "cuda:0")
    plan = ql.run()
    res = ql.results()
    assert np.array_equal(res, free)
    c = ql.cand_host
    keep = (res["status"] == 0) & (c["n_micro"].astype(np.int64) * c["dp"] * p["model"]["micro_batch_size"] == gbs)
    assert keep.any()
    obj = np.where(keep, res["objective"], np.iinfo(np.int64).max)
    assert plan["instance"] == int(np.argmin(obj)) and plan["objective"] == int(obj.min())
    assert plan["n_micro"] * plan["config"][3] * p["model"]["micro_batch_size"] == gbs
    per = ql.n // ql.n_configs
    seg = obj.reshape(ql.n_configs, per)
    exp = np.where(seg.min(axis=1) == np.iinfo(np.int64).max, -1, np.arange(ql.n_configs) * per + seg.argmin(axis=1))
    assert (ql.config_best() == exp).all()
    if n == 1:   # the oracle's own minimum over the same subset
        o = orc.Oracle(p)
        ref = [o.solve(i) for i in range(o.n_instances())]
        best = min((r["opt"], i) for i, r in enumerate(ref) if r["status"] == 0 and keep[i])
        assert (plan["objective"], plan["instance"]) == best


def test_1f1b_feasibility_equals_threshold_objective(torch):
    """Both objectives search the same feasible partitions: the same candidates
    are feasible (the bench launch, 3.86 M candidates)."""
    pl = binding.Planner(workloads.config(4), "cuda:0")
    pl.eval_cost_tables()
    pl.stage_dp(objective="1f1b")
    st = pl.results()["status"].copy()
    pl.stage_dp()
    assert np.array_equal(pl.results()["status"], st)


# ------------------------------------------ uniform layers (ablation windows)
@pytest.mark.parametrize("n,stride", [(2, 1), (3, 53)])
def test_uniform_layers(torch, n, stride):
    p = variant(workloads.config(n), **{"params.prune_window": 2})
    print(f"uniform layers config {n}: stride {stride}", flush=True)
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run()
    idx = list(range(0, pl.n, stride)) + [pl.n - 1, plan["instance"]]
    assert compare(p, pl, sorted(set(idx))) > 0
    pl.stage_dp(objective="1f1b")
    compare(p, pl, sorted(set(idx))[::7], objective="1f1b")


def test_best_plan_launcher_text(torch):
    from paper_2609_39350_amd import launcher
    p = workloads.config(1)
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run()
    text = launcher.plan_to_launcher(p, plan)
    assert f"--pipeline-model-parallel-size {plan['config'][0]}" in text
    assert 'PIPELINE_STAGE_LAYERS="' + ",".join(str(n) for n in plan["layers"]) + '"' in text


# ------------------------------------- no pruning windows on the large models
@pytest.mark.parametrize("n", [4, 5])
def test_no_windows_large_configs_sampled(torch, n):
    """Pruning-1 windows off: every stage may take 1 .. N - PP + 1 layers, so the
    split ranges reach their widest (65 split points a stage on the 96-layer
    model at PP = 32) and the sweep keeps one chain per class. Both objectives on
    a sample of the deepest pipelines (the only feasible ones) plus a stride
    sample of all candidates."""
    p = variant(workloads.config(n), **{"params.prune_window": 0})
    print(f"config {n}: no windows", flush=True)
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run()
    res = pl.results()
    pp = pl.cand_host["pp"]
    deep = np.nonzero(pp == pp.max())[0]
    idx = sorted(set(deep[::max(1, len(deep) // 48)].tolist() + list(range(5, pl.n, pl.n // 97))
                     + [plan["instance"]]))
    assert compare(p, pl, idx, res, ref=oracle_many(p, idx, pool=True)) > 0
    obj = np.where(res["status"] == 0, res["objective"], np.iinfo(np.int64).max)
    assert plan["instance"] == int(np.argmin(obj))
    pl.stage_dp(objective="1f1b")
    sub = deep[::max(1, len(deep) // 24)].tolist()
    assert compare(p, pl, sub, objective="1f1b", ref=oracle_many(p, sub, "1f1b", pool=True)) > 0
