"""Free per-stage device types on the GPU (every stage one group of a single
type, the order index walking the distinct stage-type sequences): tables,
both objectives and the best plan against the oracle, through the C ABI."""
import numpy as np
import pytest

from oracle import oracle as orc
from paper_2609_39350_amd import binding, workloads
from tests.problems import variant
from tests.test_gpu_parity import _check_tables, compare, torch  # noqa: F401  (fixture)

pytestmark = pytest.mark.gpu


def free(p):
    return variant(p, **{"space.stage_types": 1})


@pytest.mark.parametrize("n", [1, 2])
def test_free_types_tables(torch, n):
    p = free(workloads.config(n))
    print(f"free types, config {n}: tables", flush=True)
    pl = binding.Planner(p, "cuda:0", debug=True)
    pl.eval_cost_tables()
    assert pl.n_configs == len(orc.Oracle(p).configs())
    sample = range(pl.n_configs) if pl.n_configs <= 60 else \
        sorted(set(np.linspace(0, pl.n_configs - 1, 24).astype(int)))
    _check_tables(p, pl, sample)


@pytest.mark.parametrize("n", [1, 2])
def test_free_types_every_candidate(torch, n):
    p = free(workloads.config(n))
    print(f"free types, config {n}: all candidates", flush=True)
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run()
    feas = compare(p, pl, range(pl.n))
    assert feas > 0
    res = pl.results()
    obj = np.where(res["status"] == 0, res["objective"], np.iinfo(np.int64).max)
    assert plan["instance"] == int(np.argmin(obj)) and plan["objective"] == int(obj.min())
    # the chosen plan's stages are pure and follow the oracle's sequence
    o = orc.Oracle(p)
    seq = o.sequence(plan["config"][0], plan["order"])
    assert plan["stage_types"] == [1 << h for h in seq]


def test_free_types_never_worse_than_pure_block_orderings(torch):
    # a block ordering with pure stages is one of the free sequences
    p = workloads.config(2)
    pb, pf = binding.Planner(p, "cuda:0"), binding.Planner(free(p), "cuda:0")
    pb.run()
    best_f = pf.run()
    counts = [int(x) for x in p["cluster"]["count"]]
    rb = pb.results()
    pure = np.array([all(m % (sum(counts) // int(pp)) == 0 for m in counts) for pp in pb.cand_host["pp"]])
    ob = np.where((rb["status"] == 0) & pure, rb["objective"], np.iinfo(np.int64).max)
    assert best_f["objective"] <= int(ob.min())


@pytest.mark.parametrize("n,stride", [(1, 1), (2, 89)])
def test_free_types_1f1b(torch, n, stride):
    p = free(workloads.config(n))
    print(f"free types, config {n}: 1F1B, stride {stride}", flush=True)
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run(objective="1f1b")
    idx = sorted(set(list(range(0, pl.n, stride)) + [pl.n - 1] + [max(plan["instance"], 0)]))
    compare(p, pl, idx, objective="1f1b")


def test_free_types_random_tiny(torch):
    done = 0
    for s in range(40):
        p = free(workloads.random_tiny(900 + s, n_types=2 + s % 2))
        if orc.Oracle(p).n_instances() == 0:   # no type fills whole groups (refused by the library)
            continue
        done += 1
        pl = binding.Planner(p, "cuda:0")
        pl.eval_cost_tables()
        pl.stage_dp()
        compare(p, pl, range(pl.n))
    assert done >= 10


# ---------------------------------------------------------------------------
# stage_types = 2: the device-count DP (hapmoe_stage_dp_types)
def count_dp(p):
    return variant(p, **{"space.stage_types": 2})


def compare_types(problem, pl, idx, slow=False, objective="threshold"):
    """Every field of compare() plus the stage types the DP chose (slow: the
    oracle takes seconds per candidate, so it runs in worker processes)."""
    from tests.test_gpu_parity import oracle_many
    ref = oracle_many(problem, idx, objective, pool=True if slow else None)
    compare(problem, pl, idx, ref=ref, objective=objective)
    ty = pl.stage_types()
    for i, r in zip(idx, ref):
        got = [int(x) for x in ty[i]]
        if r["status"] == 0:
            assert got[:r["pp"]] == r["stage_mask"] and not any(got[r["pp"]:]), (i, got, r)
        else:
            assert not any(got), i


@pytest.mark.parametrize("n", [1, 2])
def test_count_dp_every_candidate(torch, n):
    p = count_dp(workloads.config(n))
    print(f"device-count DP, config {n}: all candidates", flush=True)
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run()
    compare_types(p, pl, range(pl.n))
    res = pl.results()
    obj = np.where(res["status"] == 0, res["objective"], np.iinfo(np.int64).max)
    assert plan["instance"] == int(np.argmin(obj)) and plan["objective"] == int(obj.min())
    assert plan["stage_types"] == [int(x) for x in pl.stage_types()[plan["instance"]][:len(plan["layers"])]]


def test_count_dp_random_tiny(torch):
    done = 0
    for s in range(40):
        p = count_dp(workloads.random_tiny(900 + s, n_types=2 + s % 2))
        if orc.Oracle(p).n_instances() == 0:
            continue
        done += 1
        pl = binding.Planner(p, "cuda:0")
        pl.eval_cost_tables()
        pl.stage_dp()
        compare_types(p, pl, range(pl.n))
    assert done >= 10


def test_count_dp_config3_sampled(torch):
    # four device types, pipelines of 4 and 8 stages (the oracle takes seconds each)
    p = variant(count_dp(workloads.config(3)), **{"space.pp_max": 8})
    print("device-count DP, config 3 (PP <= 8): sample", flush=True)
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run()
    idx = sorted(set(list(range(pl.n - 1, 0, -(pl.n // 12))) + [plan["instance"]]))
    compare_types(p, pl, idx, slow=True)


@pytest.mark.parametrize("n", [3, 5, 4])
def test_count_dp_full_space_properties(torch, n):
    # PP up to 16 (5^4 count states; on the 96-layer workload up to 32 stages and
    # 9^4 = 6,561 states): every result is a valid plan whose stage costs,
    # evaluated by the oracle, give its sum, largest stage and objective, and no
    # block ordering of the same (pi, B) does better
    base = workloads.config(n)
    p = count_dp(base)
    print(f"device-count DP, config {n}: properties", flush=True)
    pl = binding.Planner(p, "cuda:0")
    pl.run()
    res, ty = pl.results(), pl.stage_types()
    pb = binding.Planner(base, "cuda:0")
    pb.run()
    rb = pb.results()
    nB, no = len(base["space"]["micro"]), 24
    cfg_b = [tuple(int(v) for v in r) for r in
             np.stack([pb.cand_host[f] for f in ("pp", "tp", "cp", "dp", "ep", "tpe")], axis=1)[::no * nB]]
    o = orc.Oracle(p)
    cfgs = o.configs()
    big = np.iinfo(np.int64).max
    feasible = 0
    for ci, cfg in enumerate(cfgs):
        bi = cfg_b.index(cfg)
        for j in range(nB):
            i = ci * nB + j
            block = rb[(bi * no) * nB + j::nB][:no]
            best_block = min([int(r["objective"]) for r in block if r["status"] == 0], default=big)
            if res[i]["status"] != 0:
                assert best_block == big, (cfg, j)
                continue
            feasible += 1
            assert int(res[i]["objective"]) <= best_block, (cfg, j)
    assert feasible > 0
    # a stride sample re-evaluated from the oracle's cost tensor (and every
    # pipeline depth's last candidate)
    pps = pl.cand_host["pp"]
    sample = set(range(0, pl.n, max(1, pl.n // 24))) | {int(np.nonzero(pps == d)[0][-1]) for d in np.unique(pps)}
    for i in sorted(sample):
        if res[i]["status"] != 0:
            continue
        cost, rf = o.type_costs(i)
        pp, B = cfgs[i // nB][0], p["space"]["micro"][i % nB]
        types = [int(m).bit_length() - 1 for m in ty[i][:pp]]
        g = int(sum(base["cluster"]["count"])) // pp
        assert sorted(types) == sorted(h for h in range(4) for _ in range(int(base["cluster"]["count"][h]) // g))
        a, cs, rs = 0, [], []
        for s in range(pp):
            b = a + int(res[i]["layers"][s])
            hn = types[s + 1] if s + 1 < pp else 4
            cs.append(int(cost[s, types[s], hn, a, b]))
            rs.append(int(rf[s, types[s], hn, a, b]))
            a = b
        assert a == p["model"]["n_layers"] and big not in cs
        assert sum(cs) == int(res[i]["stage_sum"]) and max(cs) == int(res[i]["t_max"])
        assert rs == [(int(res[i]["recompute_mask"]) >> s) & 1 for s in range(pp)]
        assert int(res[i]["objective"]) == sum(cs) + (B - 1) * max(cs) + o.dp_const(cfgs[i // nB], 0)


def test_count_dp_subranges_match(torch):
    p = count_dp(workloads.config(2))
    pl = binding.Planner(p, "cuda:0")
    pl.eval_cost_tables()
    pl.stage_dp()
    full, tyf = pl.results().copy(), pl.stage_types().copy()
    pl.d_res.zero_()
    pl.d_types.zero_()
    for first in range(0, pl.n, 100):
        pl.stage_dp(first=first, count=min(100, pl.n - first))
    assert (pl.results() == full).all() and (pl.stage_types() == tyf).all()
    pl.stage_dp(stats=True)
    st = pl.stats()
    assert (st[:, 0] >= 1).all() and st[:, 1].sum() > 0


@pytest.mark.parametrize("n,stride", [(1, 1), (2, 5)])
def test_count_dp_1f1b(torch, n, stride):
    p = count_dp(workloads.config(n))
    print(f"device-count DP, 1F1B, config {n}: stride {stride}", flush=True)
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run(objective="1f1b")
    idx = sorted(set(list(range(0, pl.n, stride)) + [pl.n - 1, plan["instance"]]))
    compare_types(p, pl, idx, slow=True, objective="1f1b")
    res = pl.results()
    obj = np.where(res["status"] == 0, res["objective"], np.iinfo(np.int64).max)
    assert plan["instance"] == int(np.argmin(obj))


def test_count_dp_1f1b_random_tiny(torch):
    done = 0
    for s in range(40):
        p = count_dp(workloads.random_tiny(900 + s, n_types=2 + s % 2))
        if orc.Oracle(p).n_instances() == 0:
            continue
        done += 1
        pl = binding.Planner(p, "cuda:0")
        pl.eval_cost_tables()
        pl.stage_dp(objective="1f1b")
        compare_types(p, pl, range(pl.n), objective="1f1b")
    assert done >= 10


@pytest.mark.parametrize("flags", [{"params.prune_window": 0}, {"params.prune_window": 2},
                                   {"params.allow_recompute": 0, "params.prune_hetero": 0},
                                   {"space.micro": [1, 2, 3, 5, 8, 13]}])
def test_count_dp_flag_variants(torch, flags):
    # no windows (every end layer in the band), uniform windows, no recomputation
    # and no pruning 3, and B below PP (several groups of min(B, PP)): a stride
    # sample of configuration 2 against the oracle
    p = variant(count_dp(workloads.config(2)), **flags)
    print(f"device-count DP, config 2, {flags}", flush=True)
    pl = binding.Planner(p, "cuda:0")
    pl.eval_cost_tables()
    pl.stage_dp()
    idx = sorted(set(list(range(0, pl.n, 13)) + [pl.n - 1]))
    compare_types(p, pl, idx, slow=True)
