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
