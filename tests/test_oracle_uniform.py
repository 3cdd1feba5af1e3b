"""Uniform layer assignment (the window mode that disables non-uniform
partitions, as in the evaluation's ablation): pins of the oracle."""
import numpy as np

from oracle import oracle as orc
from paper_2609_39350_amd import workloads
from tests.problems import variant


def test_uniform_windows_force_the_uniform_partition():
    # N = 32 and PP in {1, 2, 4, 8}: the only partition left has N / PP layers a stage
    p = variant(workloads.config(2), **{"params.prune_window": 2})
    o = orc.Oracle(p)
    N = p["model"]["n_layers"]
    seen = set()
    for i in range(0, o.n_instances(), 97):
        r = o.solve(i)
        if r["status"] == 0:
            assert r["layers"] == [N // r["pp"]] * r["pp"], (i, r)
            seen.add(r["pp"])
        st = o.stages(o.configs()[i // (o.n_orders() * len(p["space"]["micro"]))], 0,
                      p["space"]["micro"][0])
        assert all(x["lo"] == x["hi"] == N // len(st) for x in st)
    assert len(seen) >= 3


def test_uniform_windows_ragged_and_bounds():
    # N not a multiple of PP: every stage holds floor or ceil of N / PP layers; the
    # optimum over all partitions (no windows) is never worse than the uniform one
    checked = 0
    for s in range(8):
        p = workloads.random_tiny(500 + s, n_layers=7 + s % 3, max_pp=4)
        pu = variant(p, **{"params.prune_window": 2})
        pa = variant(p, **{"params.prune_window": 0})
        ou, oa = orc.Oracle(pu), orc.Oracle(pa)
        N = p["model"]["n_layers"]
        for i in range(ou.n_instances()):
            ru, ra = ou.solve(i), oa.solve(i)
            if ru["status"] != 0:
                continue
            pp = ru["pp"]
            assert sum(ru["layers"]) == N and all(N // pp <= n <= -(-N // pp) for n in ru["layers"])
            assert ra["status"] == 0 and ra["opt"] <= ru["opt"]
            # brute force over the same windows agrees
            rb = ou.solve_brute(i)
            assert (rb["opt"], rb["layers"]) == (ru["opt"], ru["layers"])
            checked += 1
    assert checked > 50
