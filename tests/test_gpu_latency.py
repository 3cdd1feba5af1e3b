"""The least 1F1B latency on the GPU (hapmoe_stage_dp_latency) against the
oracle's exact minimum (Appendix B, Eq. 5 with Eq. 4's steady-state term; the
oracle's DP over thresholds is itself pinned to brute force over every
composition on the CPU).

The bar (integer/index work): bit-exact status, objective, stage sum, largest
stage, partition and recomputation choice for every compared candidate.
"""
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
    global _POOL
    if _POOL is None:
        _POOL = mp.get_context("spawn").Pool(max(1, min(16, os.cpu_count() or 1)))
    return _POOL


def oracle_latency(problem, idx):
    idx = [int(i) for i in idx]
    if len(idx) < 64:
        return orc.Oracle(problem).solve_latency_many(idx)
    n = _pool()._processes
    parts = [idx[k::n] for k in range(n)]
    outs = _pool().map(orc.solve_worker, [(problem, part, "latency") for part in parts])
    res = [None] * len(idx)
    for k, out in enumerate(outs):
        for j, r in enumerate(out):
            res[k + j * n] = r
    return res


@pytest.fixture(scope="module", autouse=True)
def _close_pool():
    yield
    global _POOL
    if _POOL is not None:
        _POOL.terminate()
        _POOL.join()
        _POOL = None


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def run_latency(problem, first=0, count=None, stats=False):
    pl = binding.Planner(problem, "cuda:0")
    pl.eval_cost_tables()
    pl.stage_dp(first=first, count=count, stats=stats, objective="latency")
    return pl, pl.results()


def compare(problem, res, idx):
    ref = oracle_latency(problem, idx)
    bad = []
    for i, r in zip(idx, ref):
        g = res[int(i)]
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


def _small():
    out = [("w1", worked_problem()), ("w2", worked_problem_w2()), ("config1", workloads.config(1))]
    out += [(f"tiny{s}", workloads.random_tiny(s)) for s in range(40)]
    out += [("config1_sequences", variant(workloads.config(1), **{"space.stage_types": 1})),
            ("tiny17_sequences", variant(workloads.random_tiny(17, n_types=3), **{"space.stage_types": 1})),
            ("tiny2_sequences", variant(workloads.random_tiny(2, n_types=3), **{"space.stage_types": 1})),
            ("w1_no_recompute", variant(worked_problem(), **{"params.allow_recompute": 0})),
            ("w2_eta1", variant(worked_problem_w2(), **{"params.eta_prune": 1}))]
    return out


@pytest.mark.parametrize("name,problem", _small(), ids=[n for n, _ in _small()])
def test_latency_every_candidate_small(torch, name, problem):
    print(f"least latency: {name}", flush=True)
    pl, res = run_latency(problem)
    compare(problem, res, range(pl.n))


def test_latency_config2_every_candidate(torch):
    p = workloads.config(2)
    print("least latency: config 2, every candidate", flush=True)
    pl, res = run_latency(p)
    assert compare(p, res, range(pl.n)) > 1000


def test_latency_sub_range_and_stats(torch):
    """A launch over [first, first + count) writes exactly that range, with the
    results of the whole launch; the statistics count thresholds swept."""
    p = workloads.config(2)
    pl, whole = run_latency(p)
    whole = whole.copy()
    first, count = 5003, 2111
    pl.d_res.fill_(0x5A)
    pl.stage_dp(first=first, count=count, stats=True, objective="latency")
    part = pl.results()
    assert np.array_equal(part[first:first + count], whole[first:first + count])
    raw = part.view(np.uint8).reshape(len(part), -1)
    assert (raw[:first] == 0x5A).all() and (raw[first + count:] == 0x5A).all()
    st = pl.stats()[first:first + count]
    ok = whole[first:first + count]["status"] == 0
    assert (st[ok, 0] >= 1).all() and (st[~ok, 0] == 0).all() and (st[:, 1] >= 0).all()
    # relaxations are counted once per shared sweep: on the first candidate of
    # each (key, group) -- with B in {8, 16, 32} and PP <= 8, B = 16 and 32 share
    assert st[ok, 1].sum() > 0 and (st[ok, 1] > 0).sum() < ok.sum()


def test_latency_lower_bound_of_the_frontier_rescoring(torch):
    """Every partition the frontier re-scoring may choose is one the exact
    minimum ranges over: the least latency is never above it, and both find a
    partition for exactly the same candidates (config 3, every candidate)."""
    p = workloads.config(3)
    pl = binding.Planner(p, "cuda:0")
    pl.eval_cost_tables()
    pl.stage_dp(objective="1f1b")
    f1b = pl.results().copy()
    pl.stage_dp(objective="latency")
    lat = pl.results()
    assert np.array_equal(f1b["status"] == 0, lat["status"] == 0)
    ok = lat["status"] == 0
    assert ok.sum() > 1000
    assert (lat["objective"][ok] <= f1b["objective"][ok]).all()
    # the latency of the chosen partition is at least its stage sum plus the
    # bottleneck's forward part plus the steady-state term at the last stage
    # (C, the constant of Eq. 4, read off the threshold DP's result)
    pl.stage_dp()
    thr = pl.results()
    B = pl.cand_host["n_micro"].astype(np.int64)
    PP = pl.cand_host["pp"].astype(np.int64)
    const = thr["objective"] - thr["stage_sum"] - (B - 1) * thr["t_max"]
    t = lat["t_max"]
    low = lat["stage_sum"] + (t + 2) // 3 + np.maximum(0, B - PP - 1) * t + const
    assert (lat["objective"][ok] >= low[ok]).all()
    gap = (f1b["objective"][ok] - lat["objective"][ok]) / f1b["objective"][ok]
    print(f"config 3: re-scoring above the least latency on {(gap > 0).mean():.3f} of the feasible "
          f"candidates, by {gap.max():.4f} at most", flush=True)


LDS_SMALL_BYTES = 22784    # first launch: 24 KB less the kernel's 1,792-byte header
LDS_TABLE_BYTES = 162048   # last launch: 160 KB less the header


def table_bytes(problem, o):
    """Per (configuration, ordering) key: pipeline depth and the bytes of the
    kernel's stage-cost table, from the oracle's stage windows."""
    N = int(problem["model"]["n_layers"])
    out = {}
    for ci, cfg in enumerate(o.configs()):
        for od in range(o.n_orders()):
            st = o.stages(cfg, od, problem["space"]["micro"][0])
            lo = [s["lo"] for s in st]
            hi = [s["hi"] for s in st]
            cl, ch = np.cumsum(lo), np.cumsum(hi)
            ncost = nv = 0
            for s in range(len(st)):
                blo, bhi = max(cl[s], N - (ch[-1] - ch[s])), min(ch[s], N - (cl[-1] - cl[s]))
                wd = max(0, bhi - blo + 1)
                ncost += wd * (hi[s] - lo[s] + 1)
                nv += wd
            out[ci * o.n_orders() + od] = (len(st), 8 * ncost + 16 * nv + 16 * ((ncost + 15) // 16))
    return out


def test_latency_oversized_table_reports_overflow(torch):
    """Tables too big for the first launch's 24 KB workgroups go to the later
    launches (up to 160 KB) with the same results; a candidate whose table
    exceeds that too gets HAPMOE_STATUS_OVERFLOW, not a wrong answer.  127 layers, windows
    opened to delta = 0.999 and memory that always fits: the one-stage pipelines
    fit the first launch, the two-stage ones only a later one, the four-stage
    ones neither."""
    p = workloads.random_tiny(11, n_layers=127, max_pp=4)
    p["params"]["delta_num"], p["params"]["delta_den"] = 999, 1000
    p["cluster"]["mem_bytes"] = np.full(p["cluster"]["n_types"], 10**15, dtype=np.int64)
    o = orc.Oracle(p)
    need = table_bytes(p, o)
    nb = len(p["space"]["micro"])
    pl, res = run_latency(p)
    depth = np.array([need[i // nb][0] for i in range(pl.n)])
    size = np.array([need[i // nb][1] for i in range(pl.n)])
    over = size > LDS_TABLE_BYTES
    second = (size > LDS_SMALL_BYTES) & ~over
    assert over.any() and second.any() and (~over & ~second).any()
    assert set(depth[over]) == {4} and set(depth[second]) == {2}
    assert np.array_equal(res["status"] == 2, over)
    assert compare(p, res, np.nonzero(~over)[0]) > 0
