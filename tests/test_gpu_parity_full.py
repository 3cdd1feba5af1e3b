"""GPU results against stored oracle references on the large workloads, through
the C ABI (needs an MI355X).

tests/golden/parity_refs.npz holds 32-bit digests (tests/parity_digest.py) of
the oracle's results, written by tests/golden/make_parity_refs.py from oracle/
alone: configurations 3 and 5 in full under both objectives, configuration 4
with one candidate of every (configuration, ordering) key (B rotating over
1..64) and one of every configuration under the 1F1B re-scoring, and 16
sixteen-stage candidates and every candidate of up to 8 stages of configuration
3 and twelve 4- and 8-stage ones of configuration 4 under the device-count DP,
and
stride samples of configurations 3, 4 and 5 and every candidate of
configurations 3 and 5 under the least 1F1B latency.  A digest
covers status, objective, stage sum, largest stage, recomputation mask, stage
lengths (and stage types); a mismatch is re-checked against the oracle itself
and reported field by field.
"""
import copy
import os

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2609_39350_amd import binding, workloads
from tests import parity_digest

pytestmark = pytest.mark.gpu

REFS = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "parity_refs.npz")


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


@pytest.fixture(scope="module")
def refs():
    with np.load(REFS) as f:
        return {k: f[k] for k in f.files}


def _explain(problem, res, idx, objective, types=None):
    """Field-by-field differences of a few mismatching candidates."""
    o = orc.Oracle(problem)
    out = []
    for i in idx[:3]:
        r = {"threshold": o.solve, "1f1b": o.solve_exact, "latency": o.solve_latency}[objective](int(i))
        g = res[int(i)]
        out.append((int(i), {"gpu": (int(g["status"]), int(g["objective"]), int(g["stage_sum"]), int(g["t_max"]),
                                     list(g["layers"][:r["pp"]])),
                             "oracle": (r["status"], r["opt"], r["sum"], r["tmax"], r["layers"])}))
    return out


def _check(problem, res, refs, key, objective, types=None):
    idx = refs[key + "_idx"]
    got = parity_digest.of_gpu(res, idx, types)
    bad = np.nonzero(got != refs[key])[0]
    assert len(bad) == 0, f"{key}: {len(bad)} of {len(idx)} differ: {_explain(problem, res, idx[bad], objective)}"
    return len(idx)


@pytest.mark.parametrize("n", [3, 5])
@pytest.mark.parametrize("objective", ["threshold", "1f1b"])
def test_every_candidate(torch, refs, n, objective):
    p = workloads.config(n)
    print(f"config {n}, {objective}: every candidate against the stored oracle results", flush=True)
    pl = binding.Planner(p, "cuda:0")
    plan = pl.run(objective=objective)
    res = pl.results()
    assert _check(p, res, refs, f"cfg{n}_{objective}", objective) == pl.n
    obj = np.where(res["status"] == 0, res["objective"], np.iinfo(np.int64).max)
    assert plan["instance"] == int(np.argmin(obj)) and plan["objective"] == int(obj.min())


@pytest.mark.parametrize("objective", ["threshold", "1f1b"])
def test_config4_every_key(torch, refs, objective):
    """The bench launch (3.86 M candidates): one candidate of every (configuration,
    ordering) key, B rotating over 1..64 (the 1F1B re-scoring: one of every
    configuration)."""
    p = workloads.config(4)
    print(f"config 4, {objective}: one candidate a key", flush=True)
    pl = binding.Planner(p, "cuda:0")
    pl.run(objective=objective)
    res = pl.results()
    assert _check(p, res, refs, f"cfg4_{objective}", objective) >= 2510


def test_device_count_dp_sixteen_stages(torch, refs):
    p = copy.deepcopy(workloads.config(3))
    p["space"]["stage_types"] = 2
    print("config 3, device-count DP: sixteen-stage candidates", flush=True)
    pl = binding.Planner(p, "cuda:0")
    pl.run()
    res, types = pl.results(), pl.stage_types()
    idx = refs["cfg3_types16_idx"]
    assert (pl.cand_host["pp"][idx] == 16).all() and len(idx) >= 16
    got = parity_digest.of_gpu(res, idx, types)
    assert np.array_equal(got, refs["cfg3_types16"]), np.nonzero(got != refs["cfg3_types16"])[0]
    assert (res["status"][idx] == 0).any()


@pytest.mark.parametrize("n", [3, 5, 4])
def test_least_latency_samples(torch, refs, n):
    """The least 1F1B latency (hapmoe_stage_dp_latency) on every 97th candidate
    of configurations 3 and 5 and one candidate of every 6th configuration of
    configuration 4, each from a one-candidate launch."""
    p = workloads.config(n)
    print(f"config {n}, least latency: stride sample", flush=True)
    pl = binding.Planner(p, "cuda:0")
    pl.eval_cost_tables()
    idx = refs[f"cfg{n}_latency_idx"]
    for i in idx:
        pl.stage_dp(first=int(i), count=1, objective="latency")
    res = pl.results()
    assert _check(p, res, refs, f"cfg{n}_latency", "latency") == len(idx)
    assert (res["status"][idx] == 0).sum() > 10


@pytest.mark.parametrize("n", [3, 5])
def test_least_latency_every_candidate(torch, refs, n):
    """The least 1F1B latency on every candidate of configurations 3 and 5 (one
    launch over the whole workload, as the bench runs it), against stored oracle
    digests; skipped if the references were written without them."""
    if f"cfg{n}_latency_all" not in refs:
        pytest.skip("no full least-latency references in parity_refs.npz")
    p = workloads.config(n)
    print(f"config {n}, least latency: every candidate", flush=True)
    pl = binding.Planner(p, "cuda:0")
    pl.eval_cost_tables()
    pl.stage_dp(objective="latency")
    res = pl.results()
    assert _check(p, res, refs, f"cfg{n}_latency_all", "latency") == pl.n


def test_device_count_dp_shallow_every_candidate(torch, refs):
    """The device-count DP on every candidate of configuration 3 with at most 8
    stages (one launch over the whole workload), stage types included, against
    stored oracle digests; skipped if the references were written without them."""
    if "cfg3_types_shallow" not in refs:
        pytest.skip("no shallow device-count references in parity_refs.npz")
    p = copy.deepcopy(workloads.config(3))
    p["space"]["stage_types"] = 2
    print("config 3, device-count DP: every candidate of up to 8 stages", flush=True)
    pl = binding.Planner(p, "cuda:0")
    pl.run()
    res, types = pl.results(), pl.stage_types()
    idx = refs["cfg3_types_shallow_idx"]
    assert (pl.cand_host["pp"][idx] <= 8).all() and len(idx) > 1000
    got = parity_digest.of_gpu(res, idx, types)
    bad = np.nonzero(got != refs["cfg3_types_shallow"])[0]
    assert len(bad) == 0, f"{len(bad)} of {len(idx)} differ, first: {idx[bad][:5]}"
    assert (res["status"][idx] == 0).sum() > 100


def test_device_count_dp_config4_samples(torch, refs):
    """The device-count DP on the 96-layer workload (96,128 candidates, pipelines
    up to 32 stages, one launch): twelve 4- and 8-stage candidates against the
    stored oracle results, stage types included (the oracle's sweep takes hours
    a candidate at 16 or 32 stages; those are checked by the properties of
    tests/test_gpu_free_types.py)."""
    p = copy.deepcopy(workloads.config(4))
    p["space"]["stage_types"] = 2
    print("config 4, device-count DP: 4- and 8-stage samples", flush=True)
    pl = binding.Planner(p, "cuda:0")
    pl.run()
    res, types = pl.results(), pl.stage_types()
    idx = refs["cfg4_types_idx"]
    assert set(pl.cand_host["pp"][idx]) == {4, 8} and len(idx) == 12
    got = parity_digest.of_gpu(res, idx, types)
    assert np.array_equal(got, refs["cfg4_types"]), np.nonzero(got != refs["cfg4_types"])[0]
    assert (res["status"][idx] == 0).sum() >= 6
