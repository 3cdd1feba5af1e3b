"""C-ABI checks that need no GPU: the library loads, exports every declared
symbol, validates its input and enumerates the same candidate set as the
oracle (host-only calls)."""
import os
import re

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2609_39350_amd import binding, workloads
from tests.problems import variant, worked_problem

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "hapmoe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(hapmoe_\w+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    names = _declared()
    assert len(names) >= 12
    L = binding.lib()
    for n in names:
        assert hasattr(L, n), n


def test_strerror_names_every_code():
    for code in range(-7, 1):
        assert binding.lib().hapmoe_strerror(code).decode() not in ("", "unknown status")


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5])
def test_enumeration_matches_oracle(n):
    p = workloads.config(n)
    cand = binding.enumerate_candidates(p)
    o = orc.Oracle(p)
    assert len(cand) == o.n_instances()
    cfgs = o.configs()
    per = o.n_orders() * len(p["space"]["micro"])
    got = np.stack([cand[f] for f in ("pp", "tp", "cp", "dp", "ep", "tpe")], axis=1)[::per]
    assert [tuple(int(v) for v in r) for r in got] == cfgs
    # ordering and B fields follow the documented index formula
    k = np.arange(len(cand))
    assert np.array_equal(cand["order"], (k // len(p["space"]["micro"])) % o.n_orders())
    assert np.array_equal(cand["n_micro"], np.array(p["space"]["micro"])[k % len(p["space"]["micro"])])


def test_enumeration_random_and_literal_mode():
    for s in range(30):
        p = workloads.random_tiny(s)
        cand = binding.enumerate_candidates(p)
        assert len(cand) == orc.Oracle(p).n_instances()
    assert len(binding.enumerate_candidates(workloads.config(1, mode=1))) == 110


def test_validation_rejects_bad_input():
    base = worked_problem()
    bad = [
        {"model.n_layers": 0},
        {"model.top_k": 9},
        {"cluster.t_ffn": base["cluster"]["t_dense"] + 1},
        {"params.rc_time": 0.5},
        {"params.gamma": 1.5},
        {"params.delta_num": 5},
        {"space.pp_max": 33},
        {"space.micro": [0]},
        {"space.micro": [2000]},
        {"cluster.bw": np.zeros((2, 2))},
        {"model.is_moe": np.array([2, 1], dtype=np.uint8)},
        {"params.prune_window": 3},
        {"params.prune_window": -1},
    ]
    for ch in bad:
        with pytest.raises(binding.HapmoeError) as e:
            binding.validate(variant(base, **ch))
        assert e.value.code == -1, ch
    binding.validate(base)
    binding.validate(variant(base, **{"params.prune_window": 2}))


def test_capacity_and_sizes():
    p = workloads.config(2)
    hp = binding.HostProblem(p)
    import ctypes as C
    n = C.c_int64(0)
    assert binding.lib().hapmoe_enumerate_candidates(hp.ref, None, 0, C.byref(n)) == -2
    assert n.value == 16272
    small = np.zeros(10, dtype=binding.CANDIDATE_DTYPE)
    assert binding.lib().hapmoe_enumerate_candidates(hp.ref, small.ctypes.data, 10, C.byref(n)) == -2
    assert n.value == 16272 and small["pp"][0] == 1
    L = binding.tables_layout(p)
    assert L["n_configs"] == 904 and L["n_orders"] == 6 and L["n_masks"] == 7 and L["np"] >= 33
    assert binding.tables_bytes(p) == L["total"]
    img = binding.pack_image(p)
    assert img.nbytes == binding.image_bytes(p)


def test_device_calls_refuse_bad_sizes_before_touching_the_gpu():
    # argument checks run before any HIP call: wrong candidate count is rejected
    p = worked_problem()
    hp = binding.HostProblem(p)
    f = binding.lib().hapmoe_stage_dp
    assert f(hp.ref, 1, 1, 5, 1, 10**9, 0, 1, 1, None, 1, 256, None) == -1
    assert f(hp.ref, 1, 1, 90, 1, 10**9, 80, 20, 1, None, 1, 256, None) == -7
    assert f(hp.ref, 1, 1, 90, 1, 10, 0, 1, 1, None, 1, 256, None) == -3
    assert f(hp.ref, 1, 1, 90, 1, 10**9, 0, 1, 1, None, 1, 8, None) == -3
    assert f(hp.ref, 1, 1, 90, 1, 10**9, 0, 1, 1, None, None, 256, None) == -1


def test_least_latency_entry_checks_before_the_gpu():
    """hapmoe_stage_dp_latency validates its arguments before any HIP call:
    range, table size and the modes it does not cover."""
    import ctypes as C
    p = workloads.config(1)
    hp = binding.HostProblem(p)
    n = len(binding.enumerate_candidates(p))
    fake = C.c_void_p(1 << 20)   # never dereferenced: every call below returns before device work
    tb = binding.tables_bytes(p)
    f = binding.lib().hapmoe_stage_dp_latency
    assert f(hp.ref, fake, fake, n, fake, tb, n - 5, 6, fake, None, None) == -7
    assert f(hp.ref, fake, fake, n, fake, tb, -1, 1, fake, None, None) == -7
    assert f(hp.ref, fake, fake, n, fake, tb - 1, 0, 1, fake, None, None) == -3
    assert f(hp.ref, fake, fake, n + 1, fake, tb, 0, 1, fake, None, None) == -1
    assert f(hp.ref, fake, fake, n, fake, tb, 0, 1, None, None, None) == -1
    for mode in (2, 3):
        q = variant(p, **{"space.stage_types": mode})
        hq = binding.HostProblem(q)
        assert f(hq.ref, fake, fake, 0, fake, 1 << 40, 0, 0, fake, None, None) == -1
    assert f(hp.ref, fake, fake, n, fake, tb, 0, 1, fake, None, None) in (-4, -5)   # no usable device here


def test_free_stage_types_enumeration_and_limits():
    # free per-stage types: the same candidate set as the oracle, and sequence
    # counts past the library's limit refused up front
    for p in (workloads.config(1), workloads.config(2), workloads.random_tiny(5, n_types=3)):
        q = variant(p, **{"space.stage_types": 1})
        o = orc.Oracle(q)
        cand = binding.enumerate_candidates(q)
        assert len(cand) == o.n_instances()
        per = o.n_orders() * len(q["space"]["micro"])
        got = np.stack([cand[f] for f in ("pp", "tp", "cp", "dp", "ep", "tpe")], axis=1)[::per]
        assert [tuple(int(v) for v in r) for r in got] == o.configs()
        assert binding.tables_layout(q)["n_orders"] == o.n_orders()
    q = variant(workloads.config(2), **{"space.stage_types": 1})
    assert binding.tables_layout(q)["n_orders"] == 420   # 8! / (4! 2! 2!)
    for bad in (4, -1):
        with pytest.raises(binding.HapmoeError):
            binding.validate(variant(q, **{"space.stage_types": bad}))
    # 4 types x 64 devices at PP = 16: 16! / (4!)^4 sequences
    huge = variant(workloads.config(3), **{"space.stage_types": 1})
    with pytest.raises(binding.HapmoeError):
        binding.validate(huge)
    binding.validate(variant(huge, **{"space.pp_max": 8}))
    # no configuration left: 5 + 3 devices never fill whole groups of 2, 4 or 8
    empty = variant(workloads.random_tiny(900, n_types=2), **{"space.stage_types": 1})
    assert list(empty["cluster"]["count"]) == [5, 3] and orc.Oracle(empty).n_instances() == 0
    with pytest.raises(binding.HapmoeError):
        binding.validate(empty)


def test_device_count_dp_space_and_limits():
    # stage_types = 2: one order slot per configuration, the same configurations
    # as the sequence mode, its own workspace query, and the state limit
    import ctypes as C
    for p in (workloads.config(2), workloads.random_tiny(901, n_types=3)):
        q = variant(p, **{"space.stage_types": 2})
        o = orc.Oracle(q)
        cand = binding.enumerate_candidates(q)
        assert len(cand) == o.n_instances() == len(o.configs()) * len(q["space"]["micro"])
        assert (cand["order"] == 0).all()
        assert binding.tables_layout(q)["n_orders"] == 1
        assert binding.stage_dp_types_ws_bytes(q) > 256
        with pytest.raises(binding.HapmoeError):
            binding.stage_dp_types_ws_bytes(variant(q, **{"space.stage_types": 1}))
        hp = binding.HostProblem(q)
        n = C.c_int64(0)
        # the fixed-type stage DP refuses the mode (before any device work)
        assert binding.lib().hapmoe_stage_dp(hp.ref, None, None, 0, None, 0, 0, 0, None, None, None, 0,
                                             None) == -1
    # 4 types x 64 devices at PP = 16: 5^4 count states; a 4 x 256-device cluster
    # at PP = 32 has 9^4 = 6561, inside the 8192 limit (the most four types allow
    # at 32 stages)
    binding.validate(variant(workloads.config(3), **{"space.stage_types": 2}))
    binding.validate(variant(workloads.config(4), **{"space.stage_types": 2}))
    with pytest.raises(binding.HapmoeError):
        binding.validate(variant(workloads.config(3), **{"space.stage_types": 4}))


def test_noalloc_best_plan_rejects_problems_beyond_its_workspace():
    """hapmoe_best_plan_noalloc refuses, before any device work, a problem whose
    arg-min needs more than its fixed workspace; one that fits passes the size
    check and stops only at the device check (no GPU here)."""
    import copy
    import ctypes as C
    big = copy.deepcopy(workloads.config(4))
    big["space"]["stage_types"] = 1   # 880 configurations x 2,520 stage-type sequences x 64 B values
    big["space"]["pp_max"] = 8
    small = workloads.config(2)
    assert binding.best_plan_ws_bytes(big, 1) > binding.BEST_PLAN_SCRATCH_BYTES
    assert binding.best_plan_ws_bytes(small, 1) <= binding.BEST_PLAN_SCRATCH_BYTES
    fake = C.c_void_p(1 << 20)   # never dereferenced: both calls return before device work
    codes = []
    for p in (big, small):
        hp = binding.HostProblem(p)
        plan = binding.Plan()
        codes.append(binding.lib().hapmoe_best_plan_noalloc(hp.ref, fake, fake, binding.tables_bytes(hp), fake,
                                                            None, 1, None, C.byref(plan), None))
    assert codes[0] == -3                 # HAPMOE_E_WORKSPACE
    assert codes[1] in (-4, -5)           # past the size check: no usable device here


@pytest.mark.parametrize("n,n_candidates", [(1, 290), (2, 16272), (3, 117792), (4, 3855360), (5, 117792)])
def test_library_enumeration_pinned_counts(n, n_candidates):
    p = workloads.config(n)
    assert binding.tables_layout(p)["n_configs"] * binding.tables_layout(p)["n_orders"] * \
        len(p["space"]["micro"]) == n_candidates
    if n_candidates <= 200000:
        assert len(binding.enumerate_candidates(p)) == n_candidates
