#!/usr/bin/env python3
"""Planner hot-path benchmark on one MI355X.

One step = the whole hot path over the candidate set of the workload:
cost-table kernel -> stage-DP kernel -> segmented arg-min (best plan), with
the problem image and candidate array already resident in HBM.  The metric is
candidates evaluated per second.  Each kernel is timed with HIP events on the
stream it runs on; the stage-DP kernel (the dominant one) is reported against
the VALU issue roofline of the chip.  The CPU oracle is timed on a bounded
stride sample of the same workload (single core) as a reported baseline.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 4]
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "candidate plans evaluated/sec (cost model + stage DP), % HBM/VALU roofline"

# MI355X: 256 CUs x 4 SIMD x 16 lanes at 2.4 GHz -> 32-bit VALU lane operations per second
VALU_PEAK_OPS = 256 * 64 * 2.4e9
# one DP relaxation = 3 int64 operations (stage cost <= threshold, F + c, compare with the
# running minimum) = 6 32-bit lane operations; one split-point evaluation of the feasibility
# scan = 3 int64 operations (weights + stored activations x count, + MoE buffers, compare
# with the capacity) = 6 32-bit lane operations
OPS_PER_RELAXATION = 6
OPS_PER_EVALUATION = 6

WORKLOADS = {
    1: "tiny: 8-layer MoE (H1024, E8 top-2, S2048), 4+4 devices of 2 types, B=8",
    2: "32-layer MoE (H4096, E64 top-8, S4096), 64 devices 32/16/16 of 3 types, B in {8,16,32}",
    3: "61-layer MoE (3 dense, H7168, E256 top-8, 1 shared, S4096), 4x64 devices of 4 types, B in {16,32,64}",
    4: "96-layer MoE (H8192, E128 top-4, S8192, CP<=8), 4x256 devices of 4 types, 24 orderings, B=1..64",
    5: "adversarial: 61-layer shape, +-1% near-tied layer costs, tight memory, Zipf s=2",
}


# training batch (sequences) for the fixed-batch arg-min of each workload: B * DP * mbs
GLOBAL_BATCH = {1: 16, 2: 256, 3: 1024, 4: 2048, 5: 1024}

TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "stage_dp_moe96_traffic.json")
STAGE_DP_SOURCE = os.path.join(ROOT, "paper_2609_39350_amd", "csrc", "stage_dp.hip")


def kernel_code_sha256(path=STAGE_DP_SOURCE):
    """SHA-256 of a kernel source with its // comments and blank lines removed
    (the kernel source has no string literal holding //)."""
    lines = []
    with open(path) as f:
        for line in f:
            code = line.split("//", 1)[0].rstrip()
            if code:
                lines.append(code)
    return hashlib.sha256("\n".join(lines).encode()).hexdigest()


def measured_traffic(config):
    """HBM bytes per stage-DP launch from the committed counter record, or None
    when the record is for another workload or the kernel code has changed
    since the counters were taken."""
    try:
        with open(TRAFFIC_RECORD) as f:
            rec = json.load(f)
        sha = kernel_code_sha256()
    except OSError:
        return None
    if rec.get("config") != config or rec.get("kernel_sha256") != sha:
        return None
    return rec.get("hbm_bytes_per_launch")


def copy_calibration(torch, dev, nbytes=1 << 30, reps=3):
    """A plain device-to-device copy of known size, for scaling the FETCH_SIZE /
    WRITE_SIZE counters (run under rocprofv3 --pmc next to the kernels)."""
    src = torch.ones(nbytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    return nbytes


def leg_uniform(binding, problem, pl, dev):
    """Ablation analogue (non-uniform layer assignment disabled): the same
    candidates with every stage holding floor/ceil(N/PP) layers; best objective
    of each, globally and at the largest micro-batch count."""
    import copy
    import numpy as np
    pu_problem = copy.deepcopy(problem)
    pu_problem["params"]["prune_window"] = 2
    pu = binding.Planner(pu_problem, dev)
    out = {}
    micro = np.asarray(problem["space"]["micro"])
    bmax = int(micro.max())
    big = np.iinfo(np.int64).max
    for name, planner in (("non_uniform", pl), ("uniform", pu)):
        planner.eval_cost_tables()
        planner.stage_dp()
        res = planner.results()
        obj = np.where(res["status"] == 0, res["objective"], big)
        at_bmax = obj[planner.cand_host["n_micro"] == bmax]
        out[name] = {"best_ns": int(obj.min()) if obj.min() < big else None,
                     f"best_at_B{bmax}_ns": int(at_bmax.min()) if at_bmax.min() < big else None,
                     "feasible": int((res["status"] == 0).sum())}
    nu, un = out["non_uniform"], out["uniform"]
    for key, name in (("best_ns", "latency_increase"), (f"best_at_B{bmax}_ns", f"latency_increase_at_B{bmax}")):
        out[name] = un[key] / nu[key] - 1.0 if un[key] and nu[key] else None
    return out


def leg_1f1b(torch, pl, stream, steps, warmup):
    """The same step with the stage DP re-scoring the (max, sum) frontier by the
    appendix's 1F1B latency (hapmoe_stage_dp_1f1b), timed after the main metric."""
    import numpy as np
    pl.eval_cost_tables()
    pl.stage_dp(stats=True, objective="1f1b")
    st = pl.stats()
    relax = int(st[:, 1].astype(np.int64).sum())
    for _ in range(warmup):
        pl.run(objective="1f1b")
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    t0 = time.perf_counter()
    plan = None
    for k in range(steps):
        pl.eval_cost_tables()
        ev[k][0].record(stream)
        pl.stage_dp(objective="1f1b")
        ev[k][1].record(stream)
        plan = pl.best_plan()
        ev[k][2].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    dp_ms = float(np.mean([ev[k][0].elapsed_time(ev[k][1]) for k in range(steps)]))
    return {"value": pl.n * steps / elapsed, "unit": "candidates/s", "ms_per_step": elapsed * 1e3 / steps,
            "stage_dp_ms": dp_ms, "relaxations_per_launch": relax,
            "roofline": alu_roofline(relax, int(st[:, 2].astype(np.int64).sum()), dp_ms, "stage_dp (1F1B)"),
            "dp_passes_per_candidate": {"mean": float(st[:, 0].mean()), "max": int(st[:, 0].max())},
            "best_plan": {"instance": plan["instance"], "objective_ns": plan["objective"],
                          "config": plan["config"], "order": plan["order"], "B": plan["n_micro"],
                          "layers": plan["layers"]}}


def leg_latency(torch, binding, workloads, dev, stream, cpu_sample):
    """The least 1F1B latency over every partition (hapmoe_stage_dp_latency) on
    configurations 2, 3 and 4, whole launches, with the frontier re-scoring's
    best plan beside it (the exact minimum can only be lower)."""
    import numpy as np
    out = {}
    for n_config in (2, 3, 4):   # configuration 4: about 8 s a launch
        p = workloads.config(n_config)
        pl = binding.Planner(p, dev)
        pl.eval_cost_tables()
        pl.stage_dp(stats=True, objective="latency")   # statistics, and warm
        st = pl.stats()
        res = pl.results()
        ok = res["status"] == 0
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        pl.stage_dp(objective="latency")
        e1.record(stream)
        plan = pl.best_plan()
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        ms = e0.elapsed_time(e1)
        relax = int(st[:, 1].astype(np.int64).sum())
        plan_f = pl.run(objective="1f1b")
        rec = {"workload": f"config {n_config}: {WORKLOADS[n_config]}", "candidates": pl.n,
               "value": pl.n / elapsed, "unit": "candidates/s", "stage_dp_ms": ms,
               "feasible_candidates": int(ok.sum()),
               "thresholds_per_candidate": {"mean": float(st[ok, 0].mean()) if ok.any() else 0.0,
                                            "max": int(st[:, 0].max())},
               "relaxations_per_launch": relax,
               "roofline": alu_roofline(relax, 0, ms, "latency_dp"),
               "best_objective_ns": plan["objective"], "frontier_rescoring_best_ns": plan_f["objective"],
               "best_plan": {"config": plan["config"], "order": plan["order"], "B": plan["n_micro"],
                             "layers": plan["layers"], "recompute": plan["recompute"]}}
        if cpu_sample and n_config == 2:
            from oracle.oracle import Oracle
            o = Oracle(p)
            stride = max(1, pl.n // cpu_sample)
            idx = list(range(stride // 2, pl.n, stride))[:cpu_sample]
            t0 = time.perf_counter()
            o.solve_latency_many(idx)
            dt = time.perf_counter() - t0
            rec["cpu_baseline"] = {"value": len(idx) / dt, "unit": "candidates/s", "cores": 1, "kind": "oracle",
                                   "host": host_cpu(),
                                   "sample": f"{len(idx)} candidates at stride {stride} of {pl.n}, {dt:.1f} s "
                                             f"on one host core"}
        out[f"config{n_config}"] = rec
        progress(f"least latency config {n_config}")
    return out


FP64_PEAK_FLOPS = 78.6e12            # MI355X vector fp64
HBM_PEAK_BYTES = 8.0e12
COST_FLOPS_PER_ENTRY = 40            # fp64 operations per (configuration, type set, layer) entry
ARGMIN_BYTES_PER_CANDIDATE = 16      # objective + status read per candidate


def side_rooflines(binding, pl, ms):
    """Kernel 1 (cost tables): bytes written against HBM and fp64 work against
    the fp64 peak; kernel 3 (arg-min): bytes read against HBM (its time is the
    whole hapmoe_best_plan call, plan read-back included)."""
    import numpy as np
    t = binding.decode_tables(pl.problem, pl.tables())
    L = t["layout"]
    used = np.array([bin(int(u)).count("1") for u in t["pi"]["used_masks"]], dtype=np.int64)
    N = pl.problem["model"]["n_layers"]
    entries = int(used.sum()) * N
    written = (L["n_configs"] * 152 + L["n_configs"] * L["n_orders"] * 136 + L["n_configs"] * 4 * (N + 1) * 8
               + int(used.sum()) * 3 * (N + 1) * 8)
    ct_s, bp_s = ms["cost_tables"] / 1e3, ms["best_plan"] / 1e3
    return {
        "cost_tables": {"bound": "hbm", "achieved": written / ct_s / 1e9, "peak": HBM_PEAK_BYTES / 1e9,
                        "unit": "GB/s", "frac": written / ct_s / HBM_PEAK_BYTES, "bytes_written": written,
                        "fp64_achieved_tflops": entries * COST_FLOPS_PER_ENTRY / ct_s / 1e12,
                        "fp64_frac": entries * COST_FLOPS_PER_ENTRY / ct_s / FP64_PEAK_FLOPS,
                        "entries": entries, "flops_per_entry": COST_FLOPS_PER_ENTRY},
        "best_plan": {"bound": "hbm", "achieved": pl.n * ARGMIN_BYTES_PER_CANDIDATE / bp_s / 1e9,
                      "peak": HBM_PEAK_BYTES / 1e9, "unit": "GB/s",
                      "frac": pl.n * ARGMIN_BYTES_PER_CANDIDATE / bp_s / HBM_PEAK_BYTES,
                      "bytes_per_candidate": ARGMIN_BYTES_PER_CANDIDATE},
    }


def alu_roofline(relaxations, evaluations, ms, kernel):
    """VALU roofline of one stage-DP launch from its algorithmic operation count."""
    ops = relaxations * OPS_PER_RELAXATION + evaluations * OPS_PER_EVALUATION
    achieved = ops / (ms / 1e3) if ms > 0 else 0.0
    return {"bound": "alu", "achieved": achieved / 1e12, "peak": VALU_PEAK_OPS / 1e12, "unit": "TOP/s",
            "frac": achieved / VALU_PEAK_OPS, "kernel": kernel, "relaxations_per_launch": relaxations,
            "evaluations_per_launch": evaluations}


def _timed_steps(torch, pl, stream, steps, warmup):
    """Whole steps (tables, stage DP, arg-min) and the stage-DP events of each."""
    import numpy as np
    for _ in range(warmup):
        pl.run()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
    t0 = time.perf_counter()
    plan = None
    for k in range(steps):
        pl.eval_cost_tables()
        ev[k][0].record(stream)
        pl.stage_dp()
        ev[k][1].record(stream)
        plan = pl.best_plan()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    return plan, elapsed, float(np.mean([ev[k][0].elapsed_time(ev[k][1]) for k in range(steps)]))


def leg_free_types(torch, binding, workloads, dev, stream, steps, warmup, cpu_sample):
    """Free per-stage device types: every stage-type sequence as its own candidate
    (config 2), and the DP over device counts (configs 2 and 3, pipelines up to
    16 stages, and config 4, up to 32 stages and 9^4 count states); each with the
    best objective of the block orderings beside it."""
    import copy
    import numpy as np
    out = {}
    for name, n_config, mode in (("sequences", 2, 1), ("device_count_dp", 2, 2), ("device_count_dp", 3, 2),
                                 ("device_count_dp", 4, 2)):
        base = workloads.config(n_config)
        free = copy.deepcopy(base)
        free["space"]["stage_types"] = mode
        block_best = binding.Planner(base, dev).run()["objective"]
        pf = binding.Planner(free, dev)
        pf.eval_cost_tables()
        pf.stage_dp(stats=True)
        st = pf.stats()
        # the 96-layer count DP runs about 2.4 s a launch: one timed launch after
        # the statistics launch (which also warms it)
        k_steps, k_warm = (1, 0) if n_config == 4 and mode == 2 else (steps, warmup)
        plan, elapsed, dp_ms = _timed_steps(torch, pf, stream, k_steps, k_warm)
        res = pf.results()
        rec = {"workload": f"config {n_config}: {WORKLOADS[n_config]}, every stage one device type",
               "value": pf.n * k_steps / elapsed, "unit": "candidates/s", "ms_per_step": elapsed * 1e3 / k_steps,
               "steps": k_steps,
               "stage_dp_ms": dp_ms, "candidates": pf.n,
               "feasible_candidates": int((res["status"] == 0).sum()),
               "dp_passes_per_candidate": {"mean": float(st[:, 0].mean()), "max": int(st[:, 0].max())},
               "relaxations_per_launch": int(st[:, 1].astype(np.int64).sum()),
               "roofline": alu_roofline(int(st[:, 1].astype(np.int64).sum()), int(st[:, 2].astype(np.int64).sum()),
                                        dp_ms, "stage_dp" if mode == 1 else "type_dp"),
               "best_objective_ns": plan["objective"], "block_orderings_best_ns": block_best,
               "gain_over_block_orderings": 1.0 - plan["objective"] / block_best,
               "best_plan": {"config": plan["config"], "order": plan["order"], "B": plan["n_micro"],
                             "stage_types": plan["stage_types"], "layers": plan["layers"]}}
        if mode == 1:
            # every configuration has the same number of order slots (the largest
            # arrangement count); a pipeline's own stage-type sequences fill the
            # first PP! / prod_h k_h! of them, the rest are padding that the cost
            # tables mark infeasible without DP work
            from math import factorial
            counts = [int(x) for x in free["cluster"]["count"]]
            G = sum(counts)
            real = 0
            for pp in pf.cand_host["pp"][::int(binding.tables_layout(free)["n_orders"]) * len(free["space"]["micro"])]:
                g = G // int(pp)
                arr = factorial(int(pp))
                for m in counts:
                    arr //= factorial(m // g)
                real += arr * len(free["space"]["micro"])
            rec["sequences_per_config"] = int(binding.tables_layout(free)["n_orders"])
            rec["real_sequence_candidates"] = real
            rec["padding_candidates"] = pf.n - real
            rec["value_real_sequences"] = real * k_steps / elapsed
        if mode == 2:   # the 1F1B re-scoring of the same DP (hapmoe_stage_dp_types_1f1b)
            if k_warm:
                pf.stage_dp(objective="1f1b")
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(k_steps):
                pf.stage_dp(objective="1f1b")
            e1.record(stream)
            plan_1f1b = pf.best_plan()
            rec["objective_1f1b"] = {"stage_dp_ms": e0.elapsed_time(e1) / k_steps,
                                     "best_objective_ns": plan_1f1b["objective"],
                                     "stage_types": plan_1f1b["stage_types"], "layers": plan_1f1b["layers"]}
        if mode == 2 and n_config == 2 and cpu_sample:
            rec["cpu_baseline"], _ = cpu_baseline(free, pf.n, cpu_sample)
        out[f"{name}_config{n_config}"] = rec
        progress(f"{name} config {n_config}")
    return out


def per_depth(torch, binding, pl, stream, reps=5, clocks=False):
    """Diagnostic: the stage-DP kernel on each pipeline depth's candidates alone
    (a sub-range launch each), with its executed relaxations and split-point
    evaluations and its fraction of the VALU roofline (clocks: the diagnostic
    build's section clocks of each depth's launches)."""
    import numpy as np
    pp = pl.cand_host["pp"]
    rows = []
    for d in np.unique(pp):
        at = np.nonzero(pp == d)[0]
        first, count = int(at[0]), int(len(at))
        pl.stage_dp(first=first, count=count, stats=True)
        st = pl.stats()[first:first + count]
        relax, evals = int(st[:, 1].astype(np.int64).sum()), int(st[:, 2].astype(np.int64).sum())
        slots = int(st[:, 3].astype(np.int64).sum())
        torch.cuda.synchronize()
        if clocks:
            binding.section_clocks(clear=True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            pl.stage_dp(first=first, count=count)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        roof = alu_roofline(relax, evals, ms, "stage_dp")
        row = {"pp": int(d), "candidates": count, "ms": ms, "relaxations": relax, "evaluations": evals,
               "lane_utilisation": relax / max(slots, 1),
               "passes_per_candidate": float(st[:, 0].mean()), "frac": roof["frac"]}
        if clocks:
            row["section_clocks"] = binding.section_clocks(clear=True)
        rows.append(row)
    return rows


def host_cpu():
    """Host cores and CPU model, for the CPU-baseline record."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = os.cpu_count()
    return {"nproc": usable, "cpu_count": os.cpu_count(), "cpu_model": model}


def leg_widths(torch, binding, workloads, dev, stream, steps, warmup, cpu_sample):
    """Per-stage data-parallel widths (non-uniform PP/DP, hapmoe_stage_dp_widths)
    on the 32- and 61-layer workloads: the same candidates' best objective with
    uniform widths beside it."""
    import copy
    import numpy as np
    out = {}
    for n_config in (2, 3):
        base = workloads.config(n_config)
        wp = copy.deepcopy(base)
        wp["space"]["stage_types"] = 3
        pw = binding.Planner(wp, dev)
        pw.eval_cost_tables()
        pw.stage_dp(stats=True)
        st = pw.stats()
        plan, elapsed, dp_ms = _timed_steps(torch, pw, stream, steps, warmup)
        res = pw.results()
        # the uniform plan of the same candidates (block layout, same configurations)
        pu = binding.Planner(base, dev)
        pu.run()
        ures = pu.results()
        keep = {tuple(c) for c in np.stack([pw.cand_host[f] for f in ("pp", "tp", "cp", "dp", "ep", "tpe")], 1)}
        ukey = [tuple(c) in keep for c in np.stack([pu.cand_host[f] for f in ("pp", "tp", "cp", "dp", "ep", "tpe")], 1)]
        uobj = np.where(ures["status"] == 0, ures["objective"], np.iinfo(np.int64).max)[np.array(ukey)]
        relax = int(st[:, 1].astype(np.int64).sum())
        rec = {"workload": f"config {n_config}: {WORKLOADS[n_config]}, per-stage data-parallel widths",
               "value": pw.n * steps / elapsed, "unit": "candidates/s", "ms_per_step": elapsed * 1e3 / steps,
               "stage_dp_ms": dp_ms, "candidates": pw.n, "feasible_candidates": int((res["status"] == 0).sum()),
               "dp_passes_per_candidate": {"mean": float(st[:, 0].mean()), "max": int(st[:, 0].max())},
               "relaxations_per_launch": relax,
               "roofline": alu_roofline(relax, 0, dp_ms, "width_dp"),
               "best_objective_ns": plan["objective"], "uniform_widths_best_ns": int(uobj.min()),
               "gain_over_uniform_widths": 1.0 - plan["objective"] / int(uobj.min()),
               "best_plan": {"config": plan["config"], "order": plan["order"], "B": plan["n_micro"],
                             "widths": plan["widths"], "layers": plan["layers"]}}
        if n_config == 2 and cpu_sample:
            rec["cpu_baseline"], _ = cpu_baseline(wp, pw.n, cpu_sample)
        out[f"config{n_config}"] = rec
    return out


def cpu_baseline(problem, n_total, n_sample, exact=False):
    """The oracle as it stands, single thread, on a fixed stride sample (exact:
    its 1F1B re-scoring of the frontier)."""
    from oracle.oracle import Oracle
    o = Oracle(problem)
    stride = max(1, n_total // n_sample)
    idx = list(range(stride // 2, n_total, stride))[:n_sample]
    t0 = time.perf_counter()
    res = o.solve_exact_many(idx) if exact else o.solve_many(idx)
    dt = time.perf_counter() - t0
    # the oracle's DP work (threshold objective): every pass relaxes all (stage,
    # a < b) pairs; passes = the unthresholded one, the thresholds it swept, and
    # the pass it back-traces when a partition exists
    W = problem["model"]["n_layers"] + 1
    updates = [(1 + r["thresholds"] + (r["status"] == 0)) * r["pp"] * W * (W - 1) // 2 for r in res]
    out = {"value": len(idx) / dt, "unit": "candidates/s", "cores": 1, "kind": "oracle", "host": host_cpu(),
           "sample": f"{len(idx)} candidates at stride {stride} of {n_total} (every {stride}th), "
                     f"{dt:.1f} s on one host core"}
    return out, sum(updates) / max(len(updates), 1)


_T_START = time.perf_counter()


def progress(what):
    """One line on stderr as each leg ends (the JSON line alone goes to stdout)."""
    print(f"bench: {what} ({time.perf_counter() - _T_START:.1f} s)", file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--cpu-sample", type=int, default=400)
    ap.add_argument("--cpu-sample-1f1b", type=int, default=200)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-1f1b", action="store_true", help="skip the 1F1B re-scoring leg")
    ap.add_argument("--no-free-types", action="store_true", help="skip the free per-stage device-type legs")
    ap.add_argument("--section-clocks", action="store_true",
                    help="diagnostic build: report where the stage-DP kernel's cycles go (slightly slower kernel)")
    ap.add_argument("--cpu-sample-free", type=int, default=40)
    ap.add_argument("--no-widths", action="store_true", help="skip the per-stage data-parallel width legs")
    ap.add_argument("--per-depth", action="store_true",
                    help="diagnostic: stage-DP time, work and roofline fraction of each pipeline depth alone")
    ap.add_argument("--cpu-sample-widths", type=int, default=200)
    ap.add_argument("--no-latency", action="store_true", help="skip the least-latency legs")
    ap.add_argument("--cpu-sample-latency", type=int, default=2000)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a 1 GiB device copy (counter scaling for HBM traffic)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the planner's candidates are independent and are evaluated "
              "on a single device here (there is no multi-GPU path). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_39350_amd import binding, workloads

    if args.section_clocks:
        binding.use_section_clocks()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    problem = workloads.config(args.config)
    pl = binding.Planner(problem, dev)
    n = pl.n
    stream = torch.cuda.current_stream()

    # untimed: relaxation / pass counts of one stage-DP launch (deterministic per launch)
    pl.eval_cost_tables()
    pl.stage_dp(stats=True)
    st = pl.stats()
    relax = int(st[:, 1].astype(np.int64).sum())
    evals = int(st[:, 2].astype(np.int64).sum())
    slots = int(st[:, 3].astype(np.int64).sum())
    passes = st[:, 0]
    feasible = int((pl.results()["status"] == 0).sum())
    progress(f"config {args.config}: {n} candidates, statistics launch done")

    calib = copy_calibration(torch, dev) if args.copy_calibration else None

    for _ in range(args.warmup):
        pl.run()
    torch.cuda.synchronize()
    if args.section_clocks:
        binding.section_clocks(clear=True)

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    plan = None
    for k in range(args.steps):
        e = ev[k]
        e[0].record(stream)
        pl.eval_cost_tables()
        e[1].record(stream)
        pl.stage_dp()
        e[2].record(stream)
        plan = pl.best_plan()        # waits for the stream
        e[3].record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0
    ms = {name: float(np.mean([ev[k][j].elapsed_time(ev[k][j + 1]) for k in range(args.steps)]))
          for j, name in enumerate(("cost_tables", "stage_dp", "best_plan"))}
    progress(f"timed {args.steps} steps")

    clocks = binding.section_clocks(clear=True) if args.section_clocks else None
    if clocks is not None:
        # one launch alone: its longest key and when its waves finish (wall clock)
        pl.stage_dp()
        torch.cuda.synchronize()
        one = binding.section_clocks(clear=True)
        clocks["single_launch_wall"] = {k: one[k] for k in ("longest_key_us", "longest_key_pp",
                                                           "first_wave_done_us", "last_wave_done_us") if k in one}
    dp_s = ms["stage_dp"] / 1e3
    achieved = (relax * OPS_PER_RELAXATION + evals * OPS_PER_EVALUATION) / dp_s
    out = {
        "metric": METRIC,
        "value": n * args.steps / elapsed,
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": f"config {args.config}: {WORKLOADS[args.config]}", "candidates": n,
                   "configs_6d": pl.n_configs, "feasible_candidates": feasible},
        "roofline": {"bound": "alu", "achieved": achieved / 1e12, "peak": VALU_PEAK_OPS / 1e12,
                     "unit": "TOP/s", "frac": achieved / VALU_PEAK_OPS,
                     "traffic": measured_traffic(args.config),
                     "kernel": "stage_dp", "ops_per_relaxation": OPS_PER_RELAXATION,
                     "ops_per_evaluation": OPS_PER_EVALUATION,
                     "relaxations_per_launch": relax, "evaluations_per_launch": evals},
        "kernels_ms": ms,
        "dp_cell_updates_per_s": relax / dp_s,
        "relaxation_lane_utilisation": relax / max(slots, 1),
        "threshold_passes_per_candidate": {"mean": float(passes.mean()), "max": int(passes.max())},
        "best_plan": {"instance": plan["instance"], "objective_ns": plan["objective"],
                      "config": plan["config"], "order": plan["order"], "B": plan["n_micro"],
                      "layers": plan["layers"], "recompute": plan["recompute"]},
    }
    out["side_rooflines"] = side_rooflines(binding, pl, ms)
    if args.per_depth:
        out["stage_dp_per_depth"] = per_depth(torch, binding, pl, stream, clocks=args.section_clocks)
        progress("per-depth launches")
    # the same results with the training batch fixed (B * DP * mbs = global batch):
    # the arg-min over candidates that do the same work
    gbs = GLOBAL_BATCH.get(args.config)
    if gbs:
        import copy
        fixed = copy.deepcopy(problem)
        fixed["space"]["global_batch"] = gbs
        fp = binding.best_plan(binding.HostProblem(fixed), pl.d_cand, pl.d_tables, pl.d_res, pl.n, pl.d_ws)
        out["best_plan_fixed_global_batch"] = {
            "global_batch_sequences": gbs, "instance": fp["instance"], "objective_ns": fp["objective"],
            "config": fp["config"], "order": fp["order"], "B": fp["n_micro"], "layers": fp["layers"],
            "recompute": fp["recompute"]}
    if clocks is not None:
        clocks["steps"] = args.steps
        out["stage_dp_section_clocks"] = clocks
    out["ablation_uniform_layers"] = leg_uniform(binding, problem, pl, dev)
    progress("uniform-layer ablation")
    if not args.no_1f1b:
        out["objective_1f1b"] = leg_1f1b(torch, pl, stream, args.steps, args.warmup)
        if not args.no_cpu_baseline:
            out["objective_1f1b"]["cpu_baseline"], _ = cpu_baseline(problem, n, args.cpu_sample_1f1b, exact=True)
        progress("1F1B re-scoring leg")
    if not args.no_free_types:
        out["free_stage_types"] = leg_free_types(torch, binding, workloads, dev, stream, args.steps, args.warmup,
                                                 0 if args.no_cpu_baseline else args.cpu_sample_free)
        progress("free stage-type legs")
    if not args.no_latency:
        out["least_latency"] = leg_latency(torch, binding, workloads, dev, stream,
                                           0 if args.no_cpu_baseline else args.cpu_sample_latency)
    if not args.no_widths:
        out["per_stage_widths"] = leg_widths(torch, binding, workloads, dev, stream, args.steps, args.warmup,
                                             0 if args.no_cpu_baseline else args.cpu_sample_widths)
        progress("per-stage width legs")
    if calib is not None:
        out["copy_calibration_bytes"] = calib
    if not args.no_cpu_baseline:
        out["cpu_baseline"], oracle_updates = cpu_baseline(problem, n, args.cpu_sample)
        # DP cell updates the oracle's plain sweep would do for the whole launch,
        # estimated from the sample, against the stage-DP time: pruning and sharing
        # gains are visible next to the executed figure above
        out["oracle_equivalent_dp_updates_per_s"] = oracle_updates * n / dp_s
        progress("CPU baseline")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
