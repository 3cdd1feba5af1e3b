"""Seeded synthetic planner inputs.

This module only draws inputs: model layer profiles, per-device-type
compute/memory tables, link matrices and search-space settings, in the shape
that the paper's problem statement gives them (Section 3.1: model parameters
(N, S, H, E, k), hardware inventory {m_h}, memory budgets {C_h}, profiled
bandwidth/collective characteristics; Section 3.3: compute table
t_dense/t_ffn per (TP, CP), communication primitive table, memory
calibration).  It performs none of the planner's own arithmetic (no cost
model, no partitioning, no search): both the HIP library and the CPU oracle
consume the plain dictionaries built here.

The paper's profiled tables and router statistics are not available, so every
table here is synthetic:
  * compute tables are FLOP-derived (configs 2-5) or uniform draws (config 1),
    with per-entry multiplicative jitter;
  * router statistics are a water-filled Zipf distribution of token counts
    over experts;
  * parameter and activation sizes follow the usual Transformer counts.

A problem is a dict with four sub-dicts: ``model``, ``cluster``, ``params``,
``space``.  Array fields are numpy arrays with fixed dtypes (see
``_check_problem``).
"""
from __future__ import annotations

import math

import numpy as np

TP_VALUES = (1, 2, 4, 8)
CP_VALUES = (1, 2, 4, 8)

GB = 10**9


def _zipf_counts(rng, n_layers, is_moe, n_experts, tokens, top_k, s):
    """Tokens routed to each expert per layer: water-filled Zipf(s).

    Each token picks top_k distinct experts, so an expert receives at most
    ``tokens`` tokens and the layer total is about tokens * top_k.  The
    exponent of every layer is jittered by U[0.95, 1.05] and the expert ranks
    are shuffled per layer.
    """
    out = np.zeros((n_layers, n_experts), dtype=np.int64)
    if n_experts == 0:
        return out
    target = tokens * top_k
    ranks = np.arange(1, n_experts + 1, dtype=np.float64)
    for layer in range(n_layers):
        if not is_moe[layer]:
            continue
        sl = s * rng.uniform(0.95, 1.05)
        w = ranks ** (-sl)
        lo, hi = 0.0, float(target) / w.min() + 1.0
        for _ in range(200):  # bisection on the water level
            lam = 0.5 * (lo + hi)
            tot = np.minimum(float(tokens), lam * w).sum()
            if tot < target:
                lo = lam
            else:
                hi = lam
        cnt = np.floor(np.minimum(float(tokens), hi * w)).astype(np.int64)
        out[layer] = cnt[rng.permutation(n_experts)]
    return out


def _link_matrix(rng, n_types, intra, inter_lo, inter_hi):
    bw = np.zeros((n_types, n_types), dtype=np.float64)
    for a in range(n_types):
        for b in range(a, n_types):
            if a == b:
                bw[a, b] = intra
            else:
                v = float(rng.integers(int(inter_lo), int(inter_hi) + 1))
                bw[a, b] = bw[b, a] = v
    return bw


def _alpha_matrix(n_types, intra_ns, inter_ns):
    al = np.full((n_types, n_types), float(inter_ns))
    np.fill_diagonal(al, float(intra_ns))
    return al


def _flop_tables(rng, n_layers, is_moe, seq, hidden, f_dense, f_expert, speeds, jitter):
    """FLOP-derived compute tables t_dense/t_ffn[h][tp][cp][l] in int64 ns.

    Forward FLOPs of one layer on one micro-batch of ``seq`` tokens:
    8*S*H^2 (QKV/out projections) + 4*S^2*H (attention) + 6*S*H*F (gated FFN,
    F = dense FFN width, or one expert's width for MoE layers).  Forward plus
    backward = 3x forward, at 40% of a 1 PFLOP/s device scaled by the type's
    relative speed.  TP/CP split the work with a 5% per-doubling overhead.
    ``t_ffn`` is the FFN share of the same layer.  Every entry gets its own
    multiplicative jitter U[1-jitter, 1+jitter].
    """
    n_types = len(speeds)
    td = np.zeros((n_types, 4, 4, n_layers), dtype=np.int64)
    tf = np.zeros((n_types, 4, 4, n_layers), dtype=np.int64)
    S, H = float(seq), float(hidden)
    for layer in range(n_layers):
        F = float(f_expert if is_moe[layer] else f_dense)
        ffn = 6.0 * S * H * F
        tot = 8.0 * S * H * H + 4.0 * S * S * H + ffn
        for h in range(n_types):
            base = 3.0 * tot / (0.4e6 * speeds[h])       # ns (1e6 FLOP per ns)
            base_ffn = 3.0 * ffn / (0.4e6 * speeds[h])
            for i, tp in enumerate(TP_VALUES):
                for j, cp in enumerate(CP_VALUES):
                    sc = (1.0 + 0.05 * math.log2(tp) + 0.05 * math.log2(cp)) / (tp * cp)
                    d = math.ceil(base * sc * rng.uniform(1.0 - jitter, 1.0 + jitter))
                    f = math.ceil(base_ffn * sc * rng.uniform(1.0 - jitter, 1.0 + jitter))
                    f = min(f, d - 1)
                    td[h, i, j, layer] = d
                    tf[h, i, j, layer] = max(f, 0)
    return td, tf


def _params(rng, n_layers, is_moe, hidden, n_experts, f_dense, f_expert, n_shared, seq, mbs):
    H = hidden
    p_dense = np.zeros(n_layers, dtype=np.int64)
    p_exp = np.zeros(n_layers, dtype=np.int64)
    for layer in range(n_layers):
        if is_moe[layer]:
            p_dense[layer] = 4 * H * H + H * n_experts + n_shared * 3 * H * f_expert
            p_exp[layer] = n_experts * 3 * H * f_expert
        else:
            p_dense[layer] = 4 * H * H + 3 * H * f_dense
    act = np.full(n_layers, 34 * seq * H * mbs, dtype=np.int64)
    return p_dense, p_exp, act


def _default_params():
    return {
        "gamma": 0.5,          # load-imbalance weight, in [0, 1]
        "rc_time": 1.33,       # recomputation time factor
        "rc_act": 0.4,         # activation-memory factor xi(r=1)
        "opt_coef": 0.01,      # optimizer step, ns per parameter
        "delta_num": 1,        # load-balance tolerance delta = 1/5
        "delta_den": 5,
        "eta_prune": 2,        # heterogeneous-communication pruning factor
        "prune_window": 1,
        "prune_hetero": 1,
        "allow_recompute": 1,
    }


def _space(pp_max, ep_max, micro, mode=0, tp_mask=0xF, cp_mask=0xF, tpe_mask=0xF):
    return {"pp_max": pp_max, "tp_mask": tp_mask, "cp_mask": cp_mask, "ep_max": ep_max,
            "tpe_mask": tpe_mask, "mode": mode, "micro": list(micro)}


def config1(seed=1, mode=0):
    """Tiny: 8 MoE layers (H 1024, E 8 top-2, S 2048) on 4+4 devices of 2 types."""
    rng = np.random.default_rng(seed)
    N, S, H, E, k, mbs = 8, 2048, 1024, 8, 2, 1
    is_moe = np.ones(N, dtype=np.uint8)
    sigma = (1.0, 1.7)                       # per-type cost multipliers
    c = rng.integers(1000, 100001, size=N)   # base layer cost, ns
    td = np.zeros((2, 4, 4, N), dtype=np.int64)
    tf = np.zeros((2, 4, 4, N), dtype=np.int64)
    for h in range(2):
        for i, tp in enumerate(TP_VALUES):
            for j, cp in enumerate(CP_VALUES):
                for layer in range(N):
                    d = math.ceil(int(c[layer]) * sigma[h] / (tp * cp))
                    td[h, i, j, layer] = d
                    tf[h, i, j, layer] = (2 * d) // 3
    mem = rng.uniform(0.5, 2.0, size=N) * GB   # per-layer memory, half weights half activations
    p_exp = np.rint(mem / 36.0).astype(np.int64)   # 18 B/param at DP=1 -> weights = mem/2
    act = np.rint(mem / 2.0).astype(np.int64)
    model = {
        "n_layers": N, "seq_len": S, "hidden": H, "n_experts": E, "top_k": k,
        "micro_batch_size": mbs, "elem_bytes": 2, "moe_ffn_mult": 2.0,
        "is_moe": is_moe,
        "expert_tokens": _zipf_counts(rng, N, is_moe, E, S * mbs, k, 1.1),
        "params_dense": np.zeros(N, dtype=np.int64),
        "params_expert": p_exp,
        "act_bytes": act,
    }
    cluster = {
        "n_types": 2,
        "count": np.array([4, 4], dtype=np.int32),
        "speed": np.array([170, 100], dtype=np.int32),
        "mem_bytes": np.array([16 * GB, 24 * GB], dtype=np.int64),
        "eff": np.array([1.0, 1.0]),
        "route_coef": np.array([1e-4 * sigma[0], 1e-4 * sigma[1]]),
        "bw": np.array([[400.0, 50.0], [50.0, 400.0]]),
        "alpha": _alpha_matrix(2, 5000.0, 20000.0),
        "t_dense": td, "t_ffn": tf,
    }
    return {"name": "tiny-8L-moe-2types", "model": model, "cluster": cluster,
            "params": _default_params(), "space": _space(4, 8, [8], mode=mode)}


def _moe_model(rng, N, n_dense_first, S, H, E, k, n_shared, f_dense, f_expert, zipf_s):
    is_moe = np.ones(N, dtype=np.uint8)
    is_moe[:n_dense_first] = 0
    p_dense, p_exp, act = _params(rng, N, is_moe, H, E, f_dense, f_expert, n_shared, S, 1)
    model = {
        "n_layers": N, "seq_len": S, "hidden": H, "n_experts": E, "top_k": k,
        "micro_batch_size": 1, "elem_bytes": 2, "moe_ffn_mult": float(k + n_shared),
        "is_moe": is_moe,
        "expert_tokens": _zipf_counts(rng, N, is_moe, E, S, k, zipf_s),
        "params_dense": p_dense, "params_expert": p_exp, "act_bytes": act,
    }
    return model, is_moe


def config2(seed=2):
    """32-layer MoE (H 4096, E 64 top-8, S 4096) on 64 devices of 3 types (32/16/16)."""
    rng = np.random.default_rng(seed)
    N, S, H, E, k = 32, 4096, 4096, 64, 8
    model, is_moe = _moe_model(rng, N, 0, S, H, E, k, 0, 14336, 2048, 1.1)
    speeds = (1.0, 1.4, 2.2)
    td, tf = _flop_tables(rng, N, is_moe, S, H, 14336, 2048, speeds, 0.05)
    cluster = {
        "n_types": 3,
        "count": np.array([32, 16, 16], dtype=np.int32),
        "speed": np.array([100, 140, 220], dtype=np.int32),
        "mem_bytes": np.array([80 * GB, 64 * GB, 192 * GB], dtype=np.int64),
        "eff": np.array([1.0, 0.9, 0.85]),
        "route_coef": np.array([6.0 * E / (0.4e6 * s) for s in speeds]),
        "bw": _link_matrix(rng, 3, 400.0, 25, 50),
        "alpha": _alpha_matrix(3, 5000.0, 20000.0),
        "t_dense": td, "t_ffn": tf,
    }
    return {"name": "moe-32L-H4096-E64-3types", "model": model, "cluster": cluster,
            "params": _default_params(), "space": _space(8, 64, [8, 16, 32])}


_SPEEDS4 = (1.0, 1.3, 1.8, 2.5)
_HBM4 = (64 * GB, 96 * GB, 192 * GB, 288 * GB)


def _cluster4(rng, count, N, is_moe, S, H, f_dense, f_expert, E, jitter, mem_scale=1.0,
              flat_cost=None):
    if flat_cost is None:
        td, tf = _flop_tables(rng, N, is_moe, S, H, f_dense, f_expert, _SPEEDS4, jitter)
    else:
        td, tf = flat_cost
    return {
        "n_types": 4,
        "count": np.array([count] * 4, dtype=np.int32),
        "speed": np.array([int(round(100 * s)) for s in _SPEEDS4], dtype=np.int32),
        "mem_bytes": np.array([int(m * mem_scale) for m in _HBM4], dtype=np.int64),
        "eff": np.array([1.0, 0.95, 0.9, 0.85]),
        "route_coef": np.array([6.0 * E / (0.4e6 * s) for s in _SPEEDS4]),
        "bw": _link_matrix(rng, 4, 400.0, 25, 50),
        "alpha": _alpha_matrix(4, 5000.0, 20000.0),
        "t_dense": td, "t_ffn": tf,
    }


def config3(seed=3):
    """61-layer MoE (first 3 dense, H 7168, E 256 top-8, 1 shared, S 4096) on 4x64 devices."""
    rng = np.random.default_rng(seed)
    N, S, H, E, k = 61, 4096, 7168, 256, 8
    model, is_moe = _moe_model(rng, N, 3, S, H, E, k, 1, 18432, 2048, 1.1)
    cluster = _cluster4(rng, 64, N, is_moe, S, H, 18432, 2048, E, 0.15)
    return {"name": "moe-61L-H7168-E256-4types", "model": model, "cluster": cluster,
            "params": _default_params(), "space": _space(16, 64, [16, 32, 64])}


def config4(seed=4):
    """96-layer MoE (H 8192, E 128 top-4, S 8192, CP<=8) on 4x256 devices, B = 1..64."""
    rng = np.random.default_rng(seed)
    N, S, H, E, k = 96, 8192, 8192, 128, 4
    model, is_moe = _moe_model(rng, N, 0, S, H, E, k, 0, 28672, 4096, 1.1)
    cluster = _cluster4(rng, 256, N, is_moe, S, H, 28672, 4096, E, 0.15)
    return {"name": "moe-96L-H8192-E128-4types", "model": model, "cluster": cluster,
            "params": _default_params(), "space": _space(32, 128, range(1, 65))}


# Capacity multiplier of config 5: fixed so that about 95% of its candidates
# have no memory-feasible partition (value chosen by a sweep over the oracle).
CONFIG5_MEM_SCALE = 0.35


def config5(seed=5, mem_scale=None):
    """Adversarial: config-3 shapes, near-tied layer costs (+-1%), Zipf s=2, tight memory."""
    rng = np.random.default_rng(seed)
    N, S, H, E, k = 61, 4096, 7168, 256, 8
    model, is_moe = _moe_model(rng, N, 3, S, H, E, k, 1, 18432, 2048, 2.0)
    # every t_dense/t_ffn entry = c * U[0.99, 1.01], scaled like the FLOP tables
    td = np.zeros((4, 4, 4, N), dtype=np.int64)
    tf = np.zeros((4, 4, 4, N), dtype=np.int64)
    c = 2.0e7
    for h, sp in enumerate(_SPEEDS4):
        for i, tp in enumerate(TP_VALUES):
            for j, cp in enumerate(CP_VALUES):
                sc = (1.0 + 0.05 * math.log2(tp) + 0.05 * math.log2(cp)) / (tp * cp) / sp
                for layer in range(N):
                    d = math.ceil(c * sc * rng.uniform(0.99, 1.01))
                    td[h, i, j, layer] = d
                    tf[h, i, j, layer] = math.ceil(0.3 * d * rng.uniform(0.99, 1.01))
    scale = CONFIG5_MEM_SCALE if mem_scale is None else mem_scale
    cluster = _cluster4(rng, 64, N, is_moe, S, H, 18432, 2048, E, 0.0, mem_scale=scale,
                        flat_cost=(td, tf))
    return {"name": "adversarial-61L-neartie-tightmem", "model": model, "cluster": cluster,
            "params": _default_params(), "space": _space(16, 64, [16, 32, 64])}


_WORKLOADS = {1: config1, 2: config2, 3: config3, 4: config4, 5: config5}


def config(n, **kw):
    """Synthetic problem of config ``n`` (1..5)."""
    return _check_problem(_WORKLOADS[n](**kw))


def random_tiny(seed, n_layers=None, n_types=None, max_pp=4, micro=None, flags=None):
    """Small random problem for brute-force checks (N <= 12, PP <= 4, <= 3 types)."""
    rng = np.random.default_rng(10_000 + seed)
    N = int(n_layers if n_layers is not None else rng.integers(2, 13))
    T = int(n_types if n_types is not None else rng.integers(1, 4))
    counts = [int(rng.choice([1, 2, 4])) for _ in range(T)]
    while sum(counts) & (sum(counts) - 1):   # keep the device total a power of two
        counts[int(rng.integers(0, T))] += 1
    E = int(rng.choice([0, 4, 8]))
    k = int(rng.choice([1, 2])) if E else 1
    S = int(rng.choice([256, 512, 1024]))
    H = int(rng.choice([256, 512]))
    is_moe = (rng.random(N) < 0.7).astype(np.uint8) if E else np.zeros(N, dtype=np.uint8)
    td = np.zeros((T, 4, 4, N), dtype=np.int64)
    tf = np.zeros((T, 4, 4, N), dtype=np.int64)
    for h in range(T):
        for i in range(4):
            for j in range(4):
                d = rng.integers(2000, 200000, size=N)
                td[h, i, j] = d
                tf[h, i, j] = (d * rng.uniform(0.1, 0.9, size=N)).astype(np.int64)
    p_dense = rng.integers(0, 5 * 10**7, size=N).astype(np.int64)
    p_exp = np.where(is_moe == 1, rng.integers(10**6, 10**8, size=N), 0).astype(np.int64)
    act = rng.integers(10**7, 2 * 10**9, size=N).astype(np.int64)
    bw = _link_matrix(rng, T, float(rng.integers(100, 500)), 10, 90)
    al = _alpha_matrix(T, float(rng.integers(0, 8000)), float(rng.integers(5000, 30000)))
    mem = [int(rng.integers(2, 40)) * GB for _ in range(T)]
    model = {
        "n_layers": N, "seq_len": S, "hidden": H, "n_experts": E, "top_k": k,
        "micro_batch_size": int(rng.choice([1, 2])), "elem_bytes": 2,
        "moe_ffn_mult": float(rng.choice([1.0, 2.0, 3.0])),
        "is_moe": is_moe,
        "expert_tokens": _zipf_counts(rng, N, is_moe, E, S, k, float(rng.uniform(0.0, 2.0))),
        "params_dense": p_dense, "params_expert": p_exp, "act_bytes": act,
    }
    cluster = {
        "n_types": T,
        "count": np.array(counts, dtype=np.int32),
        "speed": np.array([int(rng.integers(50, 300)) for _ in range(T)], dtype=np.int32),
        "mem_bytes": np.array(mem, dtype=np.int64),
        "eff": rng.uniform(0.5, 1.0, size=T),
        "route_coef": rng.uniform(0.0, 1e-3, size=T),
        "bw": bw, "alpha": al, "t_dense": td, "t_ffn": tf,
    }
    params = _default_params()
    params["gamma"] = float(rng.choice([0.0, 0.5, 1.0]))
    params["opt_coef"] = float(rng.uniform(0.0, 0.05))
    if flags is not None:
        params.update(flags)
    else:
        params["prune_window"] = int(rng.integers(0, 2))
        params["prune_hetero"] = int(rng.integers(0, 2))
        params["allow_recompute"] = int(rng.integers(0, 2))
    if micro is None:
        micro = sorted(set(int(x) for x in rng.choice([1, 2, 3, 8], size=2)))
    space = _space(max_pp, max(E, 1), micro, mode=int(rng.integers(0, 2)))
    return _check_problem({"name": f"tiny-random-{seed}", "model": model, "cluster": cluster,
                           "params": params, "space": space})


_INT_DT = {"is_moe": np.uint8, "expert_tokens": np.int64, "params_dense": np.int64,
           "params_expert": np.int64, "act_bytes": np.int64, "count": np.int32,
           "speed": np.int32, "mem_bytes": np.int64, "t_dense": np.int64, "t_ffn": np.int64}


def _check_problem(p):
    """Normalise dtypes/contiguity (no arithmetic of the method)."""
    m, c = p["model"], p["cluster"]
    for d in (m, c):
        for key, val in list(d.items()):
            if isinstance(val, np.ndarray):
                dt = _INT_DT.get(key, np.float64)
                d[key] = np.ascontiguousarray(val, dtype=dt)
    N, T = m["n_layers"], c["n_types"]
    assert m["is_moe"].shape == (N,)
    assert m["expert_tokens"].shape[0] == N
    assert c["t_dense"].shape == (T, 4, 4, N) and c["t_ffn"].shape == (T, 4, 4, N)
    assert c["bw"].shape == (T, T) and c["alpha"].shape == (T, T)
    return p
