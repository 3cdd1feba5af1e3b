"""Hand-built problem dictionaries for the tests (inputs only, no method arithmetic)."""
import copy
import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def worked_problem():
    """Problem W1 of tests/golden/worked_w1.json (two layers, two device types)."""
    N, T = 2, 2
    td = np.zeros((T, 4, 4, N), dtype=np.int64)
    for h in range(T):
        for i, tp in enumerate((1, 2, 4, 8)):
            for j, cp in enumerate((1, 2, 4, 8)):
                for layer in range(N):
                    td[h, i, j, layer] = 80000 * (h + 1) * (layer + 1) // (tp * cp)
    tf = td // 2
    model = {
        "n_layers": N, "seq_len": 1024, "hidden": 512, "n_experts": 4, "top_k": 2,
        "micro_batch_size": 1, "elem_bytes": 2, "moe_ffn_mult": 2.0,
        "is_moe": np.array([0, 1], dtype=np.uint8),
        "expert_tokens": np.array([[0, 0, 0, 0], [800, 400, 400, 448]], dtype=np.int64),
        "params_dense": np.array([1_000_000, 500_000], dtype=np.int64),
        "params_expert": np.array([0, 4_000_000], dtype=np.int64),
        "act_bytes": np.array([100_000_000, 50_000_000], dtype=np.int64),
    }
    cluster = {
        "n_types": T,
        "count": np.array([2, 2], dtype=np.int32),
        "speed": np.array([100, 200], dtype=np.int32),
        "mem_bytes": np.array([10 * 10**9, 20 * 10**9], dtype=np.int64),
        "eff": np.array([1.0, 0.5]),
        "route_coef": np.array([0.001, 0.002]),
        "bw": np.array([[400.0, 50.0], [50.0, 400.0]]),
        "alpha": np.array([[1000.0, 4000.0], [4000.0, 1000.0]]),
        "t_dense": td, "t_ffn": tf,
    }
    params = {"gamma": 0.5, "rc_time": 1.33, "rc_act": 0.4, "opt_coef": 0.5,
              "delta_num": 1, "delta_den": 5, "eta_prune": 2,
              "prune_window": 1, "prune_hetero": 1, "allow_recompute": 1}
    space = {"pp_max": 2, "tp_mask": 0xF, "cp_mask": 0xF, "ep_max": 4, "tpe_mask": 0xF,
             "mode": 0, "micro": [4]}
    return {"name": "worked-w1", "model": model, "cluster": cluster, "params": params,
            "space": space}


def worked_problem_w2():
    """Problem W2 of tests/golden/worked_w2.json: four layers on two device types
    with unequal counts (20 + 12 devices), so that a 4-stage pipeline of 8-device
    groups has one stage straddling the type boundary; the space holds only
    TP = 2, CP = 2, TPE = 4 and EP in {1, 2}."""
    N, T = 4, 2
    td = np.zeros((T, 4, 4, N), dtype=np.int64)
    for h in range(T):
        for i, tp in enumerate((1, 2, 4, 8)):
            for j, cp in enumerate((1, 2, 4, 8)):
                for layer in range(N):
                    td[h, i, j, layer] = 80000 * (h + 1) * (layer + 1) // (tp * cp)
    tf = td // 2
    tokens = np.zeros((N, 8), dtype=np.int64)
    tokens[1] = [256, 128, 128, 128, 128, 128, 128, 0]   # max 256 of 1024: rho = 2
    tokens[2] = 128                                       # uniform: rho = 1
    tokens[3] = [512, 64, 64, 64, 64, 64, 64, 128]      # max 512 of 1024: rho = 4
    model = {
        "n_layers": N, "seq_len": 1024, "hidden": 256, "n_experts": 8, "top_k": 2,
        "micro_batch_size": 1, "elem_bytes": 2, "moe_ffn_mult": 2.0,
        "is_moe": np.array([0, 1, 1, 1], dtype=np.uint8),
        "expert_tokens": tokens,
        "params_dense": np.array([1_000_000, 200_000, 200_000, 200_000], dtype=np.int64),
        "params_expert": np.array([0, 8_000_000, 8_000_000, 8_000_000], dtype=np.int64),
        "act_bytes": np.array([100_000_000, 50_000_000, 50_000_000, 50_000_000], dtype=np.int64),
    }
    cluster = {
        "n_types": T,
        "count": np.array([20, 12], dtype=np.int32),
        "speed": np.array([100, 300], dtype=np.int32),
        "mem_bytes": np.array([36_000_000, 100_000_000], dtype=np.int64),
        "eff": np.array([1.0, 0.5]),
        "route_coef": np.array([2.0 ** -10, 2.0 ** -9]),
        "bw": np.array([[400.0, 50.0], [50.0, 200.0]]),
        "alpha": np.array([[1000.0, 4000.0], [4000.0, 2000.0]]),
        "t_dense": td, "t_ffn": tf,
    }
    params = {"gamma": 0.5, "rc_time": 1.33, "rc_act": 0.4, "opt_coef": 0.5,
              "delta_num": 1, "delta_den": 5, "eta_prune": 2,
              "prune_window": 1, "prune_hetero": 1, "allow_recompute": 1}
    space = {"pp_max": 4, "tp_mask": 0x2, "cp_mask": 0x2, "ep_max": 2, "tpe_mask": 0x4,
             "mode": 0, "micro": [3]}
    return {"name": "worked-w2", "model": model, "cluster": cluster, "params": params,
            "space": space}


def variant(problem, **changes):
    """Deep copy with dotted-path overrides, e.g. variant(p, **{"params.gamma": 0.0})."""
    q = copy.deepcopy(problem)
    for path, val in changes.items():
        d = q
        keys = path.split(".")
        for k in keys[:-1]:
            d = d[k]
        d[keys[-1]] = val
    return q
