"""ctypes front-end of the CPU oracle -- TEST INFRASTRUCTURE ONLY.

Only the test-suite, ``__graft_entry__.smoke()`` and the bench's CPU-baseline
leg import this module.  It marshals a problem dictionary (see the package's
``workloads`` module for the fields) into the oracle's own flat C struct and
calls the plain C implementation in ``hapmoe_oracle.c``.  It imports nothing
from the HIP library's package.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from . import build as _build

MAX_TYPES = 4
MAX_STAGES = 64
MAX_MICRO = 64
INF = np.iinfo(np.int64).max


class OrcProblem(C.Structure):
    _fields_ = [
        ("n_layers", C.c_int32), ("seq_len", C.c_int32), ("hidden", C.c_int32),
        ("n_experts", C.c_int32), ("top_k", C.c_int32), ("micro_batch_size", C.c_int32),
        ("elem_bytes", C.c_int32),
        ("moe_ffn_mult", C.c_double),
        ("is_moe", C.c_void_p), ("expert_tokens", C.c_void_p), ("params_dense", C.c_void_p),
        ("params_expert", C.c_void_p), ("act_bytes", C.c_void_p),
        ("n_types", C.c_int32),
        ("count", C.c_int32 * MAX_TYPES), ("speed", C.c_int32 * MAX_TYPES),
        ("mem_bytes", C.c_int64 * MAX_TYPES),
        ("eff", C.c_double * MAX_TYPES), ("route_coef", C.c_double * MAX_TYPES),
        ("bw", C.c_double * (MAX_TYPES * MAX_TYPES)), ("alpha", C.c_double * (MAX_TYPES * MAX_TYPES)),
        ("t_dense", C.c_void_p), ("t_ffn", C.c_void_p),
        ("gamma", C.c_double), ("rc_time", C.c_double), ("rc_act", C.c_double), ("opt_coef", C.c_double),
        ("delta_num", C.c_int32), ("delta_den", C.c_int32), ("eta_prune", C.c_int32),
        ("prune_window", C.c_int32), ("prune_hetero", C.c_int32), ("allow_recompute", C.c_int32),
        ("pp_max", C.c_int32), ("tp_mask", C.c_int32), ("cp_mask", C.c_int32), ("ep_max", C.c_int32),
        ("tpe_mask", C.c_int32), ("mode", C.c_int32), ("stage_types", C.c_int32),
        ("n_micro", C.c_int32), ("micro", C.c_int32 * MAX_MICRO),
    ]


class OrcConfig(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("pp", "tp", "cp", "dp", "ep", "tpe")]


class OrcStage(C.Structure):
    _fields_ = [("mask", C.c_int32), ("speed", C.c_int32), ("lo", C.c_int32), ("hi", C.c_int32),
                ("mixed", C.c_int32), ("bdiff", C.c_int32), ("first_type", C.c_int32),
                ("last_type", C.c_int32), ("cap", C.c_int64), ("p2p", C.c_int64),
                ("m_store", C.c_int64), ("alpha", C.c_double), ("bw", C.c_double)]


class OrcTypeTerms(C.Structure):
    _fields_ = [("comp", C.c_double), ("expert", C.c_double), ("q_comp", C.c_int64),
                ("q_expert", C.c_int64)]


class OrcMaskTerms(C.Structure):
    _fields_ = [("a2a", C.c_double), ("tp", C.c_double), ("cp", C.c_double), ("q_a2a", C.c_int64),
                ("q_tp", C.c_int64), ("q_cp", C.c_int64), ("comm", C.c_int64), ("t_r0", C.c_int64),
                ("t_r1", C.c_int64)]


class OrcMemTerms(C.Structure):
    _fields_ = [("w", C.c_double), ("a0", C.c_double), ("q_w", C.c_int64), ("q_a0", C.c_int64),
                ("q_a1", C.c_int64)]


class OrcPiTerms(C.Structure):
    _fields_ = [("p_avg", C.c_double), ("dp_const_f", C.c_double), ("x_f", C.c_double),
                ("x_bytes", C.c_int64), ("tbar", C.c_int64)]


class OrcResult(C.Structure):
    _fields_ = [("status", C.c_int32), ("pp", C.c_int32), ("opt", C.c_int64), ("sum", C.c_int64),
                ("tmax", C.c_int64), ("dp_const", C.c_int64), ("thresholds", C.c_int64),
                ("layers", C.c_uint8 * MAX_STAGES), ("recompute", C.c_uint8 * MAX_STAGES),
                ("stage_mask", C.c_uint8 * MAX_STAGES), ("width", C.c_uint8 * MAX_STAGES)]


_LIB = None


def lib():
    """Load liboracle.so, compiling it first if it is not there.  The
    environment variable HAPMOE_ORACLE_LIB names another build of the same
    source to load instead (the mutation test plants mistakes in copies)."""
    global _LIB
    if _LIB is None:
        path = os.environ.get("HAPMOE_ORACLE_LIB") or _build.build(force=False)
        L = C.CDLL(path)
        P = C.POINTER
        L.orc_validate.argtypes = [P(OrcProblem)]
        L.orc_enumerate.argtypes = [P(OrcProblem), P(OrcConfig), C.c_int64]
        L.orc_enumerate.restype = C.c_int64
        L.orc_n_orders.argtypes = [P(OrcProblem)]
        L.orc_order.argtypes = [P(OrcProblem), C.c_int32, P(C.c_int32)]
        L.orc_order.restype = None
        L.orc_sequence.argtypes = [P(OrcProblem), C.c_int32, C.c_int32, P(C.c_int32)]
        L.orc_n_instances.argtypes = [P(OrcProblem)]
        L.orc_n_instances.restype = C.c_int64
        for name, T in (("orc_mask_terms_eval", OrcMaskTerms),):
            getattr(L, name).argtypes = [P(OrcProblem), P(OrcConfig), C.c_int32, C.c_int32, P(T)]
            getattr(L, name).restype = None
        L.orc_type_terms_eval.argtypes = [P(OrcProblem), P(OrcConfig), C.c_int32, C.c_int32,
                                          P(OrcTypeTerms)]
        L.orc_type_terms_eval.restype = None
        L.orc_mem_terms_eval.argtypes = [P(OrcProblem), P(OrcConfig), C.c_int32, P(OrcMemTerms)]
        L.orc_mem_terms_eval.restype = None
        L.orc_pi_terms_eval.argtypes = [P(OrcProblem), P(OrcConfig), P(OrcPiTerms)]
        L.orc_pi_terms_eval.restype = None
        L.orc_p2p.argtypes = [P(OrcProblem), P(OrcConfig), C.c_int32, C.c_int32]
        L.orc_p2p.restype = C.c_int64
        L.orc_dp_const.argtypes = [P(OrcProblem), P(OrcConfig), C.c_int32]
        L.orc_dp_const.restype = C.c_int64
        L.orc_stages.argtypes = [P(OrcProblem), P(OrcConfig), C.c_int32, C.c_int32, P(OrcStage)]
        L.orc_segment_costs.argtypes = [P(OrcProblem), C.c_int64, C.c_void_p, C.c_void_p]
        L.orc_dp.argtypes = [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, P(OrcResult)]
        L.orc_brute.argtypes = [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, P(OrcResult)]
        L.orc_solve.argtypes = [P(OrcProblem), C.c_int64, P(OrcResult)]
        L.orc_solve_brute.argtypes = [P(OrcProblem), C.c_int64, P(OrcResult)]
        L.orc_solve_many.argtypes = [P(OrcProblem), C.c_void_p, C.c_int64, P(OrcResult)]
        L.orc_latency_1f1b.argtypes = [C.c_int32, C.c_void_p, C.c_int64]
        L.orc_latency_1f1b.restype = C.c_int64
        L.orc_dp_exact.argtypes = [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, P(OrcResult)]
        L.orc_brute_exact.argtypes = [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, P(OrcResult)]
        L.orc_solve_exact.argtypes = [P(OrcProblem), C.c_int64, P(OrcResult)]
        L.orc_solve_exact_brute.argtypes = [P(OrcProblem), C.c_int64, P(OrcResult)]
        L.orc_solve_exact_many.argtypes = [P(OrcProblem), C.c_void_p, C.c_int64, P(OrcResult)]
        L.orc_width_costs.argtypes = [P(OrcProblem), C.c_int64, C.c_void_p, C.c_void_p]
        L.orc_width_terms.argtypes = [P(OrcProblem), P(OrcConfig), C.c_int32, C.c_int32, C.c_int32,
                                      P(OrcTypeTerms), P(OrcMaskTerms), P(OrcMemTerms), P(C.c_int64)]
        L.orc_width_terms.restype = None
        L.orc_width_stage.argtypes = [P(OrcProblem), P(OrcConfig), C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                      C.c_int32, P(OrcStage)]
        for name in ("orc_dp_widths", "orc_brute_widths"):
            getattr(L, name).argtypes = [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, P(OrcResult)]
        for name in ("orc_dp_latency", "orc_brute_latency"):
            getattr(L, name).argtypes = [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, P(OrcResult)]
        for name in ("orc_solve_latency", "orc_solve_latency_brute"):
            getattr(L, name).argtypes = [P(OrcProblem), C.c_int64, P(OrcResult)]
        L.orc_solve_latency_many.argtypes = [P(OrcProblem), C.c_void_p, C.c_int64, P(OrcResult)]
        L.orc_type_costs.argtypes = [P(OrcProblem), C.c_int64, C.c_void_p, C.c_void_p]
        for name in ("orc_dp_types", "orc_brute_types", "orc_dp_types_exact", "orc_brute_types_exact"):
            getattr(L, name).argtypes = [C.c_int32, C.c_int32, C.c_void_p, C.c_int32, C.c_int64, C.c_void_p,
                                         P(OrcResult)]
        _LIB = L
    return _LIB


def _ptr(a):
    return a.ctypes.data_as(C.c_void_p)


def result_dict(r: OrcResult) -> dict:
    pp = r.pp
    return {"status": r.status, "pp": pp, "opt": r.opt, "sum": r.sum, "tmax": r.tmax,
            "dp_const": r.dp_const, "thresholds": r.thresholds,
            "layers": list(r.layers[:pp]), "recompute": list(r.recompute[:pp]),
            "stage_mask": list(r.stage_mask[:pp]), "width": list(r.width[:pp])}


class Oracle:
    """Oracle bound to one problem dictionary."""

    def __init__(self, problem: dict):
        m, c, pa, sp = problem["model"], problem["cluster"], problem["params"], problem["space"]
        T = int(c["n_types"])
        self._keep = {
            "is_moe": np.ascontiguousarray(m["is_moe"], dtype=np.uint8),
            "expert_tokens": np.ascontiguousarray(m["expert_tokens"], dtype=np.int64),
            "params_dense": np.ascontiguousarray(m["params_dense"], dtype=np.int64),
            "params_expert": np.ascontiguousarray(m["params_expert"], dtype=np.int64),
            "act_bytes": np.ascontiguousarray(m["act_bytes"], dtype=np.int64),
            "t_dense": np.ascontiguousarray(c["t_dense"], dtype=np.int64),
            "t_ffn": np.ascontiguousarray(c["t_ffn"], dtype=np.int64),
        }
        P = OrcProblem()
        P.n_layers, P.seq_len, P.hidden = m["n_layers"], m["seq_len"], m["hidden"]
        P.n_experts, P.top_k, P.micro_batch_size = m["n_experts"], m["top_k"], m["micro_batch_size"]
        P.elem_bytes = m["elem_bytes"]
        P.moe_ffn_mult = float(m["moe_ffn_mult"])
        for name in ("is_moe", "expert_tokens", "params_dense", "params_expert", "act_bytes",
                     "t_dense", "t_ffn"):
            setattr(P, name, _ptr(self._keep[name]))
        P.n_types = T
        for h in range(T):
            P.count[h] = int(c["count"][h])
            P.speed[h] = int(c["speed"][h])
            P.mem_bytes[h] = int(c["mem_bytes"][h])
            P.eff[h] = float(c["eff"][h])
            P.route_coef[h] = float(c["route_coef"][h])
            for g in range(T):
                P.bw[h * MAX_TYPES + g] = float(c["bw"][h][g])
                P.alpha[h * MAX_TYPES + g] = float(c["alpha"][h][g])
        for name in ("gamma", "rc_time", "rc_act", "opt_coef"):
            setattr(P, name, float(pa[name]))
        for name in ("delta_num", "delta_den", "eta_prune", "prune_window", "prune_hetero",
                     "allow_recompute"):
            setattr(P, name, int(pa[name]))
        for name in ("pp_max", "tp_mask", "cp_mask", "ep_max", "tpe_mask", "mode"):
            setattr(P, name, int(sp[name]))
        P.stage_types = int(sp.get("stage_types", 0))
        micro = list(sp["micro"])
        P.n_micro = len(micro)
        for i, b in enumerate(micro):
            P.micro[i] = int(b)
        self.P = P
        self.problem = problem
        self.L = lib()
        if self.L.orc_validate(C.byref(P)) != 0:
            raise ValueError("oracle: invalid problem")

    # ---- enumeration -------------------------------------------------------
    def configs(self):
        n = self.L.orc_enumerate(C.byref(self.P), None, 0)
        arr = (OrcConfig * max(n, 1))()
        self.L.orc_enumerate(C.byref(self.P), arr, n)
        return [(x.pp, x.tp, x.cp, x.dp, x.ep, x.tpe) for x in arr[:n]]

    def n_orders(self):
        return self.L.orc_n_orders(C.byref(self.P))

    def order(self, o):
        perm = (C.c_int32 * MAX_TYPES)()
        self.L.orc_order(C.byref(self.P), o, perm)
        return list(perm[: self.P.n_types])

    def sequence(self, pp, o):
        """Free per-stage types: the o-th stage-type sequence of a pp-stage pipeline (None past the last)."""
        seq = (C.c_int32 * MAX_STAGES)()
        if self.L.orc_sequence(C.byref(self.P), int(pp), int(o), seq) != 0:
            return None
        return list(seq[: int(pp)])

    def n_instances(self):
        return self.L.orc_n_instances(C.byref(self.P))

    # ---- cost model --------------------------------------------------------
    @staticmethod
    def _cfg(cfg):
        return OrcConfig(*[int(v) for v in cfg])

    def type_terms(self, cfg, layer, h):
        o = OrcTypeTerms()
        self.L.orc_type_terms_eval(C.byref(self.P), C.byref(self._cfg(cfg)), layer, h, C.byref(o))
        return {k: getattr(o, k) for k, _ in o._fields_}

    def mask_terms(self, cfg, layer, mask):
        o = OrcMaskTerms()
        self.L.orc_mask_terms_eval(C.byref(self.P), C.byref(self._cfg(cfg)), layer, mask, C.byref(o))
        return {k: getattr(o, k) for k, _ in o._fields_}

    def mem_terms(self, cfg, layer):
        o = OrcMemTerms()
        self.L.orc_mem_terms_eval(C.byref(self.P), C.byref(self._cfg(cfg)), layer, C.byref(o))
        return {k: getattr(o, k) for k, _ in o._fields_}

    def pi_terms(self, cfg):
        o = OrcPiTerms()
        self.L.orc_pi_terms_eval(C.byref(self.P), C.byref(self._cfg(cfg)), C.byref(o))
        return {k: getattr(o, k) for k, _ in o._fields_}

    def p2p(self, cfg, h_from, h_to):
        return self.L.orc_p2p(C.byref(self.P), C.byref(self._cfg(cfg)), h_from, h_to)

    def dp_const(self, cfg, order):
        return self.L.orc_dp_const(C.byref(self.P), C.byref(self._cfg(cfg)), order)

    def stages(self, cfg, order, micro):
        st = (OrcStage * MAX_STAGES)()
        self.L.orc_stages(C.byref(self.P), C.byref(self._cfg(cfg)), order, micro, st)
        return [{k: getattr(s, k) for k, _ in s._fields_} for s in st[: int(cfg[0])]]

    def type_costs(self, idx):
        """Device-count DP (stage_types = 2): cost[s][h][h'][a][b] and the recomputation flags."""
        cfgs = self.configs()
        pp = cfgs[idx // (self.n_orders() * self.P.n_micro)][0]
        T, W = self.P.n_types, self.P.n_layers + 1
        cost = np.zeros((pp, T, T + 1, W, W), dtype=np.int64)
        rflag = np.zeros((pp, T, T + 1, W, W), dtype=np.uint8)
        if self.L.orc_type_costs(C.byref(self.P), idx, _ptr(cost), _ptr(rflag)) != 0:
            raise IndexError(idx)
        return cost, rflag

    def width_terms(self, cfg, layer, mask, w):
        """Per-stage widths: the terms of one layer on a width-w stage (w half-groups)."""
        T = self.P.n_types
        tt = (OrcTypeTerms * T)()
        mt, me, x = OrcMaskTerms(), OrcMemTerms(), C.c_int64(0)
        self.L.orc_width_terms(C.byref(self.P), C.byref(self._cfg(cfg)), layer, mask, w, tt, C.byref(mt),
                               C.byref(me), C.byref(x))
        return {"type": [{k: getattr(t, k) for k, _ in t._fields_} for t in tt],
                "mask": {k: getattr(mt, k) for k, _ in mt._fields_},
                "mem": {k: getattr(me, k) for k, _ in me._fields_}, "x_bytes": x.value}

    def width_stage(self, cfg, order, s, u, w, micro):
        x = OrcStage()
        if self.L.orc_width_stage(C.byref(self.P), C.byref(self._cfg(cfg)), order, s, u, w, micro, C.byref(x)) != 0:
            raise IndexError((s, u, w))
        return {k: getattr(x, k) for k, _ in x._fields_}

    def width_costs(self, idx):
        """Per-stage widths (stage_types = 3): cost[s][u][w-1][a][b] and the recomputation flags."""
        cfgs = self.configs()
        pp = cfgs[idx // (self.n_orders() * self.P.n_micro)][0]
        W = self.P.n_layers + 1
        cost = np.zeros((pp, 2 * pp + 1, 3, W, W), dtype=np.int64)
        rflag = np.zeros((pp, 2 * pp + 1, 3, W, W), dtype=np.uint8)
        if self.L.orc_width_costs(C.byref(self.P), idx, _ptr(cost), _ptr(rflag)) != 0:
            raise IndexError(idx)
        return cost, rflag

    def segment_costs(self, idx):
        cfgs = self.configs()
        per = self.n_orders() * self.P.n_micro
        pp = cfgs[idx // per][0]
        W = self.P.n_layers + 1
        cost = np.zeros((pp, W, W), dtype=np.int64)
        rflag = np.zeros((pp, W, W), dtype=np.uint8)
        if self.L.orc_segment_costs(C.byref(self.P), idx, _ptr(cost), _ptr(rflag)) != 0:
            raise IndexError(idx)
        return cost, rflag

    # ---- search ------------------------------------------------------------
    def solve(self, idx):
        r = OrcResult()
        if self.L.orc_solve(C.byref(self.P), int(idx), C.byref(r)) != 0:
            raise IndexError(idx)
        return result_dict(r)

    def solve_brute(self, idx):
        r = OrcResult()
        if self.L.orc_solve_brute(C.byref(self.P), int(idx), C.byref(r)) != 0:
            raise IndexError(idx)
        return result_dict(r)

    def solve_many(self, idx):
        idx = np.ascontiguousarray(idx, dtype=np.int64)
        res = (OrcResult * max(len(idx), 1))()
        if self.L.orc_solve_many(C.byref(self.P), _ptr(idx), len(idx), res) != 0:
            raise IndexError("instance out of range")
        return [result_dict(r) for r in res[: len(idx)]]

    # ---- 1F1B re-scoring of the (max, sum) Pareto frontier ----------------------
    def solve_exact(self, idx):
        r = OrcResult()
        if self.L.orc_solve_exact(C.byref(self.P), int(idx), C.byref(r)) != 0:
            raise IndexError(idx)
        return result_dict(r)

    def solve_exact_brute(self, idx):
        r = OrcResult()
        if self.L.orc_solve_exact_brute(C.byref(self.P), int(idx), C.byref(r)) != 0:
            raise IndexError(idx)
        return result_dict(r)

    def solve_exact_many(self, idx):
        idx = np.ascontiguousarray(idx, dtype=np.int64)
        res = (OrcResult * max(len(idx), 1))()
        if self.L.orc_solve_exact_many(C.byref(self.P), _ptr(idx), len(idx), res) != 0:
            raise IndexError("instance out of range")
        return [result_dict(r) for r in res[: len(idx)]]

    # ---- the least 1F1B latency over every partition ---------------------------
    def solve_latency(self, idx):
        r = OrcResult()
        if self.L.orc_solve_latency(C.byref(self.P), int(idx), C.byref(r)) != 0:
            raise IndexError(idx)
        return result_dict(r)

    def solve_latency_brute(self, idx):
        r = OrcResult()
        if self.L.orc_solve_latency_brute(C.byref(self.P), int(idx), C.byref(r)) != 0:
            raise IndexError(idx)
        return result_dict(r)

    def solve_latency_many(self, idx):
        idx = np.ascontiguousarray(idx, dtype=np.int64)
        res = (OrcResult * max(len(idx), 1))()
        if self.L.orc_solve_latency_many(C.byref(self.P), _ptr(idx), len(idx), res) != 0:
            raise IndexError("instance out of range")
        return [result_dict(r) for r in res[: len(idx)]]

    def best(self):
        """Global arg-min over all instances of (objective, instance index)."""
        best = None
        for i in range(self.n_instances()):
            r = self.solve(i)
            if r["status"] == 0 and (best is None or r["opt"] < best[1]["opt"]):
                best = (i, r)
        return best


def dp(pp, n, micro, cost):
    """Threshold DP on an explicit cost tensor [pp][n+1][n+1] (INF = infeasible)."""
    cost = np.ascontiguousarray(cost, dtype=np.int64)
    assert cost.shape == (pp, n + 1, n + 1)
    r = OrcResult()
    lib().orc_dp(pp, n, micro, _ptr(cost), C.byref(r))
    return result_dict(r)


def brute(pp, n, micro, cost):
    """Brute force over all compositions on an explicit cost tensor."""
    cost = np.ascontiguousarray(cost, dtype=np.int64)
    assert cost.shape == (pp, n + 1, n + 1)
    r = OrcResult()
    lib().orc_brute(pp, n, micro, _ptr(cost), C.byref(r))
    return result_dict(r)


def latency_1f1b(costs, micro):
    """1F1B iteration latency of a partition from its stage costs (see the C side)."""
    c = np.ascontiguousarray(costs, dtype=np.int64)
    return int(lib().orc_latency_1f1b(len(c), _ptr(c), int(micro)))


def dp_exact(pp, n, micro, cost):
    """1F1B re-scoring of the Pareto frontier on an explicit cost tensor."""
    cost = np.ascontiguousarray(cost, dtype=np.int64)
    assert cost.shape == (pp, n + 1, n + 1)
    r = OrcResult()
    lib().orc_dp_exact(pp, n, micro, _ptr(cost), C.byref(r))
    return result_dict(r)


def brute_exact(pp, n, micro, cost):
    """Brute force of the same objective over all compositions."""
    cost = np.ascontiguousarray(cost, dtype=np.int64)
    assert cost.shape == (pp, n + 1, n + 1)
    r = OrcResult()
    lib().orc_brute_exact(pp, n, micro, _ptr(cost), C.byref(r))
    return result_dict(r)


def dp_widths(pp, n, micro, cost):
    """Per-stage widths: the threshold DP on an explicit tensor [pp][2pp+1][3][n+1][n+1]."""
    cost = np.ascontiguousarray(cost, dtype=np.int64)
    assert cost.shape == (pp, 2 * pp + 1, 3, n + 1, n + 1)
    r = OrcResult()
    lib().orc_dp_widths(pp, n, micro, _ptr(cost), C.byref(r))
    return result_dict(r)


def brute_widths(pp, n, micro, cost):
    """Brute force over every width sequence and composition on the same tensor."""
    cost = np.ascontiguousarray(cost, dtype=np.int64)
    assert cost.shape == (pp, 2 * pp + 1, 3, n + 1, n + 1)
    r = OrcResult()
    lib().orc_brute_widths(pp, n, micro, _ptr(cost), C.byref(r))
    return result_dict(r)


def dp_latency(pp, n, micro, cost):
    """The least 1F1B latency over every partition of an explicit cost tensor."""
    cost = np.ascontiguousarray(cost, dtype=np.int64)
    assert cost.shape == (pp, n + 1, n + 1)
    r = OrcResult()
    lib().orc_dp_latency(pp, n, micro, _ptr(cost), C.byref(r))
    return result_dict(r)


def brute_latency(pp, n, micro, cost):
    """Brute force of the same minimum over all compositions."""
    cost = np.ascontiguousarray(cost, dtype=np.int64)
    assert cost.shape == (pp, n + 1, n + 1)
    r = OrcResult()
    lib().orc_brute_latency(pp, n, micro, _ptr(cost), C.byref(r))
    return result_dict(r)


def _types_call(name, k, n, micro, cost):
    cost = np.ascontiguousarray(cost, dtype=np.int64)
    pp, T = cost.shape[0], cost.shape[1]
    assert cost.shape == (pp, T, T + 1, n + 1, n + 1) and len(k) == T and sum(k) == pp
    kk = np.ascontiguousarray(k, dtype=np.int32)
    r = OrcResult()
    getattr(lib(), name)(pp, T, _ptr(kk), n, micro, _ptr(cost), C.byref(r))
    d = result_dict(r)
    d["types"] = [m.bit_length() - 1 for m in d["stage_mask"]] if d["status"] == 0 else []
    return d


def dp_types(k, n, micro, cost):
    """Device-count DP on an explicit tensor [pp][T][T+1][n+1][n+1] (k[h] stages of type h)."""
    return _types_call("orc_dp_types", k, n, micro, cost)


def brute_types(k, n, micro, cost):
    """Brute force over every stage-type sequence and composition on the same tensor."""
    return _types_call("orc_brute_types", k, n, micro, cost)


def dp_types_exact(k, n, micro, cost):
    """1F1B re-scoring of the device-count DP's frontier on an explicit tensor."""
    return _types_call("orc_dp_types_exact", k, n, micro, cost)


def brute_types_exact(k, n, micro, cost):
    """Brute force of the same objective over every sequence and composition."""
    return _types_call("orc_brute_types_exact", k, n, micro, cost)


def solve_worker(args):
    """multiprocessing helper: (problem, instance indices[, "exact"]) -> results."""
    problem, idx = args[0], args[1]
    if len(args) > 2 and args[2] == "exact":
        return Oracle(problem).solve_exact_many(idx)
    if len(args) > 2 and args[2] == "latency":
        return Oracle(problem).solve_latency_many(idx)
    return Oracle(problem).solve_many(idx)


__all__ = ["Oracle", "dp", "brute", "dp_exact", "brute_exact", "dp_types", "brute_types", "dp_types_exact",
           "brute_types_exact", "latency_1f1b", "dp_latency", "brute_latency", "dp_widths", "brute_widths",
           "INF", "lib", "solve_worker"]
