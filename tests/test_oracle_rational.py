"""Every modelled term of the oracle against exact rational arithmetic.

The oracle evaluates each term in fp64 and rounds it up once.  Here the same
quantities are evaluated in exact rationals (``fractions.Fraction``; a
real-valued input is taken as the decimal it is written as) straight from the paper's definitions (Section 3.2 Eq. 2, Eq. 3,
load imbalance, collectives and memory; Section 3.4 boundary transfers and the
pruning-3 bound; Eq. 4 T_dp-sync + T_opt), then rounded up.  A rounded term may
differ from the exact one only where fp64 rounding carries the value across an
integer; such a crossing is allowed as +-1 when the exact value lies within
1e-9 (relative) of that integer, and every crossing found is listed in the
failure message.  The fp64 values themselves must be within 1e-12 relative of
the exact ones.

This checks the oracle's arithmetic (operation order, rounding, the integer
window and bound formulas); which formula each term follows is pinned by the
hand-worked problems W1 and W2.
"""
import math
from fractions import Fraction as Fr

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2609_39350_amd import workloads
from tests.problems import worked_problem, worked_problem_w2


def _ceil(x: Fr) -> int:
    return math.ceil(x)


class Exact:
    """The cost model of one problem in exact rationals."""

    def __init__(self, p):
        self.p = p
        m, c, pa = p["model"], p["cluster"], p["params"]
        self.m, self.c, self.pa = m, c, pa
        self.T = int(c["n_types"])

    @staticmethod
    def f(x):
        # a real-valued input as the decimal it was written as (1.33, 0.4, ...):
        # the shortest decimal that reads back as the same double
        return Fr(repr(float(x)))

    def tokens(self, cfg):
        return Fr(int(self.m["seq_len"]) * int(self.m["micro_batch_size"]) // cfg[2])

    def act(self, cfg):
        return self.tokens(cfg) * int(self.m["hidden"]) * int(self.m["elem_bytes"])

    def skew(self, layer):
        E = int(self.m["n_experts"])
        cnt = [int(v) for v in self.m["expert_tokens"][layer][:E]]
        tot = sum(cnt)
        rho = Fr(max(cnt) * E, tot) if tot > 0 else Fr(1)
        return 1 + self.f(self.pa["gamma"]) * (rho - 1)

    def link(self, mask):
        pairs = [(h, g) for h in range(self.T) for g in range(self.T) if (mask >> h) & 1 and (mask >> g) & 1]
        a = max(self.f(self.c["alpha"][h][g]) for h, g in pairs)
        b = min(self.f(self.c["bw"][h][g]) for h, g in pairs)
        return a, b

    @staticmethod
    def ring(nbytes, w, a, b):
        if w == 1:
            return Fr(0)
        return 2 * (w - 1) * a + Fr(2 * (w - 1)) * nbytes / w / b

    def table(self, key, h, cfg, layer):
        tp_i, cp_i = int(math.log2(cfg[1])), int(math.log2(cfg[2]))
        return int(self.c[key][h][tp_i][cp_i][layer])

    def type_terms(self, cfg, layer, h):
        td, tf = self.table("t_dense", h, cfg, layer), self.table("t_ffn", h, cfg, layer)
        if not self.m["is_moe"][layer]:
            return Fr(td), Fr(0)
        route = self.f(self.c["route_coef"][h]) * self.tokens(cfg) * int(self.m["hidden"])
        comp = Fr(td - tf) + route
        expert = self.skew(layer) * self.f(self.m["moe_ffn_mult"]) * tf / (self.f(self.c["eff"][h]) * cfg[4] * cfg[5])
        return comp, expert

    def mask_terms(self, cfg, layer, mask):
        a, b = self.link(mask)
        D = self.act(cfg)
        if not self.m["is_moe"][layer]:
            a2a, tp = Fr(0), 4 * self.ring(D, cfg[1], a, b)
        else:
            ep = cfg[4]
            dm = D * int(self.m["top_k"]) * (1 - Fr(1, ep))
            f_a2a = (ep - 1) * a + dm / b
            f_ag = (ep - 1) * a + D * (ep - 1) / b
            a2a = self.skew(layer) * 4 * min(f_a2a, f_ag)
            tp = 2 * self.ring(D, cfg[1], a, b) + 2 * self.ring(D, cfg[5], a, b)
        cp = Fr(0) if cfg[2] == 1 else 3 * (cfg[2] - 1) * (a + 2 * D / cfg[1] / b)
        return a2a, tp, cp

    def mem_terms(self, cfg, layer):
        beta_opt = 6 + Fr(12, cfg[3])
        w = (Fr(int(self.m["params_dense"][layer]), cfg[1]) +
             Fr(int(self.m["params_expert"][layer]), cfg[4] * cfg[5])) * beta_opt
        a0 = Fr(int(self.m["act_bytes"][layer]), cfg[1] * cfg[2])
        return w, a0

    def p_avg(self, cfg):
        pd = sum(int(v) for v in self.m["params_dense"])
        pe = sum(int(v) for v in self.m["params_expert"])
        return (Fr(pd, cfg[1]) + Fr(pe, cfg[4] * cfg[5])) / cfg[0]

    def x_bytes(self, cfg):
        D = self.act(cfg)
        dm = D * int(self.m["top_k"]) * (1 - Fr(1, cfg[4]))
        return 8 * self.tokens(cfg) * int(self.m["top_k"]) + 2 * dm

    def p2p(self, cfg, h, g):
        a, b = self.f(self.c["alpha"][h][g]), self.f(self.c["bw"][h][g])
        return 2 * (a + self.act(cfg) / cfg[1] / b)


def _near_integer(x: Fr) -> bool:
    return abs(x - round(x)) <= Fr(1, 10**9) * max(1, abs(x))


def _check_term(exact: Fr, fp: float, q: int, what, crossings, bad):
    if fp is not None and exact != 0 and abs(Fr(fp) - exact) > Fr(1, 10**12) * abs(exact):
        bad.append((what, "fp64", fp, float(exact)))
    e = _ceil(exact)
    if q != e:
        if abs(q - e) == 1 and _near_integer(exact):
            crossings.append((what, q, e))
        else:
            bad.append((what, "rounded", q, e))


def _problems():
    out = [("w1", worked_problem()), ("w2", worked_problem_w2()), ("config1", workloads.config(1))]
    out += [(f"tiny{s}", workloads.random_tiny(s)) for s in range(12)]
    return out


@pytest.mark.parametrize("name,problem", _problems(), ids=[n for n, _ in _problems()])
def test_every_term_against_exact_rationals(name, problem):
    o = orc.Oracle(problem)
    X = Exact(problem)
    T, N = X.T, int(problem["model"]["n_layers"])
    cfgs = o.configs()
    sample = cfgs if len(cfgs) <= 48 else [cfgs[i] for i in np.linspace(0, len(cfgs) - 1, 48).astype(int)]
    bad, crossings = [], []
    rc_time, rc_act = Exact.f(problem["params"]["rc_time"]), Exact.f(problem["params"]["rc_act"])
    for cfg in sample:
        qce = {}
        for layer in range(N):
            for h in range(T):
                comp, expert = X.type_terms(cfg, layer, h)
                r = o.type_terms(cfg, layer, h)
                _check_term(comp, r["comp"], r["q_comp"], (cfg, layer, h, "comp"), crossings, bad)
                _check_term(expert, r["expert"], r["q_expert"], (cfg, layer, h, "expert"), crossings, bad)
                qce[layer, h] = r["q_comp"] + r["q_expert"]
            for mask in range(1, 2 ** T):
                a2a, tp, cp = X.mask_terms(cfg, layer, mask)
                r = o.mask_terms(cfg, layer, mask)
                for f, v in (("a2a", a2a), ("tp", tp), ("cp", cp)):
                    _check_term(v, r[f], r["q_" + f], (cfg, layer, mask, f), crossings, bad)
                comm = r["q_a2a"] + r["q_tp"] + r["q_cp"]
                t0 = max(qce[layer, h] for h in range(T) if (mask >> h) & 1) + comm
                if (r["comm"], r["t_r0"]) != (comm, t0):
                    bad.append(((cfg, layer, mask), "t_r0", (r["comm"], r["t_r0"]), (comm, t0)))
                _check_term(rc_time * t0, None, r["t_r1"], (cfg, layer, mask, "t_r1"), crossings, bad)
            w, a0 = X.mem_terms(cfg, layer)
            r = o.mem_terms(cfg, layer)
            _check_term(w, r["w"], r["q_w"], (cfg, layer, "w"), crossings, bad)
            _check_term(a0, r["a0"], r["q_a0"], (cfg, layer, "a0"), crossings, bad)
            _check_term(rc_act * r["q_a0"], None, r["q_a1"], (cfg, layer, "a1"), crossings, bad)
        pt = o.pi_terms(cfg)
        _check_term(X.x_bytes(cfg), pt["x_f"], pt["x_bytes"], (cfg, "x"), crossings, bad)
        if abs(Fr(pt["p_avg"]) - X.p_avg(cfg)) > Fr(1, 10**12) * max(1, X.p_avg(cfg)):
            bad.append((cfg, "p_avg", pt["p_avg"], float(X.p_avg(cfg))))
        tbar = -(-sum(max(qce[layer, h] for h in range(T)) for layer in range(N)) // cfg[0])
        if pt["tbar"] != tbar:
            bad.append((cfg, "tbar", pt["tbar"], tbar))
        for h in range(T):
            for g in range(T):
                v = X.p2p(cfg, h, g)
                _check_term(v, None, o.p2p(cfg, h, g), (cfg, "p2p", h, g), crossings, bad)
        for od in range(o.n_orders()):
            st = o.stages(cfg, od, 1)
            a = max(Fr(s["alpha"]) for s in st)
            b = min(Fr(s["bw"]) for s in st)
            pa = X.p_avg(cfg)
            c = X.ring(4 * pa, cfg[3], a, b) + Exact.f(problem["params"]["opt_coef"]) * pa / cfg[3]
            _check_term(c, None, o.dp_const(cfg, od), (cfg, od, "dp_const"), crossings, bad)
    assert not bad, f"{len(bad)} terms differ from exact arithmetic, first: {bad[:4]}"
    assert len(crossings) <= 2, f"fp64 crossings: {crossings}"


def _exact_window(p, speeds):
    N = int(p["model"]["n_layers"])
    dn, dd = int(p["params"]["delta_num"]), int(p["params"]["delta_den"])
    tot = sum(speeds)
    out = []
    for P in speeds:
        lo = max(1, math.floor(Fr((dd - dn) * P * N, dd * tot)))
        hi = min(N, math.ceil(Fr((dd + dn) * P * N, dd * tot)))
        out.append((lo, hi))
    return out


@pytest.mark.parametrize("n", [1, 2, 3])
def test_pruning1_windows_exact(n):
    """Section 3.4 pruning 1 windows from exact rationals of the stage speeds."""
    p = workloads.config(n)
    o = orc.Oracle(p)
    for cfg in o.configs()[:: max(1, len(o.configs()) // 40)]:
        for od in range(o.n_orders()):
            st = o.stages(cfg, od, 1)
            assert [(s["lo"], s["hi"]) for s in st] == _exact_window(p, [s["speed"] for s in st]), (cfg, od)
