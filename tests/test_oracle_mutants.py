"""The pins catch plausible misreadings of the paper in the oracle.

Each case plants one mistake in a copy of the oracle's C source -- a term
divided by the wrong parallel degree, a maximum taken where the paper's model
needs a minimum, a dropped factor -- builds it on the CPU, and runs the pin
tests (the hand-worked problems W1 and W2, the closed forms and the pinned
counts) against that build.  Every mutant must fail at least one of them; the
unchanged source must pass.  Nothing here touches the library or a GPU.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "hapmoe_oracle.c")
PINS = ["tests/test_oracle_pins.py", "tests/test_oracle_w2.py"]
CFLAGS = ["-O1", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", "-w"]

# (what the mistake is, text of the oracle, its replacement)
MUTANTS = [
    ("TPE ring all-reduce taken over TP (Section 3.2 collectives)",
     "2.0 * ring_allreduce(D, c->tpe, alpha, bw)", "2.0 * ring_allreduce(D, c->tp, alpha, bw)"),
    ("dense-layer TP all-reduce count 2 instead of 4",
     "o->tp = 4.0 * ring_allreduce(D, c->tp, alpha, bw);", "o->tp = 2.0 * ring_allreduce(D, c->tp, alpha, bw);"),
    ("Eq. 2 expert work divided by TP instead of TPE",
     "((p->eff[h] * (double)c->ep) * (double)c->tpe)", "((p->eff[h] * (double)c->ep) * (double)c->tp)"),
    ("Eq. 2 without the device efficiency eta_h",
     "((p->eff[h] * (double)c->ep) * (double)c->tpe)", "((1.0 * (double)c->ep) * (double)c->tpe)"),
    ("expert parameters sharded by EP * TP instead of EP * TPE",
     "(double)p->params_expert[layer] / (double)(c->ep * c->tpe)) * beta_opt",
     "(double)p->params_expert[layer] / (double)(c->ep * c->tp)) * beta_opt"),
    ("CP ring term without the split over TP",
     "((2.0 * D) / (double)c->tp) / bw", "(2.0 * D) / bw"),
    ("activations split by TP only",
     "(double)p->act_bytes[layer] / (double)(c->tp * c->cp)", "(double)p->act_bytes[layer] / (double)c->tp"),
    ("activations split by CP only",
     "(double)p->act_bytes[layer] / (double)(c->tp * c->cp)", "(double)p->act_bytes[layer] / (double)c->cp"),
    ("optimizer state not sharded over DP (18 bytes a parameter)",
     "6.0 + 12.0 / (double)c->dp", "18.0"),
    ("pruning-1 weights summed over device types instead of stages",
     "sum_speed += x->speed;", "sum_speed += s < p->n_types ? p->speed[s] : 0;"),
    ("straddling stage takes the largest capacity of its types",
     "p->mem_bytes[h] < x->cap) x->cap", "p->mem_bytes[h] > x->cap) x->cap"),
    ("straddling stage takes the fastest speed of its types",
     "p->speed[h] < x->speed) x->speed", "p->speed[h] > x->speed) x->speed"),
    ("a type set's link at its fastest bandwidth",
     "if (first || bb < b) b = bb;", "if (first || bb > b) b = bb;"),
    ("a type set's link at its smallest latency",
     "if (first || al > a) a = al;", "if (first || al < a) a = al;"),
    ("a straddling stage's compute at its fastest type",
     "if (t.q_comp + t.q_expert > ce) ce = t.q_comp + t.q_expert;",
     "if (ce < 0 || t.q_comp + t.q_expert < ce) ce = t.q_comp + t.q_expert;"),
    ("1F1B stored micro-batches PP - i + 2 (off by one)",
     "        x->m_store = min64(PP - s, micro);\n        sum_speed",
     "        x->m_store = min64(PP - s + 1, micro);\n        sum_speed"),
    ("stored micro-batches not capped by B",
     "        x->m_store = min64(PP - s, micro);\n        sum_speed",
     "        x->m_store = PP - s;\n        sum_speed"),
    ("all-to-all always, never the all-gather dispatcher",
     "double sel = f_ag < f_a2a ? f_ag : f_a2a;", "double sel = f_a2a;"),
    ("load imbalance taken as rho itself, without gamma",
     "return 1.0 + p->gamma * (rho - 1.0);", "return rho;"),
    ("boundary transfer without the split over TP",
     "(act_tensor(p, c) / (double)c->tp) / bw", "act_tensor(p, c) / bw"),
    ("MoE buffers counting the dispatch buffer once",
     "+ 2.0 * dm;", "+ dm;"),
    ("pruning-3 bound rounded down",
     "o->tbar = (s + c->pp - 1) / c->pp;", "o->tbar = s / c->pp;"),
    ("pruning 3 with >= instead of >",
     "if (hc > (int64_t)p->eta_prune * pt->tbar)", "if (hc >= (int64_t)p->eta_prune * pt->tbar)"),
    ("T_dp-sync at the fastest stage link",
     "if (s == 0 || st[s].bw < bw) bw = st[s].bw;", "if (s == 0 || st[s].bw > bw) bw = st[s].bw;"),
    ("optimizer step not divided over DP",
     "(p->opt_coef * t.p_avg) / (double)c->dp", "(p->opt_coef * t.p_avg)"),
]


def _run(tmpdir, k, old, new):
    src = open(SRC).read()
    # the width mode restates some terms: a mistake is planted in every copy
    assert old is None or 1 <= src.count(old) <= 2, f"mutant {k}: the text to replace must occur once or twice"
    path = os.path.join(tmpdir, f"mutant{k}.c")
    lib = os.path.join(tmpdir, f"libmutant{k}.so")
    with open(path, "w") as f:
        f.write(src.replace(old, new) if old else src)
    subprocess.run(["gcc", *CFLAGS, "-I", os.path.join(ROOT, "oracle"), "-o", lib, path, "-lm"], check=True)
    env = dict(os.environ, HAPMOE_ORACLE_LIB=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *PINS], cwd=ROOT,
                       env=env, capture_output=True, text=True, timeout=600)
    return r.returncode


def test_every_mutant_fails_a_pin(tmp_path):
    cases = [(k, old, new) for k, (_, old, new) in enumerate(MUTANTS)] + [(len(MUTANTS), None, None)]
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        codes = list(ex.map(lambda c: _run(str(tmp_path), *c), cases))
    assert codes[-1] == 0, "the unchanged oracle must pass its pins"
    survivors = [MUTANTS[k][0] for k, rc in enumerate(codes[:-1]) if rc == 0]
    assert not survivors, f"mistakes no pin catches: {survivors}"
    assert all(rc == 1 for rc in codes[:-1]), codes   # failed tests, not a crash
