"""ctypes binding of libhapmoe.so (C ABI in include/hapmoe.h).

Argument marshalling only: every step of the planner runs in the library's
host enumeration and gfx950 kernels.  PyTorch supplies device memory
(``tensor.data_ptr()``) and streams (``torch.cuda.current_stream()``).  The
functions keep the names of the C calls.  If the built library is missing the
import fails loudly -- there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhapmoe.so")

MAX_TYPES = 4
MAX_STAGES = 32
MAX_MICRO = 64

ERRORS = {0: "HAPMOE_OK", -1: "HAPMOE_E_INVAL", -2: "HAPMOE_E_CAPACITY", -3: "HAPMOE_E_WORKSPACE",
          -4: "HAPMOE_E_HIP", -5: "HAPMOE_E_ARCH", -6: "HAPMOE_E_INFEASIBLE", -7: "HAPMOE_E_RANGE"}
STATUS_OK, STATUS_INFEASIBLE, STATUS_OVERFLOW = 0, 1, 2


class HapmoeError(RuntimeError):
    def __init__(self, code, what):
        self.code = code
        super().__init__(f"{what}: {ERRORS.get(code, code)} ({_strerror(code)})")


class Model(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("seq_len", C.c_int32), ("hidden", C.c_int32),
                ("n_experts", C.c_int32), ("top_k", C.c_int32), ("micro_batch_size", C.c_int32),
                ("elem_bytes", C.c_int32), ("moe_ffn_mult", C.c_double),
                ("is_moe", C.c_void_p), ("expert_tokens", C.c_void_p), ("params_dense", C.c_void_p),
                ("params_expert", C.c_void_p), ("act_bytes", C.c_void_p)]


class Cluster(C.Structure):
    _fields_ = [("n_types", C.c_int32), ("count", C.c_int32 * MAX_TYPES), ("speed", C.c_int32 * MAX_TYPES),
                ("mem_bytes", C.c_int64 * MAX_TYPES), ("eff", C.c_double * MAX_TYPES),
                ("route_coef", C.c_double * MAX_TYPES),
                ("bw", (C.c_double * MAX_TYPES) * MAX_TYPES), ("alpha", (C.c_double * MAX_TYPES) * MAX_TYPES),
                ("t_dense", C.c_void_p), ("t_ffn", C.c_void_p)]


class Params(C.Structure):
    _fields_ = [("gamma", C.c_double), ("rc_time", C.c_double), ("rc_act", C.c_double),
                ("opt_coef", C.c_double), ("delta_num", C.c_int32), ("delta_den", C.c_int32),
                ("eta_prune", C.c_int32), ("prune_window", C.c_int32), ("prune_hetero", C.c_int32),
                ("allow_recompute", C.c_int32)]


class Space(C.Structure):
    _fields_ = [("pp_max", C.c_int32), ("tp_mask", C.c_int32), ("cp_mask", C.c_int32), ("ep_max", C.c_int32),
                ("tpe_mask", C.c_int32), ("mode", C.c_int32), ("stage_types", C.c_int32), ("n_micro", C.c_int32),
                ("micro", C.c_int32 * MAX_MICRO), ("global_batch", C.c_int32)]


class Problem(C.Structure):
    _fields_ = [("model", Model), ("cluster", Cluster), ("params", Params), ("space", Space)]


class Plan(C.Structure):
    _fields_ = [("instance", C.c_int64), ("objective", C.c_int64), ("stage_sum", C.c_int64),
                ("t_max", C.c_int64), ("dp_const", C.c_int64), ("cand", C.c_int32 * 8),
                ("n_stages", C.c_int32), ("recompute_mask", C.c_uint32),
                ("layers", C.c_uint8 * MAX_STAGES), ("stage_types", C.c_uint8 * MAX_STAGES)]


CANDIDATE_DTYPE = np.dtype([(n, "<i4") for n in ("pp", "tp", "cp", "dp", "ep", "tpe", "order", "n_micro")])
RESULT_DTYPE = np.dtype([("objective", "<i8"), ("stage_sum", "<i8"), ("t_max", "<i8"), ("status", "<i4"),
                         ("recompute_mask", "<u4"), ("layers", "u1", (MAX_STAGES,))])
assert CANDIDATE_DTYPE.itemsize == 32 and RESULT_DTYPE.itemsize == 64

_LIB = None


def lib():
    """The loaded libhapmoe.so.  Raises if it has not been built."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        P, i64, vp = C.POINTER, C.c_int64, C.c_void_p
        L.hapmoe_strerror.argtypes = [C.c_int32]
        L.hapmoe_strerror.restype = C.c_char_p
        L.hapmoe_validate.argtypes = [P(Problem)]
        L.hapmoe_enumerate_candidates.argtypes = [P(Problem), vp, i64, P(i64)]
        L.hapmoe_image_bytes.argtypes = [P(Problem), P(i64)]
        L.hapmoe_pack_image.argtypes = [P(Problem), vp, i64]
        L.hapmoe_tables_bytes.argtypes = [P(Problem), P(i64)]
        L.hapmoe_debug_bytes.argtypes = [P(Problem), P(i64)]
        L.hapmoe_eval_cost_tables.argtypes = [P(Problem), vp, vp, i64, i64, i64, vp, i64, vp, i64, vp]
        L.hapmoe_stage_dp.argtypes = [P(Problem), vp, vp, i64, vp, i64, i64, i64, vp, vp, vp, i64, vp]
        L.hapmoe_stage_dp_1f1b.argtypes = [P(Problem), vp, vp, i64, vp, i64, i64, i64, vp, vp, vp, i64, vp]
        L.hapmoe_stage_dp_latency.argtypes = [P(Problem), vp, vp, i64, vp, i64, i64, i64, vp, vp, vp]
        L.hapmoe_stage_dp_ws_bytes.argtypes = [P(Problem), P(i64)]
        L.hapmoe_tables_layout.argtypes = [P(Problem), P(i64)]
        L.hapmoe_debug_layout.argtypes = [P(Problem), P(i64)]
        L.hapmoe_best_plan_ws_bytes.argtypes = [P(Problem), i64, P(i64)]
        L.hapmoe_best_plan.argtypes = [P(Problem), vp, vp, i64, vp, vp, i64, vp, vp, i64, P(Plan), vp]
        L.hapmoe_best_plan_noalloc.argtypes = [P(Problem), vp, vp, i64, vp, vp, i64, vp, P(Plan), vp]
        L.hapmoe_stage_dp_types.argtypes = [P(Problem), vp, vp, i64, vp, i64, i64, i64, vp, vp, vp, vp, i64, vp]
        L.hapmoe_stage_dp_types_ws_bytes.argtypes = [P(Problem), P(i64)]
        L.hapmoe_stage_dp_types_1f1b.argtypes = L.hapmoe_stage_dp_types.argtypes
        L.hapmoe_stage_dp_widths.argtypes = [P(Problem), vp, vp, i64, vp, i64, i64, i64, vp, vp, vp, vp, vp, i64, vp]
        L.hapmoe_stage_dp_widths_ws_bytes.argtypes = [P(Problem), i64, P(i64)]
        L.hapmoe_section_clocks.argtypes = [P(C.c_uint64), C.c_int32]
        L.hapmoe_section_clocks.restype = C.c_int32
        for f in ("hapmoe_validate", "hapmoe_enumerate_candidates", "hapmoe_image_bytes", "hapmoe_pack_image",
                  "hapmoe_tables_bytes", "hapmoe_debug_bytes", "hapmoe_tables_layout", "hapmoe_debug_layout", "hapmoe_eval_cost_tables", "hapmoe_stage_dp", "hapmoe_stage_dp_1f1b", "hapmoe_stage_dp_ws_bytes",
                  "hapmoe_best_plan_ws_bytes", "hapmoe_best_plan", "hapmoe_best_plan_noalloc", "hapmoe_stage_dp_types",
                  "hapmoe_stage_dp_types_ws_bytes", "hapmoe_stage_dp_types_1f1b", "hapmoe_stage_dp_widths",
                  "hapmoe_stage_dp_widths_ws_bytes", "hapmoe_stage_dp_latency"):
            getattr(L, f).restype = C.c_int32
        _LIB = L
    return _LIB


def _strerror(code):
    try:
        return lib().hapmoe_strerror(code).decode()
    except Exception:   # noqa: BLE001 - message only
        return "?"


def _check(code, what):
    if code != 0:
        raise HapmoeError(code, what)


class HostProblem:
    """A problem dictionary marshalled into the C struct (keeps the arrays alive)."""

    def __init__(self, problem: dict):
        m, c, pa, sp = problem["model"], problem["cluster"], problem["params"], problem["space"]
        self.arrays = {
            "is_moe": np.ascontiguousarray(m["is_moe"], dtype=np.uint8),
            "expert_tokens": np.ascontiguousarray(m["expert_tokens"], dtype=np.int64),
            "params_dense": np.ascontiguousarray(m["params_dense"], dtype=np.int64),
            "params_expert": np.ascontiguousarray(m["params_expert"], dtype=np.int64),
            "act_bytes": np.ascontiguousarray(m["act_bytes"], dtype=np.int64),
            "t_dense": np.ascontiguousarray(c["t_dense"], dtype=np.int64),
            "t_ffn": np.ascontiguousarray(c["t_ffn"], dtype=np.int64),
        }
        p = Problem()
        mm = p.model
        for f in ("n_layers", "seq_len", "hidden", "n_experts", "top_k", "micro_batch_size", "elem_bytes"):
            setattr(mm, f, int(m[f]))
        mm.moe_ffn_mult = float(m["moe_ffn_mult"])
        for f in ("is_moe", "expert_tokens", "params_dense", "params_expert", "act_bytes"):
            setattr(mm, f, self.arrays[f].ctypes.data)
        cc = p.cluster
        T = int(c["n_types"])
        cc.n_types = T
        for h in range(T):
            cc.count[h] = int(c["count"][h])
            cc.speed[h] = int(c["speed"][h])
            cc.mem_bytes[h] = int(c["mem_bytes"][h])
            cc.eff[h] = float(c["eff"][h])
            cc.route_coef[h] = float(c["route_coef"][h])
            for g in range(T):
                cc.bw[h][g] = float(c["bw"][h][g])
                cc.alpha[h][g] = float(c["alpha"][h][g])
        cc.t_dense = self.arrays["t_dense"].ctypes.data
        cc.t_ffn = self.arrays["t_ffn"].ctypes.data
        for f in ("gamma", "rc_time", "rc_act", "opt_coef"):
            setattr(p.params, f, float(pa[f]))
        for f in ("delta_num", "delta_den", "eta_prune", "prune_window", "prune_hetero", "allow_recompute"):
            setattr(p.params, f, int(pa[f]))
        for f in ("pp_max", "tp_mask", "cp_mask", "ep_max", "tpe_mask", "mode"):
            setattr(p.space, f, int(sp[f]))
        p.space.stage_types = int(sp.get("stage_types", 0))
        p.space.global_batch = int(sp.get("global_batch", 0))
        micro = list(sp["micro"])
        p.space.n_micro = len(micro)
        for i, b in enumerate(micro[:MAX_MICRO]):
            p.space.micro[i] = int(b)
        self.c = p
        self.ref = C.byref(p)


def use_section_clocks():
    """Load the diagnostic build (libhapmoe_clocks.so) instead of the library;
    call before anything else touches the binding."""
    global LIB_PATH
    if _LIB is not None:
        raise RuntimeError("the library is already loaded")
    LIB_PATH = os.path.join(os.path.dirname(LIB_PATH), "libhapmoe_clocks.so")


SECTION_NAMES = ("setup", "scan", "relax", "trace", "control")


def section_clocks(clear=True) -> dict:
    """Stage-DP section clocks since the last clear (diagnostic build only)."""
    out = (C.c_uint64 * 16)()
    _check(lib().hapmoe_section_clocks(out, 1 if clear else 0), "hapmoe_section_clocks")
    v = list(out)
    total = max(v[5], 1)
    out = {"share": {n: v[i] / total for i, n in enumerate(SECTION_NAMES)}, "wave_cycles": v[5],
           "keys": v[6], "segment_batches": v[7], "passes": v[8]}
    khz = v[13]
    if khz and v[12]:
        us = 1e3 / khz   # microseconds a tick
        start, end_min, end_max = (~v[10]) & (2**64 - 1), (~v[11]) & (2**64 - 1), v[12]
        # wall-clock view of the last launch (the maxima span every launch since the clear)
        out["longest_key_us"] = (v[9] >> 6) * us
        out["longest_key_pp"] = v[9] & 63
        out["first_wave_done_us"] = (end_min - start) * us
        out["last_wave_done_us"] = (end_max - start) * us
    return out


def _hp(problem):
    return problem if isinstance(problem, HostProblem) else HostProblem(problem)


def _stream(stream):
    if stream is None:
        import torch
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    return C.c_void_p(int(stream))


def _dptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


# ---------------------------------------------------------------- host calls
def validate(problem):
    _check(lib().hapmoe_validate(_hp(problem).ref), "hapmoe_validate")


def enumerate_candidates(problem) -> np.ndarray:
    hp = _hp(problem)
    n = C.c_int64(0)
    code = lib().hapmoe_enumerate_candidates(hp.ref, None, 0, C.byref(n))
    if code not in (0, -2):
        _check(code, "hapmoe_enumerate_candidates")
    out = np.zeros(n.value, dtype=CANDIDATE_DTYPE)
    _check(lib().hapmoe_enumerate_candidates(hp.ref, out.ctypes.data, n.value, C.byref(n)),
           "hapmoe_enumerate_candidates")
    return out


def image_bytes(problem) -> int:
    n = C.c_int64(0)
    _check(lib().hapmoe_image_bytes(_hp(problem).ref, C.byref(n)), "hapmoe_image_bytes")
    return n.value


def pack_image(problem) -> np.ndarray:
    hp = _hp(problem)
    buf = np.zeros(image_bytes(hp), dtype=np.uint8)
    _check(lib().hapmoe_pack_image(hp.ref, buf.ctypes.data, buf.nbytes), "hapmoe_pack_image")
    return buf


def tables_bytes(problem) -> int:
    n = C.c_int64(0)
    _check(lib().hapmoe_tables_bytes(_hp(problem).ref, C.byref(n)), "hapmoe_tables_bytes")
    return n.value


def debug_bytes(problem) -> int:
    n = C.c_int64(0)
    _check(lib().hapmoe_debug_bytes(_hp(problem).ref, C.byref(n)), "hapmoe_debug_bytes")
    return n.value


def tables_layout(problem) -> dict:
    out = (C.c_int64 * 9)()
    _check(lib().hapmoe_tables_layout(_hp(problem).ref, out), "hapmoe_tables_layout")
    keys = ("n_configs", "n_orders", "n_masks", "np", "off_pi", "off_key", "off_mem", "off_time", "total")
    return dict(zip(keys, list(out)))


def debug_layout(problem) -> dict:
    out = (C.c_int64 * 4)()
    _check(lib().hapmoe_debug_layout(_hp(problem).ref, out), "hapmoe_debug_layout")
    return dict(zip(("per_cfg", "off_type", "off_mask", "off_mem"), list(out)))


PI_DTYPE = np.dtype([("x_bytes", "<i8"), ("tbar", "<i8"), ("p2p", "<i8", (16,)), ("status", "<i4"),
                     ("used_masks", "<u4")])
KEY_DTYPE = np.dtype([("dp_const", "<i8"), ("mask", "u1", (32,)), ("lo", "u1", (32,)), ("hi", "u1", (32,)),
                      ("bpair", "u1", (32,))])
assert PI_DTYPE.itemsize == 152 and KEY_DTYPE.itemsize == 136


def decode_tables(problem, raw: np.ndarray) -> dict:
    """Split a host copy of the cost-table buffer into its documented parts."""
    L = tables_layout(problem)
    nc, no, nm, np_ = L["n_configs"], L["n_orders"], L["n_masks"], L["np"]
    raw = np.ascontiguousarray(raw).view(np.uint8)
    pi = raw[L["off_pi"]:L["off_pi"] + nc * 152].view(PI_DTYPE)
    key = raw[L["off_key"]:L["off_key"] + nc * no * 136].view(KEY_DTYPE).reshape(nc, no)
    mem = raw[L["off_mem"]:L["off_mem"] + nc * 4 * np_ * 8].view("<i8").reshape(nc, 4, np_)
    time = raw[L["off_time"]:L["off_time"] + nc * nm * 3 * np_ * 8].view("<i8").reshape(nc, nm, 3, np_)
    return {"pi": pi, "key": key, "mem": mem, "time": time, "layout": L}


def best_plan_ws_bytes(problem, n) -> int:
    b = C.c_int64(0)
    _check(lib().hapmoe_best_plan_ws_bytes(_hp(problem).ref, int(n), C.byref(b)), "hapmoe_best_plan_ws_bytes")
    return b.value


# -------------------------------------------------------------- device calls
def eval_cost_tables(problem, d_image, d_cand, n_cand, d_tables, d_debug=None, stream=None, first=0, count=None):
    count = int(n_cand) - int(first) if count is None else count
    _check(lib().hapmoe_eval_cost_tables(_hp(problem).ref, _dptr(d_image), _dptr(d_cand), int(n_cand), int(first),
                                         int(count), _dptr(d_tables), _nbytes(d_tables), _dptr(d_debug),
                                         _nbytes(d_debug), _stream(stream)), "hapmoe_eval_cost_tables")


def stage_dp_ws_bytes(problem) -> int:
    n = C.c_int64(0)
    _check(lib().hapmoe_stage_dp_ws_bytes(_hp(problem).ref, C.byref(n)), "hapmoe_stage_dp_ws_bytes")
    return n.value


def stage_dp(problem, d_image, d_cand, n_cand, d_tables, first, count, d_res, d_ws, d_stats=None, stream=None):
    _check(lib().hapmoe_stage_dp(_hp(problem).ref, _dptr(d_image), _dptr(d_cand), int(n_cand), _dptr(d_tables),
                                 _nbytes(d_tables), int(first), int(count), _dptr(d_res), _dptr(d_stats),
                                 _dptr(d_ws), _nbytes(d_ws), _stream(stream)), "hapmoe_stage_dp")


def stage_dp_1f1b(problem, d_image, d_cand, n_cand, d_tables, first, count, d_res, d_ws, d_stats=None,
                  stream=None):
    _check(lib().hapmoe_stage_dp_1f1b(_hp(problem).ref, _dptr(d_image), _dptr(d_cand), int(n_cand),
                                      _dptr(d_tables), _nbytes(d_tables), int(first), int(count), _dptr(d_res),
                                      _dptr(d_stats), _dptr(d_ws), _nbytes(d_ws), _stream(stream)),
           "hapmoe_stage_dp_1f1b")


def stage_dp_latency(problem, d_image, d_cand, n_cand, d_tables, first, count, d_res, d_stats=None, stream=None):
    """The least 1F1B latency over every partition (no workspace)."""
    _check(lib().hapmoe_stage_dp_latency(_hp(problem).ref, _dptr(d_image), _dptr(d_cand), int(n_cand),
                                         _dptr(d_tables), _nbytes(d_tables), int(first), int(count), _dptr(d_res),
                                         _dptr(d_stats), _stream(stream)), "hapmoe_stage_dp_latency")


def stage_dp_types_ws_bytes(problem) -> int:
    n = C.c_int64(0)
    _check(lib().hapmoe_stage_dp_types_ws_bytes(_hp(problem).ref, C.byref(n)), "hapmoe_stage_dp_types_ws_bytes")
    return n.value


def stage_dp_types(problem, d_image, d_cand, n_cand, d_tables, first, count, d_res, d_types, d_ws, d_stats=None,
                   stream=None):
    _check(lib().hapmoe_stage_dp_types(_hp(problem).ref, _dptr(d_image), _dptr(d_cand), int(n_cand),
                                       _dptr(d_tables), _nbytes(d_tables), int(first), int(count), _dptr(d_res),
                                       _dptr(d_types), _dptr(d_stats), _dptr(d_ws), _nbytes(d_ws), _stream(stream)),
           "hapmoe_stage_dp_types")


def stage_dp_types_1f1b(problem, d_image, d_cand, n_cand, d_tables, first, count, d_res, d_types, d_ws,
                        d_stats=None, stream=None):
    _check(lib().hapmoe_stage_dp_types_1f1b(_hp(problem).ref, _dptr(d_image), _dptr(d_cand), int(n_cand),
                                            _dptr(d_tables), _nbytes(d_tables), int(first), int(count),
                                            _dptr(d_res), _dptr(d_types), _dptr(d_stats), _dptr(d_ws),
                                            _nbytes(d_ws), _stream(stream)), "hapmoe_stage_dp_types_1f1b")


def stage_dp_widths_ws_bytes(problem, count) -> int:
    n = C.c_int64(0)
    _check(lib().hapmoe_stage_dp_widths_ws_bytes(_hp(problem).ref, int(count), C.byref(n)),
           "hapmoe_stage_dp_widths_ws_bytes")
    return n.value


def stage_dp_widths(problem, d_image, d_cand, n_cand, d_tables, first, count, d_res, d_types, d_widths, d_ws,
                    d_stats=None, stream=None):
    _check(lib().hapmoe_stage_dp_widths(_hp(problem).ref, _dptr(d_image), _dptr(d_cand), int(n_cand),
                                        _dptr(d_tables), _nbytes(d_tables), int(first), int(count), _dptr(d_res),
                                        _dptr(d_types), _dptr(d_widths), _dptr(d_stats), _dptr(d_ws), _nbytes(d_ws),
                                        _stream(stream)), "hapmoe_stage_dp_widths")


def _plan_dict(plan):
    pp = plan.n_stages
    return {"instance": plan.instance, "objective": plan.objective, "stage_sum": plan.stage_sum,
            "t_max": plan.t_max, "dp_const": plan.dp_const,
            "config": tuple(plan.cand[:6]), "order": plan.cand[6], "n_micro": plan.cand[7],
            "layers": list(plan.layers[:pp]), "stage_types": list(plan.stage_types[:pp]),
            "recompute": [(plan.recompute_mask >> i) & 1 for i in range(pp)]}


def best_plan(problem, d_cand, d_tables, d_res, n, d_ws, d_config_best=None, stream=None, d_types=None) -> dict:
    plan = Plan()
    _check(lib().hapmoe_best_plan(_hp(problem).ref, _dptr(d_cand), _dptr(d_tables), _nbytes(d_tables),
                                  _dptr(d_res), _dptr(d_types), int(n), _dptr(d_config_best), _dptr(d_ws), _nbytes(d_ws),
                                  C.byref(plan), _stream(stream)), "hapmoe_best_plan")
    return _plan_dict(plan)


BEST_PLAN_SCRATCH_BYTES = 262144   # HAPMOE_BEST_PLAN_SCRATCH_BYTES


def best_plan_noalloc(problem, d_cand, d_tables, d_res, n, d_config_best=None, stream=None, d_types=None) -> dict:
    """hapmoe_best_plan_noalloc: the same arg-min with the library's own fixed workspace."""
    plan = Plan()
    _check(lib().hapmoe_best_plan_noalloc(_hp(problem).ref, _dptr(d_cand), _dptr(d_tables), _nbytes(d_tables),
                                          _dptr(d_res), _dptr(d_types), int(n), _dptr(d_config_best), C.byref(plan),
                                          _stream(stream)), "hapmoe_best_plan_noalloc")
    return _plan_dict(plan)


class Planner:
    """Device-resident pipeline: enumerate -> cost tables -> stage DP -> best plan.

    Buffers are torch tensors on ``device``; the problem image and candidate
    array are uploaded once, so repeated ``run()`` calls start from inputs
    resident in HBM.
    """

    def __init__(self, problem: dict, device="cuda:0", debug=False):
        import torch
        self.torch = torch
        self.problem = problem
        self.hp = HostProblem(problem)
        validate(self.hp)
        self.device = torch.device(device)
        self.cand_host = enumerate_candidates(self.hp)
        self.n = len(self.cand_host)
        u8 = dict(dtype=torch.uint8, device=self.device)
        self.d_image = torch.from_numpy(pack_image(self.hp)).to(self.device)
        self.d_cand = torch.from_numpy(self.cand_host.view(np.uint8)).to(self.device)
        self.d_tables = torch.empty(tables_bytes(self.hp), **u8)
        self.d_debug = torch.empty(debug_bytes(self.hp) // 8, dtype=torch.float64, device=self.device) if debug else None
        self.d_res = torch.empty(max(self.n, 1) * RESULT_DTYPE.itemsize, **u8)
        self.d_stats = None
        self.d_ws = torch.empty(best_plan_ws_bytes(self.hp, max(self.n, 1)), **u8)
        # stage_types = 2: the device-count DP, which also returns each candidate's stage types;
        # 3: per-stage widths, which return the stage types and widths
        self.device_count_dp = int(problem["space"].get("stage_types", 0)) == 2
        self.width_dp = int(problem["space"].get("stage_types", 0)) == 3
        self.d_widths = None
        if self.device_count_dp:
            self.d_dp_ws = torch.empty(stage_dp_types_ws_bytes(self.hp), **u8)
            self.d_types = torch.zeros(max(self.n, 1) * MAX_STAGES, **u8)
        elif self.width_dp:
            self.d_dp_ws = torch.empty(stage_dp_widths_ws_bytes(self.hp, max(self.n, 1)), **u8)
            self.d_types = torch.zeros(max(self.n, 1) * MAX_STAGES, **u8)
            self.d_widths = torch.zeros(max(self.n, 1) * MAX_STAGES, **u8)
        else:
            self.d_dp_ws = torch.empty(stage_dp_ws_bytes(self.hp), **u8)
            self.d_types = None
        n_cfg = tables_layout(self.hp)["n_configs"]
        self.n_configs = n_cfg
        self.d_config_best = torch.empty(max(n_cfg, 1), dtype=torch.int64, device=self.device)

    def eval_cost_tables(self, stream=None, first=0, count=None):
        eval_cost_tables(self.hp, self.d_image, self.d_cand, self.n, self.d_tables, self.d_debug, stream, first,
                         count)

    def stage_dp(self, first=0, count=None, stats=False, stream=None, objective="threshold"):
        """objective "threshold": sum + (B-1) max (hapmoe_stage_dp); "1f1b": the
        appendix's 1F1B latency over the Pareto frontier (hapmoe_stage_dp_1f1b);
        "latency": the least 1F1B latency over every partition
        (hapmoe_stage_dp_latency)."""
        if objective not in ("threshold", "1f1b", "latency"):
            raise ValueError(objective)
        count = self.n - first if count is None else count
        d_stats = None
        if stats:
            d_stats = self.torch.zeros(4 * max(self.n, 1), dtype=self.torch.int32, device=self.device)
            self.d_stats = d_stats
        res = self.d_res[first * RESULT_DTYPE.itemsize:]
        st = None if d_stats is None else d_stats[4 * first:]
        if objective == "latency":
            if self.width_dp or self.device_count_dp:
                raise ValueError("least latency: stage_types 0 or 1 only")
            stage_dp_latency(self.hp, self.d_image, self.d_cand, self.n, self.d_tables, first, count, res, st, stream)
            return
        if self.width_dp:
            if objective != "threshold":
                raise ValueError("per-stage widths: threshold objective only")
            stage_dp_widths(self.hp, self.d_image, self.d_cand, self.n, self.d_tables, first, count, res,
                            self.d_types[first * MAX_STAGES:], self.d_widths[first * MAX_STAGES:], self.d_dp_ws, st,
                            stream)
            return
        if self.device_count_dp:
            call = stage_dp_types if objective == "threshold" else stage_dp_types_1f1b
            call(self.hp, self.d_image, self.d_cand, self.n, self.d_tables, first, count, res,
                 self.d_types[first * MAX_STAGES:], self.d_dp_ws, st, stream)
            return
        call = stage_dp if objective == "threshold" else stage_dp_1f1b
        call(self.hp, self.d_image, self.d_cand, self.n, self.d_tables, first, count, res, self.d_dp_ws, st, stream)

    def best_plan(self, stream=None):
        plan = best_plan(self.hp, self.d_cand, self.d_tables, self.d_res, self.n, self.d_ws, self.d_config_best,
                         stream, self.d_types)
        if self.width_dp:
            self.torch.cuda.synchronize(self.device)
            i = plan["instance"]
            plan["widths"] = [int(x) for x in self.d_widths[i * MAX_STAGES:i * MAX_STAGES + len(plan["layers"])].cpu()]
        return plan

    def run(self, stats=False, stream=None, objective="threshold"):
        self.eval_cost_tables(stream)
        self.stage_dp(stats=stats, stream=stream, objective=objective)
        return self.best_plan(stream)

    # ---- host copies for checks ----
    def results(self) -> np.ndarray:
        self.torch.cuda.synchronize(self.device)
        return self.d_res.cpu().numpy()[: self.n * RESULT_DTYPE.itemsize].view(RESULT_DTYPE)

    def widths(self) -> np.ndarray:
        """Per-stage widths: the half-groups of every stage of every candidate, [n][32]."""
        self.torch.cuda.synchronize(self.device)
        return self.d_widths.cpu().numpy()[: self.n * MAX_STAGES].reshape(-1, MAX_STAGES)

    def stage_types(self) -> np.ndarray:
        """Device-count DP: the stage type masks of every candidate, [n][32]."""
        self.torch.cuda.synchronize(self.device)
        return self.d_types.cpu().numpy()[: self.n * MAX_STAGES].reshape(-1, MAX_STAGES)

    def stats(self) -> np.ndarray:
        self.torch.cuda.synchronize(self.device)
        return self.d_stats.cpu().numpy().reshape(-1, 4)[: self.n]

    def tables(self) -> np.ndarray:
        self.torch.cuda.synchronize(self.device)
        return self.d_tables.cpu().numpy()

    def debug(self) -> np.ndarray:
        self.torch.cuda.synchronize(self.device)
        return self.d_debug.cpu().numpy()

    def config_best(self) -> np.ndarray:
        self.torch.cuda.synchronize(self.device)
        return self.d_config_best.cpu().numpy()[: self.n_configs]
