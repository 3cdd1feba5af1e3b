"""A 32-bit digest of a stage-DP result, for comparing GPU results with stored
oracle references.  Test infrastructure: it holds none of the method's
arithmetic and serves both sides alike."""
import numpy as np

INF = np.iinfo(np.int64).max
_M = np.uint64(0x9E3779B97F4A7C15)


def _mix(h, x):
    with np.errstate(over="ignore"):
        h = (h ^ x.astype(np.uint64)) * _M
        return h ^ (h >> np.uint64(29))


def digest(status, objective, stage_sum, t_max, recompute_mask, layers, stage_types=None, widths=None):
    """status/objective/stage_sum/t_max/recompute_mask: [n]; layers (and the
    optional stage type masks and per-stage widths): [n][32] uint8, zero past
    the last stage.  A result that is not feasible digests its status only."""
    status = np.asarray(status, dtype=np.int64)
    ok = status == 0
    fields = [status, np.where(ok, objective, 0), np.where(ok, stage_sum, 0), np.where(ok, t_max, 0),
              np.where(ok, recompute_mask, 0)]
    lw = np.ascontiguousarray(np.where(ok[:, None], layers, 0).astype(np.uint8)).view(np.uint64)
    fields += [lw[:, k] for k in range(lw.shape[1])]
    for extra in (stage_types, widths):
        if extra is not None:
            tw = np.ascontiguousarray(np.where(ok[:, None], extra, 0).astype(np.uint8)).view(np.uint64)
            fields += [tw[:, k] for k in range(tw.shape[1])]
    h = np.full(len(status), np.uint64(0x243F6A8885A308D3))
    for f in fields:
        h = _mix(h, np.asarray(f).astype(np.int64).view(np.uint64))
    return (h >> np.uint64(32)).astype(np.uint32)


def of_oracle(results, with_types=False, with_widths=False):
    """Digests of a list of oracle result dictionaries (orc.Oracle.solve*)."""
    n = len(results)
    layers = np.zeros((n, 32), dtype=np.uint8)
    types = np.zeros((n, 32), dtype=np.uint8)
    widths = np.zeros((n, 32), dtype=np.uint8)
    st, obj, sm, tm, rm = (np.zeros(n, dtype=np.int64) for _ in range(5))
    for k, r in enumerate(results):
        st[k] = 0 if r["status"] == 0 else 1
        if r["status"] == 0:
            obj[k], sm[k], tm[k] = r["opt"], r["sum"], r["tmax"]
            rm[k] = sum(int(v) << i for i, v in enumerate(r["recompute"]))
            layers[k, :r["pp"]] = r["layers"]
            types[k, :r["pp"]] = r["stage_mask"]
            if with_widths:
                widths[k, :r["pp"]] = r["width"]
    return digest(st, obj, sm, tm, rm, layers, types if with_types else None, widths if with_widths else None)


def of_gpu(res, idx, types=None, widths=None):
    """Digests of GPU results (binding.RESULT_DTYPE records) at indices idx;
    types: the [n][32] stage type masks (device-count DP, per-stage widths);
    widths: the per-stage widths DP's [n][32] widths."""
    r = res[idx]
    st = np.where(r["status"] == 0, 0, np.where(r["status"] == 1, 1, 2))
    return digest(st, r["objective"], r["stage_sum"], r["t_max"], r["recompute_mask"], r["layers"],
                  None if types is None else types[idx], None if widths is None else widths[idx])
