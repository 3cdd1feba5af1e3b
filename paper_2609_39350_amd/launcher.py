"""Plan materialisation text (Section 4, plan materialisation): a chosen plan
as Megatron-LM style launcher settings.

The standard knobs (PP, TP, CP, EP, TPE, and DP through the batch sizes) become
the usual Megatron-LM flags; the heterogeneous parts of the plan -- the
non-uniform layer split, the device type of every stage and the per-stage
recomputation choice -- are written as explicit per-stage lists for the launcher
that builds the process mesh.  Pure host-side formatting of a result; nothing
here evaluates the cost model.
"""
from __future__ import annotations


def _types(mask: int) -> list[int]:
    return [h for h in range(8) if (mask >> h) & 1]


def plan_to_launcher(problem: dict, plan: dict) -> str:
    """Shell-style text for ``plan`` (a dict as returned by ``Planner.best_plan``)."""
    m = problem["model"]
    pp, tp, cp, dp, ep, tpe = (int(x) for x in plan["config"])
    layers = [int(n) for n in plan["layers"]]
    if len(layers) != pp or sum(layers) != int(m["n_layers"]):
        raise ValueError("plan layers do not partition the model")
    B = int(plan["n_micro"])
    mbs = int(m["micro_batch_size"])
    flags = [
        f"--num-layers {int(m['n_layers'])}",
        f"--hidden-size {int(m['hidden'])}",
        f"--seq-length {int(m['seq_len'])}",
        f"--tensor-model-parallel-size {tp}",
        f"--pipeline-model-parallel-size {pp}",
        f"--context-parallel-size {cp}",
        f"--micro-batch-size {mbs}",
        f"--global-batch-size {B * mbs * dp}",
    ]
    if int(m["n_experts"]) > 0:
        flags += [f"--num-experts {int(m['n_experts'])}", f"--moe-router-topk {int(m['top_k'])}",
                  f"--expert-model-parallel-size {ep}", f"--expert-tensor-parallel-size {tpe}"]
    starts = [sum(layers[:i]) for i in range(pp)]
    rows = []
    for i in range(pp):
        types = _types(int(plan["stage_types"][i]))
        rows.append(f"#  {i:3d}  {starts[i]:4d}-{starts[i] + layers[i] - 1:<4d} {layers[i]:4d}  "
                    f"{','.join(str(h) for h in types):>8s}  {'yes' if plan['recompute'][i] else 'no'}")
    lines = [
        f"# plan: candidate {plan['instance']}, device-type ordering {plan['order']}, "
        f"{B} micro-batches of {mbs}",
        f"# predicted iteration latency {plan['objective']} ns "
        f"(stage sum {plan['stage_sum']}, largest stage {plan['t_max']}, DP sync + optimizer {plan['dp_const']})",
        "# stage  layers     count     types  recompute",
        *rows,
        "MEGATRON_ARGS=\"" + " ".join(flags) + "\"",
        "# non-uniform pipeline split: layers held by each stage, in pipeline order",
        "PIPELINE_STAGE_LAYERS=\"" + ",".join(str(n) for n in layers) + "\"",
        "# device type(s) of each stage's device group (several: the group straddles types)",
        "PIPELINE_STAGE_DEVICE_TYPES=\"" + ";".join(
            ",".join(str(h) for h in _types(int(t))) for t in plan["stage_types"][:pp]) + "\"",
        "# stage-wise recomputation: 1 = recompute the stage's activations in the backward pass",
        "PIPELINE_STAGE_RECOMPUTE=\"" + ",".join(str(int(r)) for r in plan["recompute"][:pp]) + "\"",
        f"# data-parallel replicas per stage: {dp}",
    ]
    return "\n".join(lines) + "\n"
