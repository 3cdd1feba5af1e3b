"""Plan materialisation text: the knobs and per-stage lists of a plan."""
import pytest

from paper_2609_39350_amd import launcher, workloads


def _plan():
    return {"instance": 281, "objective": 4080259, "stage_sum": 2000000, "t_max": 900000, "dp_const": 1000,
            "config": (4, 2, 1, 1, 4, 1), "order": 1, "n_micro": 8,
            "layers": [2, 1, 3, 2], "stage_types": [1, 1, 3, 2], "recompute": [0, 1, 0, 0]}


def test_plan_text_has_the_knobs_and_lists():
    p = workloads.config(1)
    text = launcher.plan_to_launcher(p, _plan())
    assert "--pipeline-model-parallel-size 4" in text and "--tensor-model-parallel-size 2" in text
    assert "--expert-model-parallel-size 4" in text and "--expert-tensor-parallel-size 1" in text
    mbs = p["model"]["micro_batch_size"]
    assert f"--global-batch-size {8 * mbs * 1}" in text
    assert 'PIPELINE_STAGE_LAYERS="2,1,3,2"' in text
    assert 'PIPELINE_STAGE_DEVICE_TYPES="0;0;0,1;1"' in text
    assert 'PIPELINE_STAGE_RECOMPUTE="0,1,0,0"' in text
    # stage rows: first and last layer of every stage
    assert "#    2     3-5" in text


def test_plan_text_rejects_a_bad_partition():
    p = workloads.config(1)
    bad = dict(_plan(), layers=[2, 1, 3, 1])
    with pytest.raises(ValueError):
        launcher.plan_to_launcher(p, bad)
