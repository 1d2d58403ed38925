"""The knob search tool: candidate values stay inside the tuning fields'
valid ranges (CPU), and a short search on the tiny shape runs end to end,
gating, timing and reporting every candidate (GPU)."""
import json

import pytest

from paper_2606_09682_amd import amk, tune


@pytest.mark.parametrize("pos", [0, 5, 300, 8192])
def test_candidates_are_valid_tunings(pos):
    for knob in tune.KNOBS:
        vals = tune.candidates(knob, 0, pos)
        assert vals and 0 not in vals
        for v in vals:
            if knob == "attn_splits":
                assert 1 <= v <= 64
            elif knob == "max_rows_per_task":
                assert 2 <= v <= 1024
            elif knob == "tiny_context":
                assert v <= amk.AMK_TINY_MAX
            t = tune.tuning_of(amk, {knob: v})
            assert getattr(t, knob) == v


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    return torch


@pytest.mark.gpu
def test_search_runs_on_tiny(capsys, torch_cuda):
    assert tune.main(["--config", "tiny", "--pos", "3", "--pairs", "3"]) == 0
    lines = [json.loads(x) for x in capsys.readouterr().out.splitlines() if x.startswith("{")]
    assert lines[-1]["workload"] == "tiny_bf16_pos3" and "best" in lines[-1]
    results = {d["result"] for d in lines[:-1]}
    assert results <= {"kept", "reverted", "rejected", "wrong"} and "wrong" not in results
    assert all(not d.get("below_floor", False) for d in lines[:-1])
