"""The knob search tool: candidate values stay inside the tuning fields'
valid ranges (CPU), its oracle reference names its workload (CPU), and a
short search on the tiny shape runs end to end, gating every candidate on
the oracle's result, timing and reporting it (GPU)."""
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


def test_reference_file_names_its_workload(tmp_path):
    """The oracle's reference file carries its workload; the search refuses
    a reference of another workload (CPU)."""
    import numpy as np
    from oracle import reference
    path = reference.write("tiny", "bf16", 3, str(tmp_path / "ref.npz"))
    tok, lg = tune.load_reference(path, "tiny_bf16_pos3")
    assert lg.shape == (512 * 8,) and tok == int(np.argmax(lg))
    with pytest.raises(ValueError):
        tune.load_reference(path, "tiny_bf16_pos4")


@pytest.mark.gpu
def test_search_is_gated_on_the_oracle(capsys, torch_cuda, tmp_path):
    """Every configuration the search times first reproduces the oracle's
    token and logits; with a reference whose greedy token is wrong even the
    default configuration fails the gate and nothing is timed or kept."""
    import numpy as np
    from oracle import reference
    ref = reference.write("tiny", "bf16", 3, str(tmp_path / "ref.npz"))
    assert tune.main(["--config", "tiny", "--pos", "3", "--pairs", "3", "--reference", ref]) == 0
    lines = [json.loads(x) for x in capsys.readouterr().out.splitlines() if x.startswith("{")]
    assert lines[-1]["workload"] == "tiny_bf16_pos3" and "best" in lines[-1]
    results = [d["result"] for d in lines[:-1]]
    assert set(results) <= {"kept", "reverted", "rejected"} and len(results) >= 10
    assert any(d["knobs"].get("queue_assign") == 1 for d in lines[:-1])
    assert all(d["max_abs_logit_diff"] <= tune.TOL for d in lines[:-1] if "max_abs_logit_diff" in d)
    assert all(not d.get("below_floor", False) for d in lines[:-1])
    # a wrong reference: the oracle's logits with another row made the maximum
    with np.load(ref) as z:
        lg = z["logits"].copy()
        lg[(int(z["token"]) + 1) % lg.size] = lg.max() + 1.0
        np.savez(tmp_path / "bad.npz", logits=lg, token=np.int64((int(z["token"]) + 1) % lg.size),
                 workload=z["workload"])
    assert tune.main(["--config", "tiny", "--pos", "3", "--pairs", "3", "--reference",
                      str(tmp_path / "bad.npz")]) == 3
    lines = [json.loads(x) for x in capsys.readouterr().out.splitlines() if x.startswith("{")]
    assert [d["result"] for d in lines] == ["baseline_wrong"]
