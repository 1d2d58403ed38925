"""The oracle still reproduces the stored tiny-decoder greedy run (drift pin)."""
import json
import os

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tiny_greedy.json")


@pytest.mark.parametrize("fmt", ["bf16", "w8a16"])
def test_oracle_reproduces_golden(tiny_cfg, tiny_weights, fmt):
    with open(GOLDEN) as f:
        g = json.load(f)
    assert g["generator"] == synth.GENERATOR_VERSION
    kv = synth.make_kv_cache(tiny_cfg, 0)
    toks, logits = oracle.greedy(oracle.OracleModel(tiny_weights, fmt, np.float32), 1, 0, g["steps"], kv)
    assert toks == g["results"][fmt]["tokens"]
    np.testing.assert_allclose(logits[0][:8], g["results"][fmt]["first_logits_head"], atol=1e-5)
