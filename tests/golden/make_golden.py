"""Write tests/golden/tiny_greedy.json from the CPU oracle alone.

The paper prints no worked example (no token ids, logits or weights), so the
stored values here come from the oracle on the tiny seeded decoder (hidden
256, 4 layers, 4/2 heads, head_dim 64, SwiGLU 688, vocab 4096, weight seed 0):
8 greedy steps from token 1 at position 0 with the bf16 KV cache, for the bf16
weights and the W8A16 weights.  They pin the oracle against later drift; the
oracle itself is pinned by the closed-form and transformers tests.

Run:  python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
import synth  # noqa: E402


def main():
    cfg = synth.get("tiny")
    w = synth.add_w8a16(synth.make_weights(cfg, seed=0))
    out = {"config": "tiny", "weight_seed": 0, "generator": synth.GENERATOR_VERSION,
           "start_token": 1, "start_pos": 0, "steps": cfg.greedy_steps, "results": {}}
    for fmt in ("bf16", "w8a16"):
        kv = synth.make_kv_cache(cfg, 0)
        toks, logits = oracle.greedy(oracle.OracleModel(w, fmt, np.float64), 1, 0, cfg.greedy_steps, kv)
        out["results"][fmt] = {
            "tokens": toks,
            "first_logits_head": [float(v) for v in logits[0][:8]],
            "margins": [oracle.top2_margin(l) for l in logits],
        }
    with open(os.path.join(HERE, "tiny_greedy.json"), "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
