"""Write the oracle's result for one decode workload to a file (TEST
INFRASTRUCTURE ONLY: run by hand or by the tests, never by the library).

The knob search (``paper_2606_09682_amd.tune``) accepts a configuration only
if its step reproduces the oracle: the same greedy token and every logit
within 2e-2.  The search must not run the oracle itself, so it reads the
oracle's result from the ``.npz`` file this script writes:

    python -m oracle.reference --config llama3_8b --fmt bf16 --pos 0 --out ref.npz

The workload is the synthetic one every test and the benchmark use: seeded
weights (seed 0) of the named shape in the named format, token 1 at
position ``pos`` with KV slots [0, pos) filled N(0, 1) (seed 1) in a cache of
pos + 2 positions.  The file holds ``logits`` (float32 [vocab]), ``token``
and ``workload`` (a string naming config, format and position).
"""
from __future__ import annotations

import argparse
import os
import sys
from typing import List, Optional

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def workload_name(config: str, fmt: str, pos: int) -> str:
    return f"{config}_{fmt}_pos{pos}"


def write(config: str, fmt: str, pos: int, out: str) -> str:
    import synth

    from .decode import OracleModel, argmax_first, decode_step

    shape = synth.get(config)
    w = synth.make_weights(shape, seed=0)
    if fmt == "w8a16":
        synth.add_w8a16(w)
    elif fmt == "w4a16":
        synth.add_w4a16(w)
    kv = synth.make_kv_cache(shape, pos, seed=1, max_seq=pos + 2)
    model = OracleModel(w, fmt, np.float32, cache=shape.hidden <= 2048)
    logits = decode_step(model, 1, pos, kv)
    np.savez(out, logits=logits.astype(np.float32), token=np.int64(argmax_first(logits)),
             workload=np.array(workload_name(config, fmt, pos)))
    return out


def main(argv: Optional[List[str]] = None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", default="llama3_8b")
    ap.add_argument("--fmt", default="bf16", choices=["bf16", "w8a16", "w4a16"])
    ap.add_argument("--pos", type=int, default=0)
    ap.add_argument("--out", required=True)
    a = ap.parse_args(argv)
    print(write(a.config, a.fmt, a.pos, a.out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
