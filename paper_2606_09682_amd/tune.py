"""Knob search for one decode workload: the schedule knobs of amk_tuning_t
(attention splits, rows per task, the short / tiny schedule crossovers, the
round-robin or LPT queue assignment) are tried one at a time around the
current best, each candidate

* gated on correctness against the CPU oracle: the same greedy token and
  every logit within 2e-2 of the oracle's result for the same inputs, read
  from the file ``python -m oracle.reference`` writes (the search never runs
  the oracle itself); the default configuration must pass the same gate
  before anything is timed,
* timed paired and interleaved with the current best (A, B, A, B, ...
  launches on one stream, per-pair time ratios, median and p10 / p90), so a
  clock ramp affects both alike,
* guarded against the physical floor (no launch may beat the bytes / 8 TB/s
  time), and
* kept only if the median ratio is below 1 - min_gain (paper §3, the
  propose -> evaluate -> keep / revert loop, here without an agent).

    python -m oracle.reference --config llama3_8b --fmt bf16 --pos 1024 --out ref.npz
    python -m paper_2606_09682_amd.tune --config llama3_8b --fmt bf16 --pos 1024 --reference ref.npz

Prints one JSON line per candidate and a final line with the best tuning.
Seeded synthetic weights and KV cache of the named shape; one GPU.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
from typing import Dict, List, Optional

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
KNOBS = ("attn_splits", "max_rows_per_task", "short_context", "tiny_context", "queue_assign")
TOL = 2e-2


def tuning_of(amk, knobs: Dict[str, int]):
    t = amk.amk_tuning_t()
    for k, v in knobs.items():
        setattr(t, k, int(v))
    return t


def candidates(knob: str, cur: int, pos: int) -> List[int]:
    """Neighbours of the current value (0 = the library default)."""
    if knob == "attn_splits":
        return [v for v in (8, 16, 24, 32, 48, 64) if v != cur]
    if knob == "max_rows_per_task":
        return [v for v in (64, 128, 256, 512, 1024) if v != cur]
    if knob == "short_context":
        # the step's position decides the schedule: bracket it
        return [v for v in (-1, max(1, pos // 2), pos + 1, 2 * (pos + 1)) if v != cur]
    if knob == "tiny_context":
        return [v for v in (-1, 1, 2, 4, 6, 8) if v != cur]
    if knob == "queue_assign":  # round robin (0, the default) or LPT (1)
        return [v for v in (0, 1) if v != cur]
    return []


def load_reference(path: str, workload: str):
    """(token, logits) of the oracle for `workload` from an oracle.reference file."""
    with np.load(path, allow_pickle=False) as z:
        if str(z["workload"]) != workload:
            raise ValueError(f"{path} holds {z['workload']}, the search runs {workload}")
        return int(z["token"]), z["logits"].astype(np.float64)


def paired(torch, dec_a, dec_b, step_a, step_b, pairs: int):
    """Per-pair launch times (us) of A and B, interleaved A B A B ..."""
    stream = torch.cuda.current_stream()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(pairs)]
    for i in range(pairs):
        e = ev[i]
        e[0].record(stream)
        step_a()
        e[1].record(stream)
        e[2].record(stream)
        step_b()
        e[3].record(stream)
    torch.cuda.synchronize()
    ta = np.array([e[0].elapsed_time(e[1]) * 1e3 for e in ev])
    tb = np.array([e[2].elapsed_time(e[3]) * 1e3 for e in ev])
    return ta, tb


def main(argv: Optional[List[str]] = None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", default="llama3_8b")
    ap.add_argument("--fmt", default="bf16", choices=["bf16", "w8a16", "w4a16"])
    ap.add_argument("--pos", type=int, default=0)
    ap.add_argument("--pairs", type=int, default=30)
    ap.add_argument("--min-gain", type=float, default=0.005)
    ap.add_argument("--rounds", type=int, default=1)
    ap.add_argument("--reference", required=True,
                    help="the oracle's result for this workload (python -m oracle.reference ... --out FILE)")
    args = ap.parse_args(argv)
    workload = f"{args.config}_{args.fmt}_pos{args.pos}"
    tok_ref, lg_ref = load_reference(args.reference, workload)

    import torch

    import synth
    from synth.device import config_kwargs, kv_to_device, weights_to_device
    from paper_2606_09682_amd import amk

    amk.load()
    torch.cuda.set_device(0)
    shape = synth.get(args.config)
    w = synth.make_weights(shape, seed=0)
    if args.fmt == "w8a16":
        synth.add_w8a16(w)
    elif args.fmt == "w4a16":
        synth.add_w4a16(w)
    tensors = weights_to_device(w, args.fmt)
    max_seq = args.pos + 2
    cfg = amk.make_config(**config_kwargs(shape, args.fmt, max_seq))
    kv_np = synth.make_kv_cache(shape, args.pos, seed=1, max_seq=max_seq)
    floor_us = shape.algorithmic_bytes(args.fmt, args.pos) / (PEAK_HBM_GBS * 1e9) * 1e6

    def make(knobs):
        try:
            return amk.Decoder(cfg, tensors, tuning_of(amk, knobs))
        except amk.AmkError as e:  # e.g. a schedule the checker rejects
            return e

    def run_once(dec, kv):
        logits = torch.empty(shape.vocab, dtype=torch.float32, device="cuda")
        dec.step(1, args.pos, kv, logits)
        return dec.next_token(), logits.cpu().numpy()

    def gate(tok, lg):
        err = float(np.max(np.abs(lg.astype(np.float64) - lg_ref)))
        return tok == tok_ref and err <= TOL, err

    best: Dict[str, int] = {}
    kv_best = kv_to_device(kv_np)
    dec_best = make(best)
    ok, err = gate(*run_once(dec_best, kv_best))
    if not ok:
        print(json.dumps({"knobs": best, "result": "baseline_wrong", "max_abs_logit_diff": err}), flush=True)
        dec_best.close()
        return 3
    for _ in range(args.rounds):
        for knob in KNOBS:
            for v in candidates(knob, best.get(knob, 0), args.pos):
                knobs = dict(best, **{knob: v})
                dec = make(knobs)
                rec = {"knobs": knobs}
                if isinstance(dec, Exception):
                    rec.update(result="rejected", why=str(dec))
                    print(json.dumps(rec), flush=True)
                    continue
                kv = kv_to_device(kv_np)
                tok, lg = run_once(dec, kv)
                ok, err = gate(tok, lg)
                if not ok:
                    rec.update(result="wrong", token=tok, ref_token=tok_ref, max_abs_logit_diff=err)
                    print(json.dumps(rec), flush=True)
                    dec.close()
                    continue
                logits = torch.empty(shape.vocab, dtype=torch.float32, device="cuda")
                sa = lambda: dec_best.step(1, args.pos, kv_best, logits)  # noqa: E731
                sb = lambda: dec.step(1, args.pos, kv, logits)  # noqa: E731
                paired(torch, dec_best, dec, sa, sb, 5)  # warm-up pairs
                ta, tb = paired(torch, dec_best, dec, sa, sb, args.pairs)
                ratio = tb / ta
                below = bool(min(ta.min(), tb.min()) < floor_us)
                keep = (not below) and float(np.median(ratio)) < 1.0 - args.min_gain
                rec.update(result="kept" if keep else "reverted", best_us=float(np.median(ta)),
                           cand_us=float(np.median(tb)), ratio_median=float(np.median(ratio)),
                           ratio_p10=float(np.percentile(ratio, 10)), ratio_p90=float(np.percentile(ratio, 90)),
                           below_floor=below, max_abs_logit_diff=err)
                print(json.dumps(rec), flush=True)
                if keep:
                    dec_best.close()
                    dec_best, kv_best, best = dec, kv, knobs
                else:
                    dec.close()
    logits = torch.empty(shape.vocab, dtype=torch.float32, device="cuda")
    ta, _ = paired(torch, dec_best, dec_best, lambda: dec_best.step(1, args.pos, kv_best, logits),
                   lambda: dec_best.step(1, args.pos, kv_best, logits), args.pairs)
    print(json.dumps({"best": best, "workload": workload,
                      "us_median": float(np.median(ta)), "floor_us": floor_us}), flush=True)
    dec_best.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
