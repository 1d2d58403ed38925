"""Benchmark: batch-1 decode µs/token and achieved HBM GB/s of the megakernel.

Workload (default): Llama-3-8B-shaped decoder (hidden 4096, 32 layers, 32/8
heads, head_dim 128, SwiGLU 14336, vocab 128256, untied), seeded random bf16
weights N(0, 0.02), one decode step of token 1 at position 0.  Variants in
the same run: W8A16 at position 0 and both formats at position 8192 (KV cache
filled N(0, 1) bf16).  Every variant is correctness-gated against the CPU
oracle before its time is reported.

A step = one amk_decode_step (one cooperative launch: the whole decode hot
path).  Inputs are resident in HBM before timing starts; the timed region is
K back-to-back steps bracketed by torch.cuda.synchronize().
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0  # MI355X HBM3E peak


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in ("megakernel.hip", "device.h", "schedule.cpp", "schedule.h", "api.cpp"):
        with open(os.path.join(ROOT, "paper_2606_09682_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def counter_traffic(workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"megakernel_{workload}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"kernel_source_hash:\s*([0-9a-f]+)", text)
    b = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m or not b or m.group(1) != kernel_source_hash():
        return None
    return float(b.group(1))


def blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        return max((i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"), default=1)
    except Exception:
        return os.cpu_count() or 1


def run_variant(amk, torch, w, fmt, pos, steps, warmup, check=True):
    import oracle
    import synth
    from synth.device import config_kwargs, kv_to_device, weights_to_device

    cfg = w.cfg
    max_seq = pos + 2
    log(f"variant {cfg.name} {fmt} pos {pos}: upload")
    tensors = weights_to_device(w, fmt)
    kv_np = synth.make_kv_cache(cfg, pos, seed=1, max_seq=max_seq)
    dec = amk.Decoder(amk.make_config(**config_kwargs(cfg, fmt, max_seq)), tensors)
    kv = kv_to_device(kv_np)
    logits = torch.empty(cfg.vocab, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    # correctness gate (also the CPU-oracle timing sample)
    res = {"fmt": fmt, "pos": pos}
    dec.step(1, pos, kv, logits)
    tok = dec.next_token()
    if check:
        log(f"variant {fmt} pos {pos}: oracle step")
        model = oracle.OracleModel(w, fmt, np.float32, cache=False)
        kv_ref = kv_np.copy()
        t0 = time.perf_counter()
        ref_logits = oracle.decode_step(model, 1, pos, kv_ref)
        cpu_s = time.perf_counter() - t0
        ref_tok = oracle.argmax_first(ref_logits)
        err = float(np.max(np.abs(logits.cpu().numpy().astype(np.float64) - ref_logits)))
        res.update(oracle_s=cpu_s, max_abs_logit_err=err, token=tok, oracle_token=ref_tok,
                   correct=bool(tok == ref_tok and err <= 2e-2))
        log(f"variant {fmt} pos {pos}: token {tok} oracle {ref_tok} err {err:.2e} oracle {cpu_s:.1f}s")
    else:
        res.update(correct=None)

    for _ in range(warmup):
        dec.step(1, pos, kv, logits)
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        starts[i].record(stream)
        dec.step(1, pos, kv, logits)
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    launch_us = np.array([s.elapsed_time(e) * 1e3 for s, e in zip(starts, ends)])
    status = dec.status()
    dec.close()
    del tensors
    torch.cuda.empty_cache()
    nbytes = cfg.algorithmic_bytes(fmt, pos)
    med = float(np.median(launch_us))
    res.update(status=status, wall_us_per_step=wall / steps * 1e6, launch_us_median=med,
               launch_us_mean=float(np.mean(launch_us)), launch_us_p10=float(np.percentile(launch_us, 10)),
               launch_us_p90=float(np.percentile(launch_us, 90)), algorithmic_bytes=nbytes,
               achieved_gbs=nbytes / (float(np.mean(launch_us)) * 1e-6) / 1e9,
               floor_us=nbytes / (PEAK_HBM_GBS * 1e9) * 1e6)
    res["floor_ratio"] = res["launch_us_mean"] / res["floor_us"]
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="llama3_8b")
    ap.add_argument("--variants", default="all", help="'all' or 'main' (bf16 at position 0 only)")
    ap.add_argument("--no-check", action="store_true", help="skip the oracle gate (profiling runs)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES (counter calibration) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU; --gpus {args.gpus} is not supported by this build "
              f"(the decode step is a single-GPU kernel)", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_probe:
        # a plain copy kernel of known traffic: reads and writes BYTES once per launch
        torch.cuda.set_device(0)
        n = args.copy_probe // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": args.copy_probe, "launches": 3}), flush=True)
        return

    import synth
    from paper_2606_09682_amd import amk

    amk.load()
    torch.cuda.set_device(0)
    cfg = synth.get(args.config)
    log(f"generating {cfg.name} weights (seed 0)")
    t0 = time.perf_counter()
    w = synth.make_weights(cfg, seed=0)
    log(f"weights in {time.perf_counter() - t0:.1f}s")
    variants = [("bf16", cfg.positions[0])]
    if args.variants == "all":
        variants += [("w8a16", cfg.positions[0])] + [(f, cfg.positions[-1]) for f in ("bf16", "w8a16")
                                                      if cfg.positions[-1] != cfg.positions[0]]
    results = []
    for fmt, pos in variants:
        if fmt == "w8a16" and not w.q8:
            t0 = time.perf_counter()
            synth.add_w8a16(w)
            log(f"quantised in {time.perf_counter() - t0:.1f}s")
        results.append(run_variant(amk, torch, w, fmt, pos, args.steps, args.warmup, check=not args.no_check))
        if results[-1].get("correct") is False or results[-1]["status"] != 0:
            log(f"variant {fmt} pos {pos} FAILED its correctness gate: {results[-1]}")
    main_res = results[0]
    ok = all(r.get("correct") is not False and r["status"] == 0 for r in results)
    workload = f"{cfg.name}_bf16_pos{cfg.positions[0]}"
    traffic = counter_traffic(workload)
    out = {
        "metric": "µs/token batch-1 decode + achieved HBM GB/s vs weights/BW floor (bf16, W8A16)",
        "value": main_res["wall_us_per_step"] if ok else None,
        "unit": "µs/token",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_res["wall_us_per_step"] / 1e3,
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded random weights at the model's shapes, N(0,0.02) bf16)",
        "config": {"workload": workload, "model_shape": cfg.name, "batch": 1, "position": cfg.positions[0],
                   "weights": "bf16", "parallelism": "single GPU"},
        "correct": ok,
        "roofline": {"bound": "hbm", "achieved": main_res["achieved_gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": main_res["achieved_gbs"] / PEAK_HBM_GBS,
                     "traffic": traffic},
        "cpu_baseline": None,
        "variants": [{k: (round(v, 3) if isinstance(v, float) else v) for k, v in r.items()} for r in results],
    }
    if "oracle_s" in main_res:
        out["cpu_baseline"] = {"value": main_res["oracle_s"] * 1e6, "unit": "µs/token", "cores": blas_threads(),
                               "kind": "oracle",
                               "sample": f"one full decode step of {workload} (numpy fp32, weights decoded "
                                         f"from bf16 per use)"}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
