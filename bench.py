"""Benchmark: batch-1 decode µs/token and achieved HBM GB/s of the megakernel.

Workload (default): Llama-3-8B-shaped decoder (hidden 4096, 32 layers, 32/8
heads, head_dim 128, SwiGLU 14336, vocab 128256, untied), seeded random bf16
weights N(0, 0.02), one decode step of token 1 at position 0.  Variants in
the same run: W8A16 and W4A16 (int4, fp16 scales per 128 columns) at
position 0 and all three formats at position 8192 (KV cache filled N(0, 1)
bf16).  Every variant is correctness-gated against the CPU oracle before its
time is reported.

A step = one amk_decode_step (one cooperative launch: the whole decode hot
path).  Inputs are resident in HBM before timing starts; the timed region is
K back-to-back steps bracketed by torch.cuda.synchronize() (default 25
warm-ups and 100 timed steps; median and p10/p90 of the per-launch times are
reported too).  Also reported: the whole-token host time including the
next-token readback, the device's streaming-read peak (amk_read_probe over
8 GiB), a flag for any time below the bandwidth floor, GPU clocks and power
from amd-smi when it is present (sampled by a background thread while the
timed steps run), the CPU oracle's time per step (median of 3, weights
decoded to fp32 before the timed region when host memory allows) on this
host, and a same-node PyTorch-ROCm reference (per-op eager and HIP-graph
replay of the same step, paper_2606_09682_amd.torch_baseline) for the bf16
and W8A16 variants, itself checked against the oracle.
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


def blas_info():
    """(threads, library) of the BLAS numpy uses here."""
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if info:
            return max(i.get("num_threads", 1) for i in info), info[0].get("internal_api", "?")
    except Exception:
        pass
    return os.cpu_count() or 1, "?"


def host_ram_gb():
    try:
        import psutil
        return round(psutil.virtual_memory().total / 2**30, 1)
    except Exception:
        return None


def smi_snapshot():
    """GPU clock and power lines from amd-smi, or None when it is absent."""
    import shutil
    import subprocess
    exe = shutil.which("amd-smi")
    if not exe:
        return None
    try:
        out = subprocess.run([exe, "metric", "-g", "0", "-c", "-p"], capture_output=True, text=True,
                             timeout=20).stdout
    except Exception:
        return None
    keep = [ln.strip() for ln in out.splitlines()
            if any(k in ln for k in ("GFX_0", "CLK:", "SOCKET_POWER", "POWER:", "MEM_0"))]
    return keep[:12] or None


class SmiSampler:
    """amd-smi snapshots taken by a background thread while the GPU works:
    start() begins sampling, stop() ends it and returns the snapshots (the
    caller keeps the GPU busy until enough were taken)."""

    def __init__(self):
        import threading
        self.samples = []
        self._stop = threading.Event()
        self._thread = None

    def start(self):
        import threading
        if smi_snapshot() is None:  # amd-smi absent
            return self
        self._thread = threading.Thread(target=self._run, daemon=True)
        self._thread.start()
        return self

    def _run(self):
        while not self._stop.is_set():
            snap = smi_snapshot()
            if snap:
                self.samples.append({"t": round(time.perf_counter(), 3), "lines": snap})

    def running(self):
        return self._thread is not None and self._thread.is_alive()

    def stop(self):
        self._stop.set()
        if self._thread is not None:
            self._thread.join(timeout=30)
        return self.samples


def read_peak_gbs(amk, torch, nbytes=8 << 30):
    """Best streaming-read rate of this device over nbytes (amk_read_probe)."""
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    stream = torch.cuda.current_stream()
    best = 0.0
    for blocks in (n_cu, 2 * n_cu, 4 * n_cu, 8 * n_cu):
        sink = torch.empty(blocks * 512, dtype=torch.int32, device="cuda")
        for rep in range(4):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            amk.amk_read_probe(buf.data_ptr(), nbytes, blocks, sink.data_ptr(), stream.cuda_stream)
            e1.record(stream)
            e1.synchronize()
            if rep:
                best = max(best, nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del buf
    torch.cuda.empty_cache()
    return best


def cpu_baseline_leg(w, fmt, pos, kv_np, repeats):
    """The CPU baseline: the oracle's decode step for this workload on the host
    cores, timed (median of `repeats`).  Its logits also serve as the variant's
    correctness reference; this is the only place the benchmark runs the oracle."""
    import oracle

    cfg = w.cfg
    # the timed oracle (first variant) decodes its weights to fp32 before
    # the timed region when host memory holds them twice over
    upcast = repeats > 1 and host_free_bytes() > 3 * fp32_model_bytes(cfg)
    model = oracle.OracleModel(w, fmt, np.float32, cache=upcast)
    if upcast:
        t0 = time.perf_counter()
        for name in w.bf16:
            if w.bf16[name].ndim == 2 and name != "embed" or (name == "embed" and cfg.tied_embeddings):
                model.mat(name)
        log(f"oracle weights decoded to fp32 in {time.perf_counter() - t0:.1f}s (outside the timed region)")
    times = []
    logits = None
    for _ in range(repeats):
        kv_ref = kv_np.copy()
        t0 = time.perf_counter()
        logits = oracle.decode_step(model, 1, pos, kv_ref)
        times.append(time.perf_counter() - t0)
    del model
    return {"logits": logits, "token": oracle.argmax_first(logits), "seconds": float(np.median(times)),
            "upcast": upcast, "top2_margin": oracle.top2_margin(logits)}


def run_variant(amk, torch, w, fmt, pos, steps, warmup, check=True, oracle_repeats=1, baseline=True):
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
    ref_logits = None
    if check:
        log(f"variant {fmt} pos {pos}: oracle step")
        cb = cpu_baseline_leg(w, fmt, pos, kv_np, oracle_repeats)
        ref_logits, ref_tok, cpu_s = cb["logits"], cb["token"], cb["seconds"]
        err = float(np.max(np.abs(logits.cpu().numpy().astype(np.float64) - ref_logits)))
        res.update(oracle_s=cpu_s, oracle_upcast=cb["upcast"], max_abs_logit_err=err, token=tok,
                   oracle_token=ref_tok, oracle_top2_margin=cb["top2_margin"],
                   correct=bool(tok == ref_tok and err <= 2e-2))
        log(f"variant {fmt} pos {pos}: token {tok} oracle {ref_tok} err {err:.2e} oracle {cpu_s:.1f}s")
    else:
        res.update(correct=None)

    for _ in range(warmup):
        dec.step(1, pos, kv, logits)
    torch.cuda.synchronize()
    smi_before = smi_snapshot() if check else None
    sampler = SmiSampler().start() if check else None
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
    smi_during = []
    if sampler is not None:
        # the timed region is shorter than one amd-smi call: keep the same
        # step running (untimed) until two samples were taken under load
        t1 = time.perf_counter()
        while sampler.running() and len(sampler.samples) < 2 and time.perf_counter() - t1 < 20:
            for _ in range(20):
                dec.step(1, pos, kv, logits)
            torch.cuda.synchronize()
        smi_during = sampler.stop()
    smi_after = smi_snapshot() if check else None
    # whole token as a host sees it: the API call plus the next-token readback
    n_rb = max(1, min(steps, 20))
    t0 = time.perf_counter()
    for _ in range(n_rb):
        dec.step(1, pos, kv, logits)
        dec.next_token()
    token_wall_us = (time.perf_counter() - t0) / n_rb * 1e6
    status = dec.status()
    dec.close()
    if baseline and fmt in ("bf16", "w8a16"):
        res["torch_reference"] = torch_reference(torch, cfg, tensors, fmt, pos, kv_np, max_seq, steps, warmup,
                                                 ref_logits)
    del tensors
    torch.cuda.empty_cache()
    nbytes = cfg.algorithmic_bytes(fmt, pos)
    med = float(np.median(launch_us))
    res.update(status=status, wall_us_per_step=wall / steps * 1e6, token_wall_us_with_readback=token_wall_us,
               launch_us_median=med,
               launch_us_mean=float(np.mean(launch_us)), launch_us_p10=float(np.percentile(launch_us, 10)),
               launch_us_p90=float(np.percentile(launch_us, 90)), algorithmic_bytes=nbytes,
               achieved_gbs=nbytes / (float(np.mean(launch_us)) * 1e-6) / 1e9,
               floor_us=nbytes / (PEAK_HBM_GBS * 1e9) * 1e6)
    res["floor_ratio"] = res["launch_us_mean"] / res["floor_us"]
    # a time below the bandwidth floor would be a measurement artefact
    res["below_floor"] = bool(float(np.min(launch_us)) < res["floor_us"])
    if smi_before or smi_after or smi_during:
        res["amd_smi"] = {"before": smi_before, "during_load": smi_during, "after": smi_after}
    return res


def host_free_bytes() -> int:
    try:
        import psutil
        return int(psutil.virtual_memory().available)
    except Exception:
        return 0


def fp32_model_bytes(cfg) -> int:
    return 4 * (sum(o * i for _, o, i in cfg.linear_shapes()) * cfg.n_layers + cfg.vocab * cfg.hidden)


def torch_reference(torch, cfg, tensors, fmt, pos, kv_np, max_seq, steps, warmup, ref_logits):
    """The same step in plain PyTorch-ROCm, per-op eager and HIP-graph replay:
    µs per token (step plus an on-device argmax), checked against the oracle's
    logits when they were computed.  A same-node reference, not a target."""
    from paper_2606_09682_amd import torch_baseline as tb
    from synth.device import kv_to_device
    log(f"variant {fmt} pos {pos}: torch reference")
    ref = tb.TorchDecode(cfg, tensors, fmt, max_seq)
    kv = kv_to_device(kv_np)
    logits = torch.empty(cfg.vocab, dtype=torch.float32, device="cuda")
    tok = torch.tensor([1], device="cuda")
    ref.step(tok, pos, kv, logits)
    out = {"kind": "pytorch-rocm per-op eager and HIP graph (bf16 GEMV via torch.nn.functional.linear)",
           "weights_streamed": "bf16" if fmt == "bf16" else "bf16 (dequantised once from int8)"}
    if ref_logits is not None:
        err = float(np.max(np.abs(logits.cpu().numpy().astype(np.float64) - ref_logits)))
        out.update(max_abs_logit_err=err, token=ref.next_token(logits),
                   logit_bound=tb.logit_bound(ref_logits), oracle_top2_margin=float(
                       np.partition(ref_logits, -2)[-1] - np.partition(ref_logits, -2)[-2]),
                   correct=bool(err <= tb.logit_bound(ref_logits) and (
                       ref.next_token(logits) == int(np.argmax(ref_logits)) or
                       np.partition(ref_logits, -2)[-1] - np.partition(ref_logits, -2)[-2] <= 2 * err)))
    stream = torch.cuda.current_stream()

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / steps

    out["eager_us_per_token"] = timed(lambda: (ref.step(tok, pos, kv, logits), torch.argmax(logits)))
    g = tb.GraphDecode(ref, pos, kv, logits)
    out["graph_us_per_token"] = timed(lambda: (g.step(1), torch.argmax(logits)))
    del g, ref
    torch.cuda.empty_cache()
    log(f"variant {fmt} pos {pos}: torch eager {out['eager_us_per_token']:.0f} us, "
        f"graph {out['graph_us_per_token']:.0f} us")
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=25)
    ap.add_argument("--config", default="llama3_8b")
    ap.add_argument("--variants", default="all",
                    help="'all', 'main' (bf16 at position 0 only) or a comma list of FMT@POS, e.g. w4a16@0")
    ap.add_argument("--no-check", action="store_true", help="skip the oracle gate (profiling runs)")
    ap.add_argument("--no-torch-reference", action="store_true",
                    help="skip the PyTorch-ROCm eager / HIP-graph reference (implied by --no-check)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES (counter calibration) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU; --gpus {args.gpus} is not supported "
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
        variants += [("w8a16", cfg.positions[0]), ("w4a16", cfg.positions[0])] + [
            (f, cfg.positions[-1]) for f in ("bf16", "w8a16", "w4a16") if cfg.positions[-1] != cfg.positions[0]]
    elif args.variants != "main":
        variants = [(v.split("@")[0], int(v.split("@")[1])) for v in args.variants.split(",")]
    try:
        cfg.int4_group
    except ValueError as e:  # int4 rows need input widths that are multiples of 32
        log(f"skipping W4A16 variants: {e}")
        variants = [v for v in variants if v[0] != "w4a16"]
    results = []
    for fmt, pos in variants:
        if fmt == "w8a16" and not w.q8:
            t0 = time.perf_counter()
            synth.add_w8a16(w)
            log(f"quantised (int8) in {time.perf_counter() - t0:.1f}s")
        if fmt == "w4a16" and not w.q4:
            t0 = time.perf_counter()
            synth.add_w4a16(w)
            log(f"quantised (int4, group {w.group4}) in {time.perf_counter() - t0:.1f}s")
        results.append(run_variant(amk, torch, w, fmt, pos, args.steps, args.warmup, check=not args.no_check,
                                   oracle_repeats=3 if not results else 1,
                                   baseline=not (args.no_check or args.no_torch_reference)))
        if results[-1].get("correct") is False or results[-1]["status"] != 0:
            log(f"variant {fmt} pos {pos} FAILED its correctness gate: {results[-1]}")
    main_res = results[0]
    ok = all(r.get("correct") is not False and r["status"] == 0 and not r["below_floor"] for r in results)
    peak = None if args.no_check else read_peak_gbs(amk, torch)
    if peak:
        log(f"streaming-read peak {peak:.0f} GB/s")
    workload = f"{cfg.name}_{main_res['fmt']}_pos{main_res['pos']}"
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
        "config": {"workload": workload, "model_shape": cfg.name, "batch": 1, "position": main_res["pos"],
                   "weights": main_res["fmt"], "parallelism": "single GPU"},
        "correct": ok,
        "roofline": {"bound": "hbm", "achieved": main_res["achieved_gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": main_res["achieved_gbs"] / PEAK_HBM_GBS,
                     "traffic": traffic},
        "measured_read_peak_gbs": peak,
        "frac_of_measured_peak": (main_res["achieved_gbs"] / peak) if peak else None,
        "cpu_baseline": None,
        "same_node_reference": main_res.get("torch_reference"),
        "variants": [{k: (round(v, 3) if isinstance(v, float) else v) for k, v in r.items()} for r in results],
    }
    if "oracle_s" in main_res:
        threads, blas = blas_info()
        out["cpu_baseline"] = {"value": main_res["oracle_s"] * 1e6, "unit": "µs/token", "cores": threads,
                               "kind": "oracle",
                               "sample": f"median of 3 full decode steps of {workload} (numpy fp32, weights "
                                         + ("decoded to fp32 before the timed region" if main_res.get("oracle_upcast")
                                            else "decoded from bf16 per use (host memory too small to hold fp32)")
                                         + f"; BLAS {blas}, {os.cpu_count()} host CPUs, {host_ram_gb()} GiB RAM)"}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
