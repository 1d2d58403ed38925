"""The same-node PyTorch-ROCm reference decode (per-op eager and HIP-graph
replay) against the CPU oracle: the baseline the megakernel's time is put
beside must compute the same model.  Bar: fed the oracle's greedy tokens,
every step's logits within torch_baseline.logit_bound (5% of the step's
largest |logit|: its GEMV inputs and outputs are bf16) and the same greedy token wherever the oracle's top-2
margin exceeds twice that step's error; graph replays equal the eager step
bit for bit, replay after replay."""
import sys

import numpy as np
import pytest

import oracle
import synth
from synth.device import kv_from_device, kv_to_device, weights_to_device

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[gpu-test] {msg}", file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    return torch


def make(torch, name, fmt, max_seq):
    from paper_2606_09682_amd import torch_baseline as tb
    cfg = synth.get(name)
    if fmt == "w4a16" and name == "tiny":
        cfg = cfg.with_(name="tiny_i768", intermediate=768)
    w = synth.make_weights(cfg, seed=0)
    if fmt == "w8a16":
        synth.add_w8a16(w)
    elif fmt == "w4a16":
        synth.add_w4a16(w)
    tensors = weights_to_device(w, fmt)
    dec = tb.TorchDecode(cfg, tensors, fmt, max_seq, group=w.group4)
    return w, tensors, dec


def eager_forced(torch, dec, kv, pos0, inputs, vocab):
    """Steps fed the given input tokens (the oracle's greedy path), so that a
    greedy decision the bf16 activations flip does not change later inputs;
    returns each step's argmax and logits."""
    logits = torch.empty(vocab, dtype=torch.float32, device="cuda")
    toks, lgs = [], []
    for i, t in enumerate(inputs):
        dec.step(torch.tensor([t], device="cuda"), pos0 + i, kv, logits)
        toks.append(dec.next_token(logits))
        lgs.append(logits.cpu().numpy().astype(np.float64))
    return toks, lgs


@pytest.mark.parametrize("name,fmt,pos,steps", [
    ("tiny", "bf16", 0, 8), ("tiny", "w8a16", 0, 8), ("tiny", "w4a16", 0, 8),
    ("smollm2_135m", "bf16", 0, 4), ("smollm2_135m", "w8a16", 0, 4),
    ("tinyllama_1b", "bf16", 1024, 1), ("llama32_1b", "w8a16", 4096, 1),
    ("llama3_8b", "bf16", 0, 1), ("llama3_8b", "w8a16", 8192, 1)])
def test_eager_matches_oracle(torch_cuda, name, fmt, pos, steps):
    from paper_2606_09682_amd import torch_baseline as tb
    torch = torch_cuda
    max_seq = pos + steps + 1
    w, tensors, dec = make(torch, name, fmt, max_seq)
    kv_np = synth.make_kv_cache(w.cfg, pos, seed=1, max_seq=max_seq)
    say(f"torch eager {name} {fmt} pos {pos} steps {steps}")
    model = oracle.OracleModel(w, fmt, np.float32, cache=w.cfg.hidden <= 2048)
    kv_ref = kv_np.copy()
    o_toks, o_lgs = oracle.greedy(model, 1, pos, steps, kv_ref)
    kv = kv_to_device(kv_np)
    toks, lgs = eager_forced(torch, dec, kv, pos, [1] + o_toks[:-1], w.cfg.vocab)
    errs = [float(np.max(np.abs(a - b))) for a, b in zip(lgs, o_lgs)]
    margins = [oracle.top2_margin(l) for l in o_lgs]
    say(f"torch eager {name} {fmt}: |dlogit| vs oracle per step {[f'{e:.2e}' for e in errs]}, "
        f"argmax {toks} (oracle {o_toks}, top-2 margins {[f'{m:.2e}' for m in margins]})")
    bounds = [tb.logit_bound(l) for l in o_lgs]
    assert all(e <= b for e, b in zip(errs, bounds)), (errs, bounds)
    # the greedy token agrees wherever the oracle's decision is wider than the
    # baseline's error can flip
    for t, ot, e, mg in zip(toks, o_toks, errs, margins):
        assert t == ot or mg <= 2 * e, (t, ot, e, mg)
    # the appended rows land in the library's layout, other slots untouched
    g = kv_from_device(kv)
    sl = slice(pos, pos + steps)
    mask = np.ones(g.shape[3], bool)
    mask[sl] = False
    assert np.array_equal(g[:, :, :, mask], kv_ref[:, :, :, mask])
    a = oracle.bf16_decode(g[:, :, :, sl]).astype(np.float64)
    b = oracle.bf16_decode(kv_ref[:, :, :, sl]).astype(np.float64)
    # deeper layers carry the bf16 activations' error, within the same relative bound
    assert np.linalg.norm(a - b) <= tb.LOGIT_REL_TOL * np.linalg.norm(b)


@pytest.mark.parametrize("name,fmt,pos", [("tiny", "bf16", 3), ("smollm2_135m", "w8a16", 5),
                                          ("llama3_8b", "bf16", 0)])
def test_graph_replays_equal_eager(torch_cuda, name, fmt, pos):
    """Replays of the captured step, with eager work and synchronisation
    between them, give the eager step's logits and KV rows bit for bit."""
    from paper_2606_09682_amd import torch_baseline as tb
    torch = torch_cuda
    max_seq = pos + 2
    w, tensors, dec = make(torch, name, fmt, max_seq)
    kv_np = synth.make_kv_cache(w.cfg, pos, seed=1, max_seq=max_seq)
    kv_e = kv_to_device(kv_np)
    lg_e = torch.empty(w.cfg.vocab, dtype=torch.float32, device="cuda")
    dec.step(torch.tensor([1], device="cuda"), pos, kv_e, lg_e)
    want_lg, want_kv = lg_e.cpu().numpy(), kv_from_device(kv_e)
    kv_g = kv_to_device(kv_np)
    lg_g = torch.empty_like(lg_e)
    g = tb.GraphDecode(dec, pos, kv_g, lg_g)
    for r in range(4):
        lg_g.fill_(float("nan"))
        g.step(1)
        torch.cuda.synchronize()
        assert np.array_equal(lg_g.cpu().numpy(), want_lg), r
        assert np.array_equal(kv_from_device(kv_g), want_kv), r
        dec.step(torch.tensor([1], device="cuda"), pos, kv_e, lg_e)  # eager work between replays
        torch.cuda.synchronize()
    say(f"torch graph {name} {fmt} pos {pos}: 4 replays equal the eager step")
