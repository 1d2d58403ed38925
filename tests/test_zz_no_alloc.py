"""amk_create_static, the entry point for callers that cannot allocate device
memory, against amk_create: the same decode through the C ABI on the same
seeded inputs, twice in a row with the second model smaller than the first
(the static array keeps the first handle's contents), plus its limits: a
model beyond the array is refused, one live static handle per device, and a
forced timeout is reported through the device-side status word."""
import numpy as np
import pytest

import synth
from synth.device import config_kwargs, kv_from_device, kv_to_device, weights_to_device

pytestmark = pytest.mark.gpu

TOL = 2e-2


@pytest.fixture(scope="module")
def env():
    import os
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    from paper_2606_09682_amd import amk
    if not os.path.exists(amk.LIB_PATH):
        from paper_2606_09682_amd import build
        build.build()
    amk.load()
    return amk, torch


def decode(amk, torch, w, fmt, steps, static, tuning=None):
    cfg = w.cfg
    dec = amk.Decoder(amk.make_config(**config_kwargs(cfg, fmt, cfg.seq_capacity)), weights_to_device(w, fmt),
                      tuning, static=static)
    kv = kv_to_device(synth.make_kv_cache(cfg, 0))
    logits = torch.empty(cfg.vocab, dtype=torch.float32, device="cuda")
    toks, lg = [], []
    t = 1
    for i in range(steps):
        dec.step(t, i, kv, logits)
        t = dec.next_token()
        toks.append(t)
        lg.append(logits.cpu().numpy().astype(np.float64))
    assert dec.status() == amk.AMK_OK
    out = (toks, lg, kv_from_device(kv))
    dec.close()
    return out


def test_static_handle_matches_allocating_handle(env):
    amk, torch = env
    # two static handles in a row, the second model smaller than the first
    for name, fmt, steps in (("smollm2_135m", "bf16", 8), ("tiny", "w8a16", 8)):
        w = synth.make_weights(synth.get(name), seed=0)
        if fmt == "w8a16":
            synth.add_w8a16(w)
        s = decode(amk, torch, w, fmt, steps, static=True)
        a = decode(amk, torch, w, fmt, steps, static=False)
        err = max(float(np.max(np.abs(x - y))) for x, y in zip(s[1], a[1]))
        print(f"{name} {fmt}: static vs allocating max |dlogit| {err:.3e}, tokens {s[0]}")
        assert s[0] == a[0]
        assert err <= TOL
        assert np.array_equal(s[2], a[2])


def test_static_handle_limits(env):
    amk, torch = env
    cfg = synth.get("tiny")
    w = synth.make_weights(cfg, seed=0)
    tensors = weights_to_device(w, "bf16")
    # a RoPE table of 300000 positions alone exceeds the static array
    big = amk.make_config(**config_kwargs(cfg, "bf16", 300000))
    with pytest.raises(amk.AmkError) as e:
        amk.Decoder(big, tensors, static=True)
    assert e.value.status == amk.AMK_ERR_OUT_OF_MEMORY
    small = amk.make_config(**config_kwargs(cfg, "bf16", 16))
    first = amk.Decoder(small, tensors, static=True)
    with pytest.raises(amk.AmkError) as e:
        amk.Decoder(small, tensors, static=True)
    assert e.value.status == amk.AMK_ERR_BAD_STATE
    assert amk.load().amk_set_abort(first.handle, 1) == amk.AMK_ERR_UNSUPPORTED
    first.close()
    # a forced timeout is reported by the device-side status word and cleared by reset
    t = amk.amk_tuning_t(0, 1, 0, 0, 0, 0)
    dec = amk.Decoder(small, tensors, t, static=True)
    kv = kv_to_device(synth.make_kv_cache(cfg, 0, max_seq=16))
    logits = torch.empty(cfg.vocab, dtype=torch.float32, device="cuda")
    dec.step(1, 0, kv, logits)
    assert dec.status() == amk.AMK_ERR_TIMEOUT
    dec.reset()
    assert dec.status() == amk.AMK_OK
    dec.close()
