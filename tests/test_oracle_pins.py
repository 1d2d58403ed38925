"""Pins of the CPU oracle against closed forms, brute force, invariants and
library routines (no GPU).  Each test names what would break it."""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
import synth


# ---------------------------------------------------------------- bf16 storage
def test_bf16_decode_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0000, 0x8000, 0x4049], dtype=np.uint16)
    want = [1.0, -2.0, 1.0078125, 0.0, -0.0, 3.140625]
    assert oracle.bf16_decode(bits).tolist() == want


def test_bf16_round_ties_to_even():
    one = 1.0
    ulp = 2.0 ** -7
    vals = np.array([one, one + ulp / 2, one + 3 * ulp / 2, one + ulp / 2 + 2 ** -20, -one - ulp / 2],
                    dtype=np.float32)
    got = oracle.bf16_round(vals)
    assert got.tolist() == [0x3F80, 0x3F80, 0x3F82, 0x3F81, 0xBF80]


def test_bf16_round_matches_torch():
    rng = np.random.default_rng(5)
    x = (rng.standard_normal(100_000) * 10 ** rng.uniform(-6, 6, 100_000)).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.bf16_round(x), ref)


# ---------------------------------------------------------------- RMSNorm
def test_rmsnorm_hand_computed():
    x = np.array([3.0, 4.0], dtype=np.float64)
    out = oracle.rmsnorm(x, np.ones(2), 1e-5)
    want = x / math.sqrt(12.5 + 1e-5)
    np.testing.assert_allclose(out, want, rtol=0, atol=1e-15)


def test_rmsnorm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(257)
    out = oracle.rmsnorm(x, np.ones(257), 0.0)
    assert abs(np.sqrt(np.mean(out ** 2)) - 1.0) < 1e-12
    np.testing.assert_allclose(oracle.rmsnorm(7.5 * x, np.ones(257), 0.0), out, atol=1e-12)


def test_rmsnorm_gain_and_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(64)
    g = rng.standard_normal(64)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (64,), torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(oracle.rmsnorm(x, g, 1e-5), ref, atol=1e-12)


# ---------------------------------------------------------------- RoPE
def _rotation_matrix(pos, d, theta):
    """Block rotation acting on the coordinate pairs (i, i + d/2)."""
    R = np.zeros((d, d))
    for i in range(d // 2):
        a = pos * theta ** (-2.0 * i / d)
        c, s = math.cos(a), math.sin(a)
        R[i, i], R[i, i + d // 2] = c, -s
        R[i + d // 2, i], R[i + d // 2, i + d // 2] = s, c
    return R


@pytest.mark.parametrize("pos,d,theta", [(0, 8, 1e4), (5, 8, 1e4), (1023, 64, 1e4), (8192, 128, 5e5)])
def test_rope_equals_rotation_matrix(pos, d, theta):
    rng = np.random.default_rng(pos)
    u = rng.standard_normal((3, d))
    got = oracle.rope(u, pos, theta)
    want = u @ _rotation_matrix(pos, d, theta).T
    np.testing.assert_allclose(got, want, atol=1e-12)


def test_rope_two_dims_closed_form():
    # d = 2: one pair, frequency theta^0 = 1, so the angle is the position itself
    for p in (0, 1, 3, 10):
        out = oracle.rope(np.array([1.0, 0.0]), p, 1e4)
        np.testing.assert_allclose(out, [math.cos(p), math.sin(p)], atol=1e-15)


def test_rope_invariants():
    rng = np.random.default_rng(2)
    d, th = 64, 1e4
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    np.testing.assert_allclose(oracle.rope(q, 0, th), q, atol=0)
    for p in (1, 17, 300):
        assert abs(np.linalg.norm(oracle.rope(q, p, th)) - np.linalg.norm(q)) < 1e-12
    np.testing.assert_allclose(oracle.rope(oracle.rope(q, 7, th), 11, th), oracle.rope(q, 18, th), atol=1e-12)
    # inner product depends only on the position difference
    a = oracle.rope(q, 20, th) @ oracle.rope(k, 5, th)
    b = oracle.rope(q, 115, th) @ oracle.rope(k, 100, th)
    assert abs(a - b) < 1e-10


# ---------------------------------------------------------------- attention
def test_attention_pos0_returns_v_row():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((4, 16))
    K = rng.standard_normal((2, 1, 16))
    V = rng.standard_normal((2, 1, 16))
    out = oracle.attention(q, K, V)
    for h in range(4):
        np.testing.assert_array_equal(out[h], V[h // 2, 0])


def test_attention_identical_keys_give_mean():
    rng = np.random.default_rng(4)
    q = rng.standard_normal((2, 8))
    K = np.repeat(rng.standard_normal((1, 1, 8)), 5, axis=1)
    V = rng.standard_normal((1, 5, 8))
    out = oracle.attention(q, K, V)
    np.testing.assert_allclose(out, np.repeat(V[0].mean(0)[None], 2, 0), atol=1e-14)


def test_attention_bruteforce_loops():
    rng = np.random.default_rng(6)
    nq, nkv, n, d = 6, 2, 7, 5
    q = rng.standard_normal((nq, d))
    K = rng.standard_normal((nkv, n, d))
    V = rng.standard_normal((nkv, n, d))
    out = oracle.attention(q, K, V)
    for h in range(nq):
        g = h // (nq // nkv)
        s = [sum(q[h, t] * K[g, j, t] for t in range(d)) / math.sqrt(d) for j in range(n)]
        m = max(s)
        e = [math.exp(v - m) for v in s]
        z = sum(e)
        for t in range(d):
            want = sum(e[j] / z * V[g, j, t] for j in range(n))
            assert abs(out[h, t] - want) < 1e-12


def test_attention_gqa_mapping():
    nq, nkv, n, d = 8, 2, 3, 4
    q = np.ones((nq, d))
    K = np.zeros((nkv, n, d))
    V = np.zeros((nkv, n, d))
    for g in range(nkv):
        V[g] = 10.0 * g + 1.0
    out = oracle.attention(q, K, V)
    for h in range(nq):
        assert np.all(out[h] == 10.0 * (h // 4) + 1.0)


def test_attention_matches_torch_sdpa():
    rng = np.random.default_rng(8)
    nq, nkv, n, d = 8, 2, 9, 16
    q = rng.standard_normal((nq, d))
    K = rng.standard_normal((nkv, n, d))
    V = rng.standard_normal((nkv, n, d))
    Kr = torch.from_numpy(K).repeat_interleave(nq // nkv, 0)
    Vr = torch.from_numpy(V).repeat_interleave(nq // nkv, 0)
    ref = torch.nn.functional.scaled_dot_product_attention(torch.from_numpy(q)[:, None, :], Kr, Vr)[:, 0]
    np.testing.assert_allclose(oracle.attention(q, K, V), ref.numpy(), atol=1e-12)


# ---------------------------------------------------------------- SiLU / softmax
def test_silu_identities():
    z = np.linspace(-20, 20, 101)
    s = oracle.silu(z)
    assert oracle.silu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(s - oracle.silu(-z), z, atol=1e-12)
    np.testing.assert_allclose(s, torch.nn.functional.silu(torch.from_numpy(z)).numpy(), atol=1e-14)


def test_softmax_closed_form():
    p = oracle.softmax(np.array([0.0, math.log(2.0)]))
    np.testing.assert_allclose(p, [1 / 3, 2 / 3], atol=1e-15)
    x = np.random.default_rng(9).standard_normal(20)
    np.testing.assert_allclose(oracle.softmax(x + 100.0), oracle.softmax(x), atol=1e-14)
    assert abs(oracle.softmax(x).sum() - 1) < 1e-14


# ---------------------------------------------------------------- GEMV / int8
def test_linear_bruteforce_integers():
    rng = np.random.default_rng(10)
    W = rng.integers(-5, 6, size=(7, 13)).astype(np.float32)
    x = rng.integers(-5, 6, size=13).astype(np.float32)
    y = oracle.linear(W, x)
    for r in range(7):
        assert y[r] == sum(W[r, c] * x[c] for c in range(13))


def test_dequantize_bruteforce():
    q = np.array([[1, -2, 127], [0, 0, 0]], dtype=np.int8)
    s = np.array([0.5, 0.0], dtype=np.float32)
    np.testing.assert_array_equal(oracle.dequantize(q, s), [[0.5, -1.0, 63.5], [0, 0, 0]])


def test_quantizer_bounds():
    rng = np.random.default_rng(11)
    w = synth.f32_to_bf16_bits((rng.standard_normal((64, 96)) * 0.02).astype(np.float32))
    w[3] = 0  # an all-zero row
    q, s = synth.quantize_rows(w)
    wf = oracle.bf16_decode(w).astype(np.float64)
    deq = oracle.dequantize(q, s, np.float64)
    # half a quantisation step, plus one float32 rounding of w / s (the quantiser divides in float32)
    bound = s[:, None].astype(np.float64) * 0.5 + np.abs(wf) * 2.0 ** -22
    assert np.all(np.abs(wf - deq) <= bound)
    nz = s > 0
    assert np.all(np.abs(q[nz]).max(axis=1) == 127)
    assert np.all(q[3] == 0) and s[3] == 0
    assert np.all(np.sign(q.astype(np.int32)) * np.sign(wf) >= 0)


def test_dequantized_gemv_within_fp32_bound():
    rng = np.random.default_rng(12)
    w = synth.f32_to_bf16_bits((rng.standard_normal((128, 4096)) * 0.02).astype(np.float32))
    q, s = synth.quantize_rows(w)
    x = rng.standard_normal(4096).astype(np.float32)
    y32 = oracle.linear(oracle.dequantize(q, s, np.float32), x)
    y64 = (q.astype(np.float64) * s.astype(np.float64)[:, None]) @ x.astype(np.float64)
    bound = 4096 * np.finfo(np.float32).eps * (np.abs(q) * s[:, None]) @ np.abs(x)
    assert np.all(np.abs(y32 - y64) <= bound)


# ---------------------------------------------------------------- int4 (W4A16)
GOLDEN_W4 = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "w4a16_layout.json")


def test_int4_layout_golden():
    """Hand-worked example of the packed layout and the group dequantisation
    (a swapped nibble, a wrong word / byte index, a missing zero point or a
    wrong group index fails it)."""
    g = json.load(open(GOLDEN_W4))
    packed = np.array(g["packed"], dtype=np.uint8)
    assert oracle.unpack_int4(packed).tolist() == g["codes"]
    s = np.array(g["scales"], dtype=np.float16)
    assert oracle.dequantize_int4(packed, s, g["group"]).tolist() == g["dequantized"]
    # the inputs' packer writes the same bytes for the same codes
    assert synth.pack_int4(np.array(g["codes"], dtype=np.int8)).tolist() == g["packed"]


def test_int4_pack_unpack_are_inverse():
    # two independent codings of the layout (the inputs' packer, the oracle's unpacker)
    rng = np.random.default_rng(20)
    codes = rng.integers(-8, 8, size=(37, 256)).astype(np.int8)
    assert np.array_equal(oracle.unpack_int4(synth.pack_int4(codes)), codes)


@pytest.mark.parametrize("group", [32, 64, 128])
def test_int4_quantizer_bounds(group):
    rng = np.random.default_rng(21 + group)
    w = synth.f32_to_bf16_bits((rng.standard_normal((48, 512)) * 0.02).astype(np.float32))
    w[5, group:2 * group] = 0  # an all-zero group
    packed, s = synth.quantize_groups4(w, group)
    assert packed.shape == (48, 256) and s.shape == (48, 512 // group) and s.dtype == np.float16
    wf = oracle.bf16_decode(w).astype(np.float64)
    deq = oracle.dequantize_int4(packed, s, group, np.float64)
    sc = np.repeat(s.astype(np.float64), group, axis=1)
    # half a quantisation step, plus one float32 rounding of w / s
    assert np.all(np.abs(wf - deq) <= sc * 0.5 + np.abs(wf) * 2.0 ** -22)
    q = oracle.unpack_int4(packed).reshape(48, 512 // group, group)
    nz = s > 0
    # s = fp16(max|w| / 7): the largest magnitude of every nonzero group maps to code +-7
    assert np.all(np.abs(q).max(axis=2)[nz] == 7)
    assert s[5, 1] == 0 and np.all(q[5, 1] == 0)
    assert np.all(np.sign(q.reshape(48, 512).astype(np.int32)) * np.sign(wf) >= 0)
    # the scale is max|w| / 7 rounded to fp16
    amax = np.abs(wf).reshape(48, 512 // group, group).max(axis=2)
    assert np.array_equal(s, (amax / 7.0).astype(np.float32).astype(np.float16))


def test_int4_quantizer_exact_on_representable_weights():
    # w = q * 2^-7 with a +-7 in every group: quantisation must return q and s exactly
    rng = np.random.default_rng(22)
    q = rng.integers(-7, 8, size=(16, 256))
    q[:, ::64] = 7 * rng.choice([-1, 1], size=(16, 4))
    w = synth.f32_to_bf16_bits((q * 2.0 ** -7).astype(np.float32))
    packed, s = synth.quantize_groups4(w, 64)
    assert np.all(s == np.float16(2.0 ** -7))
    assert np.array_equal(oracle.unpack_int4(packed), q)
    assert np.array_equal(oracle.dequantize_int4(packed, s, 64), oracle.bf16_decode(w).reshape(16, 256))


def test_int4_gemv_bruteforce():
    rng = np.random.default_rng(23)
    w = synth.f32_to_bf16_bits((rng.standard_normal((6, 96)) * 0.02).astype(np.float32))
    packed, s = synth.quantize_groups4(w, 32)
    x = rng.standard_normal(96).astype(np.float32)
    y = oracle.linear(oracle.dequantize_int4(packed, s, 32), x)
    for r in range(6):
        acc = 0.0
        for k in range(96):
            byte = int(packed[r, k // 8 * 4 + k % 4])
            nib = (byte >> 4) if (k % 8) >= 4 else (byte & 15)
            acc += (nib - 8) * float(s[r, k // 32]) * float(x[k])
        assert abs(y[r] - acc) <= 96 * 2.0 ** -23 * np.sum(np.abs(oracle.dequantize_int4(packed, s, 32)[r] * x)) + 1e-12


W4_TINY = synth.get("tiny").with_(name="tiny_i768", intermediate=768)


def test_int4_decode_equals_bf16_decode_on_representable_weights():
    """Weights that int4 with power-of-two group scales holds exactly: the W4A16
    decode must equal the bf16 decode bit for bit (wrong matrix, group or
    LM-head wiring of the int4 path fails it)."""
    cfg = W4_TINY
    w = synth.make_weights(cfg, seed=3)
    rng = np.random.default_rng(24)
    for name in w.quantized_names():
        o, k = w.bf16[name].shape
        q = rng.integers(-7, 8, size=(o, k))
        q[:, ::64] = 7
        w.bf16[name] = synth.f32_to_bf16_bits((q * 2.0 ** -9).astype(np.float32))
    synth.add_w4a16(w, group=64)
    for name in w.quantized_names():
        assert np.all(w.scale4[name] == np.float16(2.0 ** -9)), name
    kv_a = np.zeros(synth.kv_cache_shape(cfg, 4), dtype=np.uint16)
    kv_b = kv_a.copy()
    mb = oracle.OracleModel(w, "bf16")
    m4 = oracle.OracleModel(w, "w4a16")
    for pos, tok in enumerate((1, 77, 4095)):
        lb = oracle.decode_step(mb, tok, pos, kv_a)
        l4 = oracle.decode_step(m4, tok, pos, kv_b)
        assert np.array_equal(lb, l4)
    assert np.array_equal(kv_a, kv_b)


# ---------------------------------------------------------------- argmax
def test_top2_margin_hand_values():
    """The reported greedy margin: largest minus second-largest logit, so a tie
    gives 0 and the margin ignores order and all but the top two values."""
    assert oracle.top2_margin(np.array([1.0, 3.0, 2.0])) == 1.0
    assert oracle.top2_margin(np.array([-5.0, 0.25, -0.5, 0.0])) == 0.25
    assert oracle.top2_margin(np.array([7.0, 7.0, 1.0])) == 0.0
    assert oracle.top2_margin(np.array([2.0, -1.0])) == 3.0
    v = np.random.default_rng(3).standard_normal(1000)
    a, b = sorted(v)[-2:]
    assert oracle.top2_margin(v) == b - a
    assert oracle.top2_margin(v[::-1]) == b - a


def test_argmax_ties_lowest_index_and_nan():
    assert oracle.argmax_first(np.array([1.0, 3.0, 3.0, 2.0])) == 1
    with pytest.raises(FloatingPointError):
        oracle.argmax_first(np.array([1.0, np.nan]))


# ---------------------------------------------------------------- whole step
def test_fp32_oracle_close_to_fp64(tiny_cfg, tiny_weights):
    kv32 = np.zeros(synth.kv_cache_shape(tiny_cfg), dtype=np.float64)
    kv64 = np.zeros_like(kv32)
    m32 = oracle.OracleModel(tiny_weights, "bf16", np.float32)
    m64 = oracle.OracleModel(tiny_weights, "bf16", np.float64)
    for pos in range(3):
        l32 = oracle.decode_step(m32, 1, pos, kv32, round_kv=False)
        l64 = oracle.decode_step(m64, 1, pos, kv64, round_kv=False)
        assert np.max(np.abs(l32 - l64)) < 1e-4


def test_kv_append_is_rounded_bf16(tiny_cfg, tiny_weights):
    kv = synth.make_kv_cache(tiny_cfg, 0)
    m = oracle.OracleModel(tiny_weights, "bf16", np.float64)
    kvf = np.zeros(kv.shape, dtype=np.float64)
    oracle.decode_step(m, 1, 0, kvf, round_kv=False)
    oracle.decode_step(m, 1, 0, kv, round_kv=True)
    # layer 0 sees identical inputs on both runs, so its cached row must be the rounded exact row
    ref = torch.from_numpy(kvf[0, :, :, 0, :].astype(np.float32)).to(torch.bfloat16)
    assert np.array_equal(kv[0, :, :, 0, :], ref.view(torch.int16).numpy().view(np.uint16))
