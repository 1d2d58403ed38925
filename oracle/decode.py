"""CPU oracle for one batch-1 Llama decode step (TEST INFRASTRUCTURE ONLY).

This is the plain, slow, obviously-correct definition that the GPU decode
step is checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run it; the product path
(the HIP library and its Python binding) never does.  It shares no code with
the GPU path: the only common module is ``synth`` (seeded inputs, no method
arithmetic).

What is computed.  The paper runs the forward pass of a bias-free,
full-rotary, SiLU-SwiGLU, RMSNorm, GQA Llama (paper §6 "Architecture
coverage") as one launch per decoded token, with the KV cache persisting in
memory across launches (paper §4 "Synchronization model") and greedy decoding
compared token-for-token with HuggingFace (paper §5 "Correctness and
retargeting").  The method is a re-scheduling of exactly this arithmetic, so
the oracle is the plain definition written out, step by step:

    x   = E[token]
    per layer:  h = RMSNorm(x, g_attn);  q, k, v = Wq h, Wk h, Wv h
                q, k <- RoPE(., pos);  cache[pos] <- (k, v) rounded to bf16
                o_h = softmax(q_h . K / sqrt(d)) V   (KV head = h // group)
                x = x + Wo o
                h2 = RMSNorm(x, g_mlp);  x = x + Wd (silu(Wg h2) * (Wu h2))
    logits = W_lm RMSNorm(x, g_final);  next = argmax(logits)

W8A16 and W4A16 (paper §5 "Quantized generation": int8 / int4 weight-only,
dequantisation folded into the GEMV) equal the same decode with W' = q * s
(s per row for int8, per row and group of input columns for int4), so the
oracle dequantises explicitly and then runs the plain product.

Readings where the paper is silent (each also listed in the design notes):
RMSNorm is x / sqrt(mean(x^2) + eps) * g with eps inside the root; RoPE is
the rotate-half form pairing i with i + d/2, angles pos * theta^(-2i/d)
evaluated in float64 then rounded to the compute precision, applied to q and
k before k is cached; the K/V row appended at ``pos`` is rounded to bf16
(round-to-nearest-even) and attention reads the rounded row back like every
older row; attention scales by 1/sqrt(head_dim) and subtracts the row max
before the exponential; silu(z) = z / (1 + exp(-z)); argmax takes the lowest
index among equal maxima.

Parity of this module is pinned by tests/test_oracle_pins.py (closed forms,
brute force, invariants) and tests/test_oracle_vs_transformers.py (an
independent implementation of the same model family).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional, Tuple

import numpy as np


# --------------------------------------------------------------------------
# storage formats
# --------------------------------------------------------------------------
def bf16_decode(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float32 values (exact)."""
    wide = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return wide.view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bf16 value, ties to even; returns the bit patterns.

    Used where the decode step stores a value in bf16: the new K and V rows
    appended to the KV cache."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    return ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)


# --------------------------------------------------------------------------
# the operations of one layer (paper §3, Layer 1 "GEMV, attention, RMSNorm,
# RoPE"; §6 supported family)
# --------------------------------------------------------------------------
def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g."""
    x = np.asarray(x)
    ms = np.mean(x * x)
    return x / np.sqrt(ms + x.dtype.type(eps)) * g


def rope_angles(pos: int, head_dim: int, theta: float) -> Tuple[np.ndarray, np.ndarray]:
    """cos and sin of pos * theta^(-2i/d) for i < d/2, evaluated in float64."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = np.power(np.float64(theta), -2.0 * i / head_dim)
    ang = np.float64(pos) * inv_freq
    return np.cos(ang), np.sin(ang)


def rope(u: np.ndarray, pos: int, theta: float) -> np.ndarray:
    """Rotate-half RoPE of head vectors u[..., d] at position ``pos``.

    out[i]       = u[i] cos(a_i) - u[i+d/2] sin(a_i)
    out[i+d/2]   = u[i+d/2] cos(a_i) + u[i] sin(a_i)"""
    d = u.shape[-1]
    c, s = rope_angles(pos, d, theta)
    c = c.astype(u.dtype)
    s = s.astype(u.dtype)
    lo, hi = u[..., : d // 2], u[..., d // 2:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (z.dtype.type(1) + np.exp(-z))


def softmax(s: np.ndarray) -> np.ndarray:
    e = np.exp(s - np.max(s))
    return e / np.sum(e)


def attention(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """Grouped-query decode attention.

    q: [n_heads, d]; K, V: [n_kv_heads, n_pos, d] (positions 0..pos).
    Query head h reads KV head h // (n_heads / n_kv_heads)."""
    n_heads, d = q.shape
    group = n_heads // K.shape[0]
    scale = q.dtype.type(1.0 / np.sqrt(d))
    out = np.empty_like(q)
    for h in range(n_heads):
        kv = h // group
        p = softmax((K[kv] @ q[h]) * scale)
        out[h] = p @ V[kv]
    return out


def linear(W: np.ndarray, x: np.ndarray) -> np.ndarray:
    """y = W x for a row-major [out, in] weight (nn.Linear layout, no bias)."""
    return W @ x


def dequantize(q: np.ndarray, s: np.ndarray, dtype=np.float32) -> np.ndarray:
    """W' = q * s[row] for symmetric per-output-channel int8 weights."""
    return q.astype(dtype) * s.astype(dtype)[:, None]


def unpack_int4(packed: np.ndarray, dtype=np.int16) -> np.ndarray:
    """Signed int4 codes [out, in] of a packed W4A16 matrix [out, in / 2], as ``dtype``.

    Storage layout: byte i of a row belongs to 32-bit word d = i // 4 at byte
    position b = i % 4 and holds column 8d + b in its low nibble and column
    8d + 4 + b in its high nibble, each as the unsigned value code + 8."""
    p = np.asarray(packed, dtype=np.uint8)
    rows, nbytes = p.shape
    if nbytes % 4:
        raise ValueError("a packed row is a whole number of 32-bit words")
    words = p.reshape(rows, nbytes // 4, 4)                    # [row, word d, byte b]
    codes = np.empty((rows, nbytes // 4, 8), dtype=dtype)     # [row, word d, column 8d + j]
    codes[:, :, 0:4] = words & 0x0F                            # column 8d + b
    codes[:, :, 4:8] = words >> 4                              # column 8d + 4 + b
    codes -= 8
    return codes.reshape(rows, 2 * nbytes)


def dequantize_int4(packed: np.ndarray, s: np.ndarray, group: int, dtype=np.float32) -> np.ndarray:
    """W'[r, k] = q[r, k] * s[r, k // group] for int4 weights with one scale
    per row and group of ``group`` consecutive input columns."""
    q = unpack_int4(packed, dtype)
    rows, k = q.shape
    if s.shape != (rows, k // group) or k % group:
        raise ValueError("scale shape does not match the packed matrix and group")
    q.reshape(rows, k // group, group)[...] *= s.astype(dtype)[:, :, None]  # column k takes scale k // group
    return q


def argmax_first(v: np.ndarray) -> int:
    """Index of the maximum, lowest index on ties; NaN is an error."""
    if np.isnan(v).any():
        raise FloatingPointError("NaN in logits")
    return int(np.argmax(v))


# --------------------------------------------------------------------------
# model access
# --------------------------------------------------------------------------
@dataclass
class OracleModel:
    """Read-only view of the weights in the oracle's compute precision.

    ``weights`` is a ``synth.Weights``; ``fmt`` is 'bf16', 'w8a16' or 'w4a16'.
    Matrices are decoded on demand and optionally cached."""
    weights: object
    fmt: str = "bf16"
    dtype: type = np.float32
    cache: bool = True

    def __post_init__(self):
        self.cfg = self.weights.cfg
        self._cache: Dict[str, np.ndarray] = {}
        if self.fmt not in ("bf16", "w8a16", "w4a16"):
            raise ValueError(self.fmt)

    def vec(self, name: str) -> np.ndarray:
        return bf16_decode(self.weights.bf16[name]).astype(self.dtype)

    def mat(self, name: str) -> np.ndarray:
        if name in self._cache:
            return self._cache[name]
        if self.fmt == "w8a16" and name in self.weights.q8:
            m = dequantize(self.weights.q8[name], self.weights.scale[name], self.dtype)
        elif self.fmt == "w4a16" and name in self.weights.q4:
            m = dequantize_int4(self.weights.q4[name], self.weights.scale4[name], self.weights.group4, self.dtype)
        else:
            m = bf16_decode(self.weights.bf16[name]).astype(self.dtype)
        if self.cache:
            self._cache[name] = m
        return m

    def embed_row(self, token: int) -> np.ndarray:
        return bf16_decode(self.weights.bf16["embed"][token]).astype(self.dtype)

    def lm_head(self) -> np.ndarray:
        return self.mat("embed" if self.cfg.tied_embeddings else "lm_head")


# --------------------------------------------------------------------------
# one decode step
# --------------------------------------------------------------------------
def decode_step(model: OracleModel, token: int, pos: int, kv: np.ndarray,
                round_kv: bool = True, trace: Optional[dict] = None) -> np.ndarray:
    """Run one decode step; appends K/V at ``pos`` into ``kv`` and returns logits.

    kv: uint16 bf16 bits [L][2][n_kv][max_seq][d] when ``round_kv``;
    a float array of the same shape otherwise (the exact variant used to
    compare with a float32 reference implementation)."""
    cfg = model.cfg
    dt = model.dtype
    nq, nkv, d = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    if not (0 <= token < cfg.vocab):
        raise ValueError("token out of range")
    if not (0 <= pos < kv.shape[3]):
        raise ValueError("pos out of range")

    x = model.embed_row(token)
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        h = rmsnorm(x, model.vec(p + "attn_norm"), cfg.rms_eps)
        q = linear(model.mat(p + "wq"), h).reshape(nq, d)
        k = linear(model.mat(p + "wk"), h).reshape(nkv, d)
        v = linear(model.mat(p + "wv"), h).reshape(nkv, d)
        q = rope(q, pos, cfg.rope_theta)
        k = rope(k, pos, cfg.rope_theta)
        if round_kv:
            kv[l, 0, :, pos, :] = bf16_round(k)
            kv[l, 1, :, pos, :] = bf16_round(v)
            K = bf16_decode(kv[l, 0, :, : pos + 1, :]).astype(dt)
            V = bf16_decode(kv[l, 1, :, : pos + 1, :]).astype(dt)
        else:
            kv[l, 0, :, pos, :] = k
            kv[l, 1, :, pos, :] = v
            K = kv[l, 0, :, : pos + 1, :].astype(dt)
            V = kv[l, 1, :, : pos + 1, :].astype(dt)
        o = attention(q, K, V).reshape(nq * d)
        x = x + linear(model.mat(p + "wo"), o)
        h2 = rmsnorm(x, model.vec(p + "mlp_norm"), cfg.rms_eps)
        a = silu(linear(model.mat(p + "wg"), h2)) * linear(model.mat(p + "wu"), h2)
        x = x + linear(model.mat(p + "wd"), a)
        if trace is not None:
            trace.setdefault("x", []).append(x.copy())
    hf = rmsnorm(x, model.vec("final_norm"), cfg.rms_eps)
    return linear(model.lm_head(), hf)


def greedy(model: OracleModel, token: int, pos: int, steps: int, kv: np.ndarray,
           round_kv: bool = True) -> Tuple[List[int], List[np.ndarray]]:
    """``steps`` greedy decode steps starting from ``token`` at ``pos``.

    Returns the generated tokens and the logits of every step."""
    toks, logits = [], []
    t = token
    for i in range(steps):
        lg = decode_step(model, t, pos + i, kv, round_kv=round_kv)
        t = argmax_first(lg)
        toks.append(t)
        logits.append(lg)
    return toks, logits


def top2_margin(logits: np.ndarray) -> float:
    """Gap between the largest and second-largest logit (greedy robustness)."""
    part = np.partition(np.asarray(logits, dtype=np.float64), -2)
    return float(part[-1] - part[-2])
