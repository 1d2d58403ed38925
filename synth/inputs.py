"""Seeded synthetic inputs for the decode step: weights, W8A16 / W4A16 weights, KV cache.

This module is shared by the CPU oracle and the GPU path so that both read
byte-identical inputs.  It holds no arithmetic of the decode method itself:
it draws random numbers, rounds them to bf16 storage, and prepares the int8
and int4 weight-only formats that the decode step consumes.

Recipe (stands in for the checkpoints the paper uses; the decode latency of a
batch-1 step depends on shapes and bytes only, paper §5 "Beating cuBLAS with
int8", which also runs on random-initialised weights at real Llama shapes):

* every projection, the embedding table and an untied LM head: i.i.d.
  N(0, 0.02), rounded to bf16 (round-to-nearest-even);
* RMSNorm gains: 1 + N(0, 0.01), rounded to bf16;
* KV cache slots [0, pos) of every layer / K-V / KV head: N(0, 1) bf16,
  slots >= pos zero;
* W8A16 (paper §5 "Quantized generation": per-output-channel int8 weight-only
  quantisation): symmetric, one fp32 scale per output row,
  s = max|w| / 127, q = clamp(round_half_even(w / s), -127, 127); an all-zero
  row has s = 0 and q = 0.  The embedding table and a tied LM head stay bf16.
* W4A16 (paper §5 "Quantized generation": int4 weight-only, round to
  nearest, fp16 dequantisation scales): symmetric, one fp16 scale per output
  row and group of ``group`` consecutive input columns,
  s = fp16(max|w| / 7), q = clamp(round_half_even(w / s), -8, 7) with the
  division in float32 by the stored (fp16-rounded) scale; an all-zero group
  has s = 0 and q = 0.  Codes are stored as unsigned nibbles q + 8 in the
  packed layout of ``pack_int4``.  Same tensors as W8A16 stay bf16.

Every tensor has its own stream: chunk ``c`` of tensor number ``t`` in the
fixed tensor order is drawn from ``SeedSequence(seed, spawn_key=(t, c))`` with
numpy's PCG64, so any tensor can be regenerated alone and the result does not
depend on the number of threads.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

from .configs import ModelShape

CHUNK = 1 << 22  # elements per independent random stream inside a tensor
GENERATOR_VERSION = "pcg64-seedseq-chunk22-v1"

_KV_STREAM = 1_000_000  # spawn-key offset that keeps KV streams apart from weights


def _threads(threads: Optional[int]) -> int:
    if threads:
        return threads
    return max(1, min(16, os.cpu_count() or 1))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even) and return the bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def tensor_names(cfg: ModelShape) -> List[Tuple[str, Tuple[int, ...], str]]:
    """Fixed tensor order: (name, shape, kind) with kind 'w' (N(0,0.02)) or 'g' (1+N(0,0.01))."""
    H, I, V = cfg.hidden, cfg.intermediate, cfg.vocab
    out: List[Tuple[str, Tuple[int, ...], str]] = [("embed", (V, H), "w")]
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        out += [(p + "attn_norm", (H,), "g"),
                (p + "wq", (cfg.q_dim, H), "w"),
                (p + "wk", (cfg.kv_dim, H), "w"),
                (p + "wv", (cfg.kv_dim, H), "w"),
                (p + "wo", (H, cfg.q_dim), "w"),
                (p + "mlp_norm", (H,), "g"),
                (p + "wg", (I, H), "w"),
                (p + "wu", (I, H), "w"),
                (p + "wd", (H, I), "w")]
    out.append(("final_norm", (H,), "g"))
    if not cfg.tied_embeddings:
        out.append(("lm_head", (V, H), "w"))
    return out


def _fill_chunk(seed: int, key: Tuple[int, int], n: int, kind: str, dst: np.ndarray) -> None:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=key)))
    a = rng.standard_normal(n, dtype=np.float32)
    if kind == "w":
        a *= np.float32(0.02)
    elif kind == "g":
        a *= np.float32(0.01)
        a += np.float32(1.0)
    elif kind == "n":
        pass
    else:
        raise ValueError(kind)
    dst[:] = f32_to_bf16_bits(a)


@dataclass
class Weights:
    """bf16 weights (uint16 bit patterns) plus optional W8A16 / W4A16 copies."""
    cfg: ModelShape
    seed: int
    bf16: Dict[str, np.ndarray]
    q8: Dict[str, np.ndarray] = field(default_factory=dict)     # int8 [out, in]
    scale: Dict[str, np.ndarray] = field(default_factory=dict)  # fp32 [out]
    q4: Dict[str, np.ndarray] = field(default_factory=dict)     # packed int4, uint8 [out, in / 2]
    scale4: Dict[str, np.ndarray] = field(default_factory=dict) # fp16 [out, in / group4]
    group4: int = 0                                             # input columns per int4 scale

    def lm_head_name(self) -> str:
        return "embed" if self.cfg.tied_embeddings else "lm_head"

    def quantized_names(self) -> List[str]:
        names = [f"layers.{l}.{m}" for l in range(self.cfg.n_layers)
                 for m in ("wq", "wk", "wv", "wo", "wg", "wu", "wd")]
        if not self.cfg.tied_embeddings:
            names.append("lm_head")
        return names


def make_weights(cfg: ModelShape, seed: int = 0, threads: Optional[int] = None,
                 names: Optional[List[str]] = None) -> Weights:
    """Draw every bf16 tensor of ``cfg`` (or only ``names``) from its own seeded streams."""
    order = tensor_names(cfg)
    want = set(names) if names is not None else None
    bufs: Dict[str, np.ndarray] = {}
    jobs = []
    for t, (name, shape, kind) in enumerate(order):
        if want is not None and name not in want:
            continue
        buf = np.empty(int(np.prod(shape)), dtype=np.uint16)
        bufs[name] = buf.reshape(shape)
        for c, start in enumerate(range(0, buf.size, CHUNK)):
            n = min(CHUNK, buf.size - start)
            jobs.append((seed, (t, c), n, kind, buf[start:start + n]))
    with ThreadPoolExecutor(_threads(threads)) as ex:
        list(ex.map(lambda j: _fill_chunk(*j), jobs))
    return Weights(cfg=cfg, seed=seed, bf16=bufs)


def quantize_rows(w_bits: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Symmetric per-output-row int8 quantisation of a bf16 matrix [out, in].

    Returns (q int8 [out, in], s float32 [out]) with s = max|w| / 127 and
    q = clamp(round_half_even(w / s), -127, 127), computed in float32."""
    w = bf16_bits_to_f32(w_bits).reshape(w_bits.shape)
    amax = np.max(np.abs(w), axis=1)
    s = (amax / np.float32(127.0)).astype(np.float32)
    safe = np.where(s > 0, s, np.float32(1.0)).astype(np.float32)
    q = np.rint(w / safe[:, None])
    q = np.clip(q, -127, 127)
    q[s == 0, :] = 0
    return q.astype(np.int8), s


def add_w8a16(w: Weights, threads: Optional[int] = None, row_block: int = 1024) -> Weights:
    """Fill ``w.q8`` / ``w.scale`` for every projection (and an untied LM head)."""
    jobs = []
    for name in w.quantized_names():
        src = w.bf16[name]
        q = np.empty(src.shape, dtype=np.int8)
        s = np.empty(src.shape[0], dtype=np.float32)
        w.q8[name], w.scale[name] = q, s
        for r0 in range(0, src.shape[0], row_block):
            jobs.append((src, q, s, r0, min(src.shape[0], r0 + row_block)))

    def run(j):
        src, q, s, r0, r1 = j
        q[r0:r1], s[r0:r1] = quantize_rows(src[r0:r1])

    with ThreadPoolExecutor(_threads(threads)) as ex:
        list(ex.map(run, jobs))
    return w


def pack_int4(q: np.ndarray) -> np.ndarray:
    """Pack int4 codes q in [-8, 7] of a matrix [out, in] (in a multiple of 8)
    into bytes [out, in / 2]: the 4 bytes of each 32-bit little-endian word d
    hold columns 8d .. 8d + 7, byte 4d + b carrying q[8d + b] + 8 in its low
    nibble and q[8d + 4 + b] + 8 in its high nibble."""
    q = np.asarray(q)
    if q.ndim != 2 or q.shape[1] % 8:
        raise ValueError("need [out, in] with in a multiple of 8")
    if q.min(initial=0) < -8 or q.max(initial=0) > 7:
        raise ValueError("int4 codes outside [-8, 7]")
    u = (q.astype(np.int16) + 8).astype(np.uint8).reshape(q.shape[0], q.shape[1] // 8, 2, 4)
    return (u[:, :, 0, :] | (u[:, :, 1, :] << np.uint8(4))).reshape(q.shape[0], q.shape[1] // 2)


def quantize_groups4(w_bits: np.ndarray, group: int) -> Tuple[np.ndarray, np.ndarray]:
    """Symmetric round-to-nearest int4 quantisation of a bf16 matrix [out, in]
    with one fp16 scale per row and ``group`` consecutive input columns.

    Returns (packed uint8 [out, in / 2] in the ``pack_int4`` layout,
    s float16 [out, in / group]) with s = fp16(max|w| / 7) and
    q = clamp(round_half_even(w / s), -8, 7) computed in float32 with the
    stored scale (q = 0 where s == 0)."""
    w = bf16_bits_to_f32(w_bits).reshape(w_bits.shape)
    out, k = w.shape
    if group < 8 or group % 8 or k % group:
        raise ValueError(f"group {group} must be a multiple of 8 dividing {k}")
    wg = w.reshape(out, k // group, group)
    s16 = (np.max(np.abs(wg), axis=2) / np.float32(7.0)).astype(np.float16)
    if not np.all(np.isfinite(s16)):
        raise OverflowError("int4 scale outside the fp16 range")
    s32 = s16.astype(np.float32)
    safe = np.where(s32 > 0, s32, np.float32(1.0)).astype(np.float32)
    q = np.clip(np.rint(wg / safe[:, :, None]), -8, 7)
    q[s32 == 0, :] = 0
    return pack_int4(q.reshape(out, k).astype(np.int8)), s16


def add_w4a16(w: Weights, group: Optional[int] = None, threads: Optional[int] = None,
              row_block: int = 1024) -> Weights:
    """Fill ``w.q4`` / ``w.scale4`` / ``w.group4`` for every projection (and an untied LM head)."""
    g = group if group else w.cfg.int4_group
    w.group4 = g
    jobs = []
    for name in w.quantized_names():
        src = w.bf16[name]
        q = np.empty((src.shape[0], src.shape[1] // 2), dtype=np.uint8)
        s = np.empty((src.shape[0], src.shape[1] // g), dtype=np.float16)
        w.q4[name], w.scale4[name] = q, s
        for r0 in range(0, src.shape[0], row_block):
            jobs.append((src, q, s, r0, min(src.shape[0], r0 + row_block)))

    def run(j):
        src, q, s, r0, r1 = j
        q[r0:r1], s[r0:r1] = quantize_groups4(src[r0:r1], g)

    with ThreadPoolExecutor(_threads(threads)) as ex:
        list(ex.map(run, jobs))
    return w


def kv_cache_shape(cfg: ModelShape, max_seq: Optional[int] = None) -> Tuple[int, ...]:
    """KV cache layout: [layer][K=0 / V=1][kv_head][position][head_dim], bf16."""
    S = max_seq if max_seq is not None else cfg.seq_capacity
    return (cfg.n_layers, 2, cfg.n_kv_heads, S, cfg.head_dim)


def make_kv_cache(cfg: ModelShape, pos: int, seed: int = 1, max_seq: Optional[int] = None,
                  threads: Optional[int] = None) -> np.ndarray:
    """bf16 KV cache with slots [0, pos) drawn N(0, 1) and the rest zero."""
    shape = kv_cache_shape(cfg, max_seq)
    if pos > shape[3]:
        raise ValueError("pos exceeds the cache capacity")
    kv = np.zeros(shape, dtype=np.uint16)
    if pos == 0:
        return kv
    jobs = []
    idx = 0
    for l in range(shape[0]):
        for t in range(2):
            for h in range(shape[2]):
                dst = kv[l, t, h, :pos, :].reshape(-1)
                jobs.append((seed, (_KV_STREAM + idx, 0), dst.size, "n", (l, t, h)))
                idx += 1

    def run(j):
        s, key, n, kind, (l, t, h) = j
        tmp = np.empty(n, dtype=np.uint16)
        _fill_chunk(s, key, n, kind, tmp)
        kv[l, t, h, :pos, :] = tmp.reshape(pos, shape[4])

    with ThreadPoolExecutor(_threads(threads)) as ex:
        list(ex.map(run, jobs))
    return kv
