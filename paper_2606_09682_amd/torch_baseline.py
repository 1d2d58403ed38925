"""Same-node reference decode in plain PyTorch-ROCm: per-op eager, or the same
ops captured once into a HIP graph and replayed (paper §5 "Baselines": the
eager and graph-captured library decodes the megakernel is compared with).

This is a BASELINE for context, not the product: every projection is one
torch.nn.functional.linear call on bf16 weights (rocBLAS / hipBLASLt GEMV),
every other step a handful of stock torch kernels, so a step is a few hundred
kernel launches instead of one.  It reads the same device tensors the library
reads (bf16 bit patterns as int16; W8A16 and W4A16 are dequantised to bf16
once at construction, so those variants stream bf16 bytes like a naive
weight-only deployment does) and writes the same KV-cache layout.

Precision, the usual bf16 inference layout: each GEMV takes a bf16 input and
returns a bf16 output (fp32 accumulation inside the library), while the
residual stream, the norms, RoPE, softmax and the attention products stay in
fp32 and the appended K/V rows are rounded to bf16 like the library's.  The
bf16 rounding of GEMV inputs and outputs is an error the library does not
make, so this baseline is checked against the oracle on the greedy token and
a looser logit bound (``logit_bound``).

HIP graph: ``GraphDecode`` captures one step for a fixed position (the
benchmark's workload is a single position) with the token in a device
tensor; replays only re-run the kernels.  argmax is taken eagerly after each
replay.
"""
from __future__ import annotations

import math
from typing import Dict

# Logit bound of the bf16-activation baseline against the fp32 oracle,
# relative to the largest |logit| of the step: the bf16 input and output of
# each of the 7 L + 1 GEMVs (and, for the quantised formats, the bf16
# rounding of the dequantised weights) carry relative rounding errors of up
# to 2^-9 that add up roughly like a random walk over the GEMV stages,
# 2^-9 * sqrt(7 * 32 + 1) = 0.03 for 32 layers; the bound allows 5%.
LOGIT_REL_TOL = 5e-2


def logit_bound(ref_logits) -> float:
    """Largest |logit - oracle logit| the baseline may show on this step."""
    import numpy as np
    return LOGIT_REL_TOL * float(np.max(np.abs(ref_logits)))


def _bf16(t):
    import torch
    return t.view(torch.bfloat16) if t.dtype == torch.int16 else t


def dequantize_to_bf16(tensors: Dict[str, object], name: str, fmt: str, group: int):
    """bf16 [out, in] copy of a quantised projection (int8 + fp32 row scales,
    or packed int4 + fp16 group scales in the library's nibble layout)."""
    import torch
    q = tensors[name]
    s = tensors[name + ".scale"]
    if fmt == "w8a16":
        return (q.to(torch.float32) * s.to(torch.float32)[:, None]).to(torch.bfloat16)
    # int4: byte 4d + b of a row holds column 8d + b (low nibble) and
    # 8d + 4 + b (high nibble), each as code + 8
    out, half = q.shape
    b = q.to(torch.int16).view(out, half // 4, 4)
    lo = (b & 0xF) - 8
    hi = ((b >> 4) & 0xF) - 8
    codes = torch.stack((lo, hi), dim=2).reshape(out, 2 * half).to(torch.float32)
    scale = s.to(torch.float32).repeat_interleave(group, dim=1)
    return (codes * scale).to(torch.bfloat16)


class TorchDecode:
    """Per-op eager decode step of a Llama-family decoder on device tensors.

    ``tensors``: the name -> device tensor map the library reads (see
    ``amk.Decoder``); ``shape``: the model's dimensions (hidden, n_layers,
    n_heads, n_kv_heads, head_dim, intermediate, vocab, rope_theta, rms_eps,
    tied_embeddings); ``fmt``: the tensors' weight format."""

    def __init__(self, shape, tensors: Dict[str, object], fmt: str, max_seq: int, group: int = 0):
        import torch
        self.s = shape
        self.fmt = fmt
        dev = tensors["embed"].device
        L = shape.n_layers
        quant = fmt in ("w8a16", "w4a16")

        def mat(name):
            if quant and name + ".scale" in tensors:
                return dequantize_to_bf16(tensors, name, fmt, group)
            return _bf16(tensors[name])

        self.embed = _bf16(tensors["embed"])
        self.layers = []
        for l in range(L):
            p = f"layers.{l}."
            self.layers.append({k: mat(p + k) for k in ("wq", "wk", "wv", "wo", "wg", "wu", "wd")})
            self.layers[-1]["attn_norm"] = _bf16(tensors[p + "attn_norm"]).to(torch.float32)
            self.layers[-1]["mlp_norm"] = _bf16(tensors[p + "mlp_norm"]).to(torch.float32)
        self.final_norm = _bf16(tensors["final_norm"]).to(torch.float32)
        self.lm = self.embed if shape.tied_embeddings else mat("lm_head")
        # RoPE: angles p * theta^(-2i/d) in float64, cos / sin stored float32
        half = shape.head_dim // 2
        inv = torch.tensor([shape.rope_theta ** (-2.0 * i / shape.head_dim) for i in range(half)],
                           dtype=torch.float64)
        ang = torch.arange(max_seq, dtype=torch.float64)[:, None] * inv[None, :]
        self.cos = torch.cos(ang).to(torch.float32).to(dev)
        self.sin = torch.sin(ang).to(torch.float32).to(dev)
        self.scale = 1.0 / math.sqrt(shape.head_dim)

    def _rmsnorm(self, x, g):
        import torch
        return x * torch.rsqrt(torch.mean(x * x) + self.s.rms_eps) * g

    def _rope(self, u, pos):
        import torch
        h = u.shape[-1] // 2
        c, s = self.cos[pos], self.sin[pos]
        a, b = u[..., :h], u[..., h:]
        return torch.cat((a * c - b * s, b * c + a * s), dim=-1)

    def step(self, token, pos: int, kv, logits) -> None:
        """One decode step: token is a 1-element int64 device tensor, kv the
        bf16 cache as int16 [L][2][n_kv][max_seq][d], logits fp32 [vocab]
        (written in place)."""
        import torch
        import torch.nn.functional as F
        s = self.s
        nq, nkv, d = s.n_heads, s.n_kv_heads, s.head_dim
        grp = nq // nkv
        kvb = _bf16(kv)
        x = self.embed.index_select(0, token).reshape(-1).to(torch.float32)
        for l, w in enumerate(self.layers):
            hb = self._rmsnorm(x, w["attn_norm"]).to(torch.bfloat16)
            q = F.linear(hb, w["wq"]).to(torch.float32).view(nq, d)
            k = F.linear(hb, w["wk"]).to(torch.float32).view(nkv, d)
            v = F.linear(hb, w["wv"])
            q = self._rope(q, pos)
            k = self._rope(k, pos)
            kvb[l, 0, :, pos].copy_(k.to(torch.bfloat16))
            kvb[l, 1, :, pos].copy_(v.view(nkv, d))
            K = kvb[l, 0, :, : pos + 1].to(torch.float32)          # [nkv, T, d]
            V = kvb[l, 1, :, : pos + 1].to(torch.float32)
            qg = (q * self.scale).view(nkv, grp, d).transpose(1, 2).contiguous()  # [nkv, d, grp]
            sc = torch.bmm(K, qg)                                    # [nkv, T, grp]
            p = torch.softmax(sc, dim=1).transpose(1, 2).contiguous()  # [nkv, grp, T]
            o = torch.bmm(p, V).reshape(nq * d)                      # [nq * d]
            x = x + F.linear(o.to(torch.bfloat16), w["wo"]).to(torch.float32)
            h2 = self._rmsnorm(x, w["mlp_norm"]).to(torch.bfloat16)
            gte = F.linear(h2, w["wg"]).to(torch.float32)
            up = F.linear(h2, w["wu"]).to(torch.float32)
            a = (gte / (1.0 + torch.exp(-gte)) * up).to(torch.bfloat16)
            x = x + F.linear(a, w["wd"]).to(torch.float32)
        hf = self._rmsnorm(x, self.final_norm).to(torch.bfloat16)
        logits.copy_(F.linear(hf, self.lm).to(torch.float32))

    def next_token(self, logits) -> int:
        import torch
        return int(torch.argmax(logits).item())


class GraphDecode:
    """The eager step at one position, captured once into a HIP graph."""

    def __init__(self, eager: TorchDecode, pos: int, kv, logits, token: int = 1, warmup: int = 2):
        import torch
        self.eager = eager
        self.pos = pos
        self.kv = kv
        self.logits = logits
        self.token = torch.tensor([token], dtype=torch.int64, device=logits.device)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for _ in range(warmup):  # library workspaces and kernels settle before capture
                eager.step(self.token, pos, kv, logits)
        torch.cuda.current_stream().wait_stream(side)
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            eager.step(self.token, pos, kv, logits)

    def step(self, token: int) -> None:
        self.token.fill_(token)
        self.graph.replay()
