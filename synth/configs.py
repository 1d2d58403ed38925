"""Model shapes of the Llama-family decoders the decode step is exercised on.

These are plain shape records: no arithmetic of the method lives here.  The
five shapes follow the workloads the paper's evaluation talks about (a tiny
toy decoder, SmolLM2-135M, TinyLlama-1.1B, a Llama-3.2-1B-shaped model and a
Llama-3-8B-shaped model; paper §5 "Correctness and retargeting",
"Performance scaling and roofline", Table tab:int8), with random weights
instead of checkpoints.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Dict, List, Tuple


@dataclass(frozen=True)
class ModelShape:
    name: str
    hidden: int
    n_layers: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    intermediate: int
    vocab: int
    tied_embeddings: bool
    rope_theta: float
    rms_eps: float = 1e-5
    # positions the workload decodes at (single steps) and greedy step count
    positions: Tuple[int, ...] = (0,)
    greedy_steps: int = 1
    max_seq: int = 0  # 0 -> derived: max(positions) + greedy_steps + 1

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads

    @property
    def seq_capacity(self) -> int:
        if self.max_seq:
            return self.max_seq
        return max(self.positions) + self.greedy_steps + 1

    @property
    def int4_group(self) -> int:
        """Default W4A16 group: the largest of 128, 64, 32 that divides every
        projection's input width (hidden, intermediate, n_heads * head_dim)."""
        for g in (128, 64, 32):
            if self.hidden % g == 0 and self.intermediate % g == 0 and self.q_dim % g == 0:
                return g
        raise ValueError(f"{self.name}: no int4 group of 32, 64 or 128 divides every input width")

    def with_(self, **kw) -> "ModelShape":
        return replace(self, **kw)

    # ---- byte accounting (used by the benchmark's roofline) -------------
    def linear_shapes(self) -> List[Tuple[str, int, int]]:
        """(name, out_features, in_features) of the seven per-layer projections."""
        H, I = self.hidden, self.intermediate
        return [("wq", self.q_dim, H), ("wk", self.kv_dim, H), ("wv", self.kv_dim, H),
                ("wo", H, self.q_dim), ("wg", I, H), ("wu", I, H), ("wd", H, I)]

    def algorithmic_bytes(self, fmt: str, pos: int, group: int = 0) -> int:
        """HBM bytes one decode step must read at least once.

        All GEMV weights (+ fp32 per-row scales for int8, fp16 per-group
        scales for int4 with ``group`` columns per scale, default
        ``int4_group``), the norm vectors,
        one gathered embedding row and the K and V rows 0..pos of every layer
        and KV head.  Writes (one K/V row per layer, the logits) are below
        0.01% of this on the large shapes and are not counted."""
        H, L, V = self.hidden, self.n_layers, self.vocab
        lin_elems = sum(o * i for _, o, i in self.linear_shapes()) * L
        lin_rows = sum(o for _, o, _ in self.linear_shapes()) * L
        norms = (2 * L + 1) * H * 2
        emb_row = H * 2
        if fmt == "bf16":
            lin = lin_elems * 2
            lm = V * H * 2
        elif fmt == "w8a16":
            lin = lin_elems + 4 * lin_rows
            lm = V * H * 2 if self.tied_embeddings else V * H + 4 * V
        elif fmt == "w4a16":
            g = group or self.int4_group
            lin = lin_elems // 2 + 2 * (lin_elems // g)
            lm = V * H * 2 if self.tied_embeddings else V * H // 2 + 2 * (V * H // g)
        else:
            raise ValueError(fmt)
        kv_read = L * 2 * self.n_kv_heads * (pos + 1) * self.head_dim * 2
        return lin + lm + norms + emb_row + kv_read


CONFIGS: Dict[str, ModelShape] = {
    "tiny": ModelShape("tiny", hidden=256, n_layers=4, n_heads=4, n_kv_heads=2, head_dim=64,
                       intermediate=688, vocab=4096, tied_embeddings=False, rope_theta=10000.0,
                       positions=(0,), greedy_steps=8),
    "smollm2_135m": ModelShape("smollm2_135m", hidden=576, n_layers=30, n_heads=9, n_kv_heads=3,
                               head_dim=64, intermediate=1536, vocab=49152, tied_embeddings=True,
                               rope_theta=10000.0, positions=(0,), greedy_steps=32),
    "tinyllama_1b": ModelShape("tinyllama_1b", hidden=2048, n_layers=22, n_heads=32, n_kv_heads=4,
                               head_dim=64, intermediate=5632, vocab=32000, tied_embeddings=False,
                               rope_theta=10000.0, positions=(0, 1024)),
    "llama32_1b": ModelShape("llama32_1b", hidden=2048, n_layers=16, n_heads=32, n_kv_heads=8,
                             head_dim=64, intermediate=8192, vocab=128256, tied_embeddings=True,
                             rope_theta=500000.0, positions=(0, 4096)),
    "llama3_8b": ModelShape("llama3_8b", hidden=4096, n_layers=32, n_heads=32, n_kv_heads=8,
                            head_dim=128, intermediate=14336, vocab=128256, tied_embeddings=False,
                            rope_theta=500000.0, positions=(0, 8192)),
}


def get(name: str) -> ModelShape:
    return CONFIGS[name]
