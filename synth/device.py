"""Copy seeded host inputs to device tensors (plumbing only, no arithmetic)."""
from __future__ import annotations

from typing import Dict

import numpy as np

from .configs import ModelShape
from .inputs import Weights


def weights_to_device(w: Weights, fmt: str, device: str = "cuda") -> Dict[str, "object"]:
    """Name -> contiguous device tensor in the layout libamk expects.

    bf16 tensors are uploaded as torch.int16 bit patterns; under 'w8a16' the
    quantised projections are int8 with fp32 '<name>.scale' tensors, under
    'w4a16' packed uint8 [out, in/2] with fp16 '<name>.scale' tensors."""
    import torch

    out: Dict[str, object] = {}
    qset = set(w.quantized_names()) if fmt in ("w8a16", "w4a16") else set()
    for name, arr in w.bf16.items():
        if name in qset and fmt == "w8a16":
            out[name] = torch.from_numpy(np.ascontiguousarray(w.q8[name])).to(device)
            out[name + ".scale"] = torch.from_numpy(np.ascontiguousarray(w.scale[name])).to(device)
        elif name in qset:
            out[name] = torch.from_numpy(np.ascontiguousarray(w.q4[name])).to(device)
            out[name + ".scale"] = torch.from_numpy(np.ascontiguousarray(w.scale4[name])).to(device)
        else:
            out[name] = torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(device)
    return out


def kv_to_device(kv: np.ndarray, device: str = "cuda"):
    import torch

    return torch.from_numpy(np.ascontiguousarray(kv).view(np.int16)).to(device)


def kv_from_device(t) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


def config_kwargs(cfg: ModelShape, fmt: str, max_seq: int, group: int = 0) -> dict:
    kw = dict(hidden=cfg.hidden, n_layers=cfg.n_layers, n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads,
              head_dim=cfg.head_dim, intermediate=cfg.intermediate, vocab=cfg.vocab, max_seq=max_seq,
              rope_theta=cfg.rope_theta, rms_eps=cfg.rms_eps, tied_embeddings=cfg.tied_embeddings,
              weight_format=fmt)
    if fmt == "w4a16":
        kw["group_size"] = group or cfg.int4_group
    return kw
