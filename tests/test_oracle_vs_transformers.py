"""Pin the whole oracle decode step against an independent implementation of
the same model family: transformers' LlamaForCausalLM (CPU, float32) with the
same weights.  A dropped term, a wrong sign, a transposed operand or a wrong
GQA/RoPE convention anywhere in the oracle breaks these tests; the mutation
tests below plant such mistakes in the oracle and check that they do."""
import numpy as np
import pytest
import torch

import oracle
import oracle.decode as od
import synth

STEPS = 8


def _hf_model(cfg, weights, fmt="bf16"):
    from transformers import LlamaConfig, LlamaForCausalLM

    hc = LlamaConfig(hidden_size=cfg.hidden, intermediate_size=cfg.intermediate,
                     num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
                     num_key_value_heads=cfg.n_kv_heads, head_dim=cfg.head_dim, vocab_size=cfg.vocab,
                     rms_norm_eps=cfg.rms_eps, tie_word_embeddings=cfg.tied_embeddings,
                     rope_parameters={"rope_type": "default", "rope_theta": cfg.rope_theta},
                     max_position_embeddings=4096, attention_bias=False, mlp_bias=False,
                     hidden_act="silu")
    hc._attn_implementation = "eager"
    m = LlamaForCausalLM(hc).eval()

    def bf(name):
        return torch.from_numpy(synth.bf16_bits_to_f32(weights.bf16[name]).reshape(weights.bf16[name].shape))

    def mat(name):
        if fmt == "w8a16" and name in weights.q8:
            return torch.from_numpy(weights.q8[name].astype(np.float32) * weights.scale[name][:, None])
        return bf(name)

    sd = {"model.embed_tokens.weight": bf("embed"), "model.norm.weight": bf("final_norm")}
    hf_names = {"wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
                "wo": "self_attn.o_proj", "wg": "mlp.gate_proj", "wu": "mlp.up_proj", "wd": "mlp.down_proj"}
    for l in range(cfg.n_layers):
        for ours, theirs in hf_names.items():
            sd[f"model.layers.{l}.{theirs}.weight"] = mat(f"layers.{l}.{ours}")
        sd[f"model.layers.{l}.input_layernorm.weight"] = bf(f"layers.{l}.attn_norm")
        sd[f"model.layers.{l}.post_attention_layernorm.weight"] = bf(f"layers.{l}.mlp_norm")
    sd["lm_head.weight"] = mat("embed" if cfg.tied_embeddings else "lm_head")
    missing, unexpected = m.load_state_dict(sd, strict=False)
    assert not unexpected and all("rotary" in k for k in missing), (missing, unexpected)
    return m


def _hf_greedy(m, token, steps):
    from transformers import DynamicCache
    cache = DynamicCache()
    toks, logits = [], []
    t = token
    with torch.no_grad():
        for i in range(steps):
            out = m(input_ids=torch.tensor([[t]]), past_key_values=cache, use_cache=True,
                    position_ids=torch.tensor([[i]]))
            cache = out.past_key_values
            lg = out.logits[0, -1].double().numpy()
            t = int(np.argmax(lg))
            toks.append(t)
            logits.append(lg)
    return toks, logits


def _oracle_greedy(cfg, weights, fmt, steps, dtype=np.float32):
    kv = np.zeros(synth.kv_cache_shape(cfg), dtype=np.float64)
    return oracle.greedy(oracle.OracleModel(weights, fmt, dtype), 1, 0, steps, kv, round_kv=False)


@pytest.fixture(scope="module")
def hf_ref(tiny_cfg, tiny_weights):
    torch.manual_seed(0)
    return {fmt: _hf_greedy(_hf_model(tiny_cfg, tiny_weights, fmt), 1, STEPS) for fmt in ("bf16", "w8a16")}


@pytest.mark.parametrize("fmt", ["bf16", "w8a16"])
def test_oracle_equals_transformers(tiny_cfg, tiny_weights, hf_ref, fmt):
    toks, logits = _oracle_greedy(tiny_cfg, tiny_weights, fmt, STEPS)
    ref_toks, ref_logits = hf_ref[fmt]
    assert toks == ref_toks
    for a, b in zip(logits, ref_logits):
        assert np.max(np.abs(a - b)) < 2e-5


def test_oracle_equals_transformers_tied(tiny_cfg):
    cfg = tiny_cfg.with_(tied_embeddings=True, n_kv_heads=1, rope_theta=500000.0)
    w = synth.make_weights(cfg, seed=3)
    toks, logits = _oracle_greedy(cfg, w, "bf16", 4)
    ref_toks, ref_logits = _hf_greedy(_hf_model(cfg, w), 1, 4)
    assert toks == ref_toks
    assert max(np.max(np.abs(a - b)) for a, b in zip(logits, ref_logits)) < 2e-5


# ---------------------------------------------------------------- mutations
def _mut_rope_sign(u, pos, theta):
    d = u.shape[-1]
    c, s = od.rope_angles(pos, d, theta)
    lo, hi = u[..., : d // 2], u[..., d // 2:]
    return np.concatenate([lo * c + hi * s, hi * c - lo * s], axis=-1).astype(u.dtype)


def _mut_rope_interleaved(u, pos, theta):
    d = u.shape[-1]
    c, s = od.rope_angles(pos, d, theta)
    a, b = u[..., 0::2], u[..., 1::2]
    out = np.empty_like(u)
    out[..., 0::2], out[..., 1::2] = a * c - b * s, b * c + a * s
    return out


def _mut_rmsnorm_no_mean(x, g, eps):
    return x / np.sqrt(np.sum(x * x) + eps) * g


def _mut_attn_no_scale(q, K, V):
    n_heads, d = q.shape
    group = n_heads // K.shape[0]
    out = np.empty_like(q)
    for h in range(n_heads):
        p = od.softmax(K[h // group] @ q[h])
        out[h] = p @ V[h // group]
    return out


def _mut_attn_modulo_group(q, K, V):
    n_heads, d = q.shape
    out = np.empty_like(q)
    for h in range(n_heads):
        kv = h % K.shape[0]
        p = od.softmax((K[kv] @ q[h]) / np.sqrt(d))
        out[h] = p @ V[kv]
    return out


def _mut_linear_transposed(W, x):
    if W.shape[0] == W.shape[1]:
        return W.T @ x
    return W @ x


def _mut_silu_sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


MUTATIONS = {
    "rope_sign": ("rope", lambda u, p, t: _mut_rope_sign(u, p, t)),
    "rope_interleaved": ("rope", lambda u, p, t: _mut_rope_interleaved(u, p, t)),
    "rmsnorm_sum": ("rmsnorm", _mut_rmsnorm_no_mean),
    "attn_no_scale": ("attention", _mut_attn_no_scale),
    "attn_modulo_group": ("attention", _mut_attn_modulo_group),
    "linear_transposed": ("linear", _mut_linear_transposed),
    "silu_is_sigmoid": ("silu", _mut_silu_sigmoid),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(tiny_cfg, tiny_weights, hf_ref, monkeypatch, name):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(od, attr, fn)
    toks, logits = _oracle_greedy(tiny_cfg, tiny_weights, "bf16", 3)
    ref_toks, ref_logits = hf_ref["bf16"]
    worst = max(np.max(np.abs(a - b)) for a, b in zip(logits, ref_logits[:3]))
    assert worst > 1e-3, f"mutation {name} not detected (max diff {worst})"


def test_planted_missing_residual_is_caught(tiny_cfg, tiny_weights, hf_ref, monkeypatch):
    real = od.linear
    calls = {"n": 0}

    def drop_down_proj(W, x):
        calls["n"] += 1
        y = real(W, x)
        # the down projection is the only product whose input length is the intermediate size
        return y * 0 if x.shape[0] == tiny_cfg.intermediate else y

    monkeypatch.setattr(od, "linear", drop_down_proj)
    _, logits = _oracle_greedy(tiny_cfg, tiny_weights, "bf16", 1)
    assert np.max(np.abs(logits[0] - hf_ref["bf16"][1][0])) > 1e-3
