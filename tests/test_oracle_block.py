"""Pin the oracle's decoder against independent library implementations.

The decoder maths (RMSNorm, rotate-half RoPE, grouped-query causal attention,
SwiGLU, tied/untied heads, Qwen's QKV bias) is checked against Hugging Face's
Llama / Qwen2 modules run in float64, and attention / normalisation against
torch's own routines.  These share no code with the oracle.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from dataclasses import replace

import oracle
import pard_inputs as pi
from oracle.model import attention, rms_norm, rope, rope_inv_freq

transformers = pytest.importorskip("transformers")


def _hf_model(spec, weights, family):
    common = dict(vocab_size=spec.vocab, hidden_size=spec.d_model,
                  intermediate_size=spec.ffn_dim, num_hidden_layers=spec.n_layers,
                  num_attention_heads=spec.n_heads, num_key_value_heads=spec.n_kv_heads,
                  rms_norm_eps=spec.rms_eps, rope_theta=spec.rope_theta,
                  tie_word_embeddings=spec.tied, max_position_embeddings=4096)
    if spec.rope_scaling is not None:
        factor, low, high, orig = spec.rope_scaling
        common["rope_scaling"] = {"rope_type": "llama3", "factor": factor, "low_freq_factor": low,
                                  "high_freq_factor": high, "original_max_position_embeddings": orig}
    if family == "llama":
        cfg = transformers.LlamaConfig(head_dim=spec.head_dim, attention_bias=False,
                                       mlp_bias=False, **common)
        cls = transformers.LlamaForCausalLM
    else:
        cfg = transformers.Qwen2Config(**common)
        cls = transformers.Qwen2ForCausalLM
    cfg._attn_implementation = "eager"
    m = cls(cfg).double().eval()
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    sd = {"model.embed_tokens.weight": t(weights["embed"]),
          "model.norm.weight": t(weights["final_norm"])}
    if not spec.tied:
        sd["lm_head.weight"] = t(weights["lm_head"])
    for l, lw in weights["layers"].items():
        p = f"model.layers.{l}."
        sd[p + "self_attn.q_proj.weight"] = t(lw["wq"])
        sd[p + "self_attn.k_proj.weight"] = t(lw["wk"])
        sd[p + "self_attn.v_proj.weight"] = t(lw["wv"])
        sd[p + "self_attn.o_proj.weight"] = t(lw["wo"])
        sd[p + "mlp.gate_proj.weight"] = t(lw["w_gate"])
        sd[p + "mlp.up_proj.weight"] = t(lw["w_up"])
        sd[p + "mlp.down_proj.weight"] = t(lw["w_down"])
        sd[p + "input_layernorm.weight"] = t(lw["attn_norm"])
        sd[p + "post_attention_layernorm.weight"] = t(lw["mlp_norm"])
        if spec.qkv_bias:
            sd[p + "self_attn.q_proj.bias"] = t(lw["bq"])
            sd[p + "self_attn.k_proj.bias"] = t(lw["bk"])
            sd[p + "self_attn.v_proj.bias"] = t(lw["bv"])
    missing, unexpected = m.load_state_dict(sd, strict=False)
    assert not unexpected
    assert all(k == "lm_head.weight" for k in missing)   # tied head aliases the embedding
    if spec.tied:
        assert m.lm_head.weight.data_ptr() == m.model.embed_tokens.weight.data_ptr()
    return m


def _tiny_qwen_like():
    # A small Qwen2-family shape: QKV bias, tied embeddings, group size 7 as in
    # Qwen2.5-0.5B / 7B (14 query heads over 2 KV heads).
    return pi.ModelSpec(n_layers=2, d_model=224, n_heads=14, n_kv_heads=2, head_dim=16,
                        ffn_dim=96, vocab=512, rms_eps=1e-6, rope_theta=1e6, qkv_bias=True,
                        tied=True, dtype="bf16", seed=9, stream=0)


# LLaMA-3.1-style rotary scaling with an original length of 32 positions: at
# head_dim 64 and theta 1e4 the wavelengths span the kept, blended and divided
# regimes (below 8, 8..32, above 32)
SCALING = (8.0, 1.0, 4.0, 32)


@pytest.mark.parametrize("which", ["target", "draft", "qwen", "target_scaled"])
def test_forward_full_matches_hf(which):
    wl = pi.WORKLOADS["tiny"]
    spec = {"target": wl.target, "draft": wl.draft, "qwen": _tiny_qwen_like(),
            "target_scaled": replace(wl.target, rope_scaling=SCALING)}[which]
    family = "qwen" if which == "qwen" else "llama"
    model = oracle.build_model(spec)
    ids = pi.gen_prompt(5, spec.vocab, 48)
    ours = oracle.forward_full(model, ids)
    hf = _hf_model(spec, model.weights, family)
    with torch.no_grad():
        ref = hf(input_ids=torch.from_numpy(ids.astype(np.int64))[None]).logits[0].numpy()
    # HF evaluates its rotary angles in float32; everything else is float64.
    scale = np.abs(ref).max()
    assert np.abs(ours - ref).max() <= 1e-5 * max(1.0, scale)
    assert np.array_equal(np.argmax(ours, -1), np.argmax(ref, -1)) or \
        np.abs(ours - ref).max() < 1e-6


def test_rope_scaling_matches_hf_frequencies_and_regimes():
    from transformers.modeling_rope_utils import ROPE_INIT_FUNCTIONS
    cfg = transformers.LlamaConfig(hidden_size=256, num_attention_heads=4, head_dim=64, rope_theta=1e4,
                                   rope_scaling={"rope_type": "llama3", "factor": 8.0, "low_freq_factor": 1.0,
                                                 "high_freq_factor": 4.0, "original_max_position_embeddings": 32})
    hf, _ = ROPE_INIT_FUNCTIONS["llama3"](cfg, "cpu")
    ours = rope_inv_freq(64, 1e4, SCALING)
    assert np.allclose(ours, hf.double().numpy(), rtol=1e-6, atol=0)
    plain = rope_inv_freq(64, 1e4)
    wavelen = 2 * np.pi / plain
    kept, divided = wavelen < 8, wavelen > 32
    assert kept.any() and divided.any() and (~kept & ~divided).any()
    assert np.array_equal(ours[kept], plain[kept])
    assert np.allclose(ours[divided], plain[divided] / 8, rtol=1e-15)
    mid = ~kept & ~divided                                           # blended: between w / 8 and w
    assert np.all((ours[mid] <= plain[mid]) & (ours[mid] >= plain[mid] / 8))


def test_attention_matches_torch_sdpa_gqa():
    rng = np.random.default_rng(0)
    n, hq, hkv, hd = 11, 8, 2, 32
    q, k, v = (rng.standard_normal((n, h, hd)) for h in (hq, hkv, hkv))
    pos = np.arange(n)
    ours = attention(q, k, v, pos, pos)
    tq, tk, tv = (torch.from_numpy(a).permute(1, 0, 2)[None] for a in (q, k, v))
    ref = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True, enable_gqa=True)
    assert np.allclose(ours, ref[0].permute(1, 0, 2).numpy(), atol=1e-12, rtol=0)


def test_attention_offset_queries_match_sdpa_mask():
    # A block of queries after a cached prefix: the causal rule is by absolute position.
    rng = np.random.default_rng(1)
    m, n, hq, hkv, hd = 20, 5, 4, 4, 16
    q = rng.standard_normal((n, hq, hd))
    k, v = rng.standard_normal((m, hkv, hd)), rng.standard_normal((m, hkv, hd))
    qpos, kpos = np.arange(m - n, m), np.arange(m)
    ours = attention(q, k, v, qpos, kpos)
    mask = torch.from_numpy(kpos[None, :] <= qpos[:, None])
    tq, tk, tv = (torch.from_numpy(a).permute(1, 0, 2)[None] for a in (q, k, v))
    ref = F.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask)
    assert np.allclose(ours, ref[0].permute(1, 0, 2).numpy(), atol=1e-12, rtol=0)


def test_rms_norm_matches_torch():
    rng = np.random.default_rng(2)
    x, g = rng.standard_normal((7, 96)) * 3, rng.standard_normal(96)
    ref = F.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), eps=1e-5).numpy()
    assert np.allclose(rms_norm(x, g, 1e-5), ref, atol=1e-12, rtol=0)


def test_rope_two_dims_is_plane_rotation_by_position():
    # head_dim 2: the single frequency is theta**0 = 1 rad per position.
    x = np.array([[[1.0, 0.0]], [[0.3, -0.7]]])
    pos = np.array([1, 5])
    out = rope(x, pos, 1e4)
    for i in range(2):
        c, s = np.cos(pos[i]), np.sin(pos[i])
        R = np.array([[c, -s], [s, c]])
        assert np.allclose(out[i, 0], R @ x[i, 0], atol=1e-15)


def test_rope_scores_depend_on_relative_position_only():
    rng = np.random.default_rng(3)
    q, k = rng.standard_normal((1, 1, 64)), rng.standard_normal((1, 1, 64))
    d1 = (rope(q, np.array([40]), 5e5) * rope(k, np.array([33]), 5e5)).sum()
    d2 = (rope(q, np.array([1007]), 5e5) * rope(k, np.array([1000]), 5e5)).sum()
    assert abs(d1 - d2) < 1e-10
    assert np.allclose(np.linalg.norm(rope(q, np.array([123]), 1e4)), np.linalg.norm(q))
