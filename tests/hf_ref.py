"""Independent textbook LLaMA decoder layer (Hugging Face transformers) used to
pin the oracle.  A cascade layer of FastEagle is a single pre-norm LLaMA
decoder layer (Section 2.1); evaluated over a whole causal sequence, its last
row must equal the oracle's decode-style computation over a prefix KV cache.
"""
from __future__ import annotations

import numpy as np
import torch

_HF = None


def _hf():
    global _HF
    if _HF is None:
        from transformers import LlamaConfig
        from transformers.models.llama import modeling_llama as ml
        _HF = (LlamaConfig, ml)
    return _HF


def llama_config(cfg):
    LlamaConfig, _ = _hf()
    c = LlamaConfig(hidden_size=cfg.hidden, num_attention_heads=cfg.n_q_heads,
                    num_key_value_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                    intermediate_size=cfg.intermediate, rope_theta=float(cfg.rope_theta),
                    rms_norm_eps=float(cfg.rms_eps), attention_bias=False, mlp_bias=False,
                    max_position_embeddings=1 << 16, vocab_size=cfg.draft_vocab)
    c._attn_implementation = "eager"
    return c


def decoder_layer(cfg, lw, widen):
    """HF LlamaDecoderLayer in float64 holding one cascade layer's weights."""
    _, ml = _hf()
    layer = ml.LlamaDecoderLayer(llama_config(cfg), 0).double().eval()
    t = lambda a: torch.from_numpy(widen(a))
    with torch.no_grad():
        layer.self_attn.q_proj.weight.copy_(t(lw.wq))
        layer.self_attn.k_proj.weight.copy_(t(lw.wk))
        layer.self_attn.v_proj.weight.copy_(t(lw.wv))
        layer.self_attn.o_proj.weight.copy_(t(lw.wo))
        layer.mlp.gate_proj.weight.copy_(t(lw.w_gate))
        layer.mlp.up_proj.weight.copy_(t(lw.w_up))
        layer.mlp.down_proj.weight.copy_(t(lw.w_down))
        layer.input_layernorm.weight.copy_(t(lw.attn_norm))
        layer.post_attention_layernorm.weight.copy_(t(lw.mlp_norm))
    return layer


def rotary(cfg):
    _, ml = _hf()
    return ml.LlamaRotaryEmbedding(llama_config(cfg))


def run_sequence(cfg, layer, seq: np.ndarray, positions: np.ndarray):
    """Run the layer over seq [L, d] (float64) with a causal mask and the given
    position ids.  Returns (outputs [L, d], rotated K [L, Hkv, D], V [L, Hkv, D])."""
    _, ml = _hf()
    L = seq.shape[0]
    x = torch.from_numpy(np.ascontiguousarray(seq, dtype=np.float64))[None]
    pos = torch.from_numpy(np.asarray(positions, dtype=np.int64))[None]
    cos, sin = rotary(cfg)(x, pos)
    cos, sin = cos.double(), sin.double()
    mask = torch.full((L, L), torch.finfo(torch.float64).min, dtype=torch.float64).triu(1)[None, None]
    captured = {}
    h1 = layer.self_attn.k_proj.register_forward_hook(lambda m, i, o: captured.__setitem__("k", o))
    h2 = layer.self_attn.v_proj.register_forward_hook(lambda m, i, o: captured.__setitem__("v", o))
    try:
        with torch.no_grad():
            out = layer(x, attention_mask=mask, position_ids=pos, position_embeddings=(cos, sin))
    finally:
        h1.remove()
        h2.remove()
    out = out[0] if isinstance(out, tuple) else out
    D, Hkv = cfg.head_dim, cfg.n_kv_heads
    k = captured["k"].view(1, L, Hkv, D).transpose(1, 2)       # [1, Hkv, L, D]
    q_dummy = torch.zeros_like(k)
    _, k_rot = ml.apply_rotary_pos_emb(q_dummy, k, cos, sin)
    k_rot = k_rot.transpose(1, 2)[0].numpy()                    # [L, Hkv, D]
    v = captured["v"].view(L, Hkv, D).numpy()
    return out[0].detach().numpy(), k_rot, v
