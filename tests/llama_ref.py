"""An independent LLaMA forward for pinning the oracle: Hugging Face Transformers'
LlamaForCausalLM (the target-model code the paper ran, Appendix: Hardware and
Software), loaded with the synthetic weights and run in float64 on the CPU.

It shares nothing with the oracle beyond the seeded weights it is given.
"""
from __future__ import annotations

import numpy as np


def build(shape, get_tensor, drop_layers=()):
    import torch
    from transformers import LlamaConfig, LlamaForCausalLM

    keep = [l for l in range(shape.n_layers) if l not in set(drop_layers)]
    cfg = LlamaConfig(
        vocab_size=shape.vocab, hidden_size=shape.d_model, intermediate_size=shape.ffn_dim,
        num_hidden_layers=len(keep), num_attention_heads=shape.n_heads, num_key_value_heads=shape.n_heads,
        head_dim=shape.head_dim, max_position_embeddings=8192, rms_norm_eps=shape.rms_eps,
        rope_theta=shape.rope_base, tie_word_embeddings=False, attention_bias=False, mlp_bias=False,
    )
    cfg._attn_implementation = "eager"
    torch.manual_seed(0)
    m = LlamaForCausalLM(cfg).eval().to(torch.float64)

    def put(param, arr):
        with torch.no_grad():
            param.copy_(torch.from_numpy(np.asarray(arr, dtype=np.float64)))

    put(m.model.embed_tokens.weight, get_tensor("embed", -1))
    for j, l in enumerate(keep):
        lay = m.model.layers[j]
        put(lay.input_layernorm.weight, get_tensor("attn_norm", l))
        put(lay.self_attn.q_proj.weight, get_tensor("wq", l))
        put(lay.self_attn.k_proj.weight, get_tensor("wk", l))
        put(lay.self_attn.v_proj.weight, get_tensor("wv", l))
        put(lay.self_attn.o_proj.weight, get_tensor("wo", l))
        put(lay.post_attention_layernorm.weight, get_tensor("mlp_norm", l))
        put(lay.mlp.gate_proj.weight, get_tensor("w_gate", l))
        put(lay.mlp.up_proj.weight, get_tensor("w_up", l))
        put(lay.mlp.down_proj.weight, get_tensor("w_down", l))
    put(m.model.norm.weight, get_tensor("final_norm", -1))
    put(m.lm_head.weight, get_tensor("lm_head", -1))
    return m


def logits(model, tokens) -> np.ndarray:
    """Causal forward over one token sequence; logits [T][V] in float64."""
    import torch
    ids = torch.as_tensor(np.asarray(tokens, dtype=np.int64))[None, :]
    with torch.no_grad():
        out = model(input_ids=ids, use_cache=False)
    return out.logits[0].double().numpy()
