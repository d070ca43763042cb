"""Decoder shapes used by the verification-step workloads.

The 7B and 13B shapes are the LLaMA target models of the paper's evaluation
(Appendix, Experimental Setup / Models: Vicuna-7B with 32 layers, hidden 4096,
32 heads, intermediate 11008, vocabulary 32000; Llama-2-13B with 40 layers,
hidden 5120, 40 heads, intermediate 13824).  The tiny shape is a 4-layer
decoder small enough for the plain CPU oracle to finish in seconds, and the
33B shape is a LLaMA-33B-sized decoder for a one-GPU, 65 GB weight footprint.
All shapes use multi-head attention (one KV head per query head), SwiGLU MLPs,
RMSNorm and rotate-half rotary embeddings with base 10000.
"""
from dataclasses import dataclass


@dataclass(frozen=True)
class ModelShape:
    name: str
    shape_id: int          # stable integer used to key the seeded generators
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    dtype: str = "bf16"    # storage/compute type of weights and KV on the GPU: "bf16" or "f32"
    rope_base: float = 10000.0
    rms_eps: float = 1e-6

    @property
    def n_tensors(self) -> int:
        return n_tensors(self.n_layers)


# Tensor order of one model: embed; per layer the nine tensors below; final_norm; lm_head.
LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")


def n_tensors(n_layers: int) -> int:
    return 3 + len(LAYER_TENSORS) * n_layers


def tensor_names(n_layers: int):
    """(index, layer, name) for every tensor of a model, in load order."""
    out = [(0, -1, "embed")]
    for l in range(n_layers):
        for j, nm in enumerate(LAYER_TENSORS):
            out.append((1 + len(LAYER_TENSORS) * l + j, l, nm))
    out.append((1 + len(LAYER_TENSORS) * n_layers, -1, "final_norm"))
    out.append((2 + len(LAYER_TENSORS) * n_layers, -1, "lm_head"))
    return out


def tensor_shape(shape: ModelShape, name: str):
    d, f, v = shape.d_model, shape.ffn_dim, shape.vocab
    return {
        "embed": (v, d), "lm_head": (v, d),
        "attn_norm": (d,), "mlp_norm": (d,), "final_norm": (d,),
        "wq": (d, d), "wk": (d, d), "wv": (d, d), "wo": (d, d),
        "w_gate": (f, d), "w_up": (f, d), "w_down": (d, f),
    }[name]


TINY = ModelShape("tiny-4L-d256", 1, n_layers=4, d_model=256, n_heads=4, head_dim=64,
                  ffn_dim=704, vocab=4096, dtype="f32")
LLAMA_7B = ModelShape("llama-7b-shape", 2, n_layers=32, d_model=4096, n_heads=32, head_dim=128,
                      ffn_dim=11008, vocab=32000)
LLAMA_13B = ModelShape("llama-13b-shape", 3, n_layers=40, d_model=5120, n_heads=40, head_dim=128,
                       ffn_dim=13824, vocab=32000)
LLAMA_33B = ModelShape("llama-33b-shape", 4, n_layers=60, d_model=6656, n_heads=52, head_dim=128,
                       ffn_dim=17920, vocab=32000)

SHAPES = {s.name: s for s in (TINY, LLAMA_7B, LLAMA_13B, LLAMA_33B)}
