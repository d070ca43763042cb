"""Seeded synthetic inputs for the sparse-depth verification step.

This package holds the model shapes and the seeded generators of every input
(weights, context tokens, draft chains and trees, skip masks).  It is shared by
the CPU oracle and by the GPU path's tests and benchmark, and on purpose holds
none of the method's arithmetic: no normalisation, attention, projection,
argmax or acceptance logic lives here.  Where an input depends on a model
output (a draft that follows the target's greedy tokens) the caller passes
those greedy tokens in.
"""
from .shapes import ModelShape, TINY, LLAMA_7B, LLAMA_13B, LLAMA_33B, SHAPES, tensor_names, n_tensors
from .gen import (
    BASE_SEED,
    bf16_round,
    bf16_bits,
    weight_tensor,
    context_tokens,
    chain_draft,
    random_tree,
    topk_tree_parents,
    tree_draft_tokens,
    nested_skip_masks,
    random_skip_mask,
    mask_from_layers,
    abi_tensor_loader,
)
from .drafter import ReferenceDrafter

__all__ = [
    "ModelShape", "TINY", "LLAMA_7B", "LLAMA_13B", "LLAMA_33B", "SHAPES", "tensor_names", "n_tensors",
    "BASE_SEED", "bf16_round", "bf16_bits", "weight_tensor", "context_tokens", "chain_draft",
    "random_tree", "topk_tree_parents", "tree_draft_tokens", "nested_skip_masks",
    "random_skip_mask", "mask_from_layers", "abi_tensor_loader", "ReferenceDrafter",
]
