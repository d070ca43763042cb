"""Seeded generators for every input of the verification step.

Random streams are numpy PCG64 generators keyed by
``SeedSequence(seed, spawn_key=(shape_id, purpose, ...))`` so each tensor (and
each row chunk of a large tensor) can be regenerated on its own, in any order
and in parallel.  The base seed 42 is the seed the paper's data protocol uses
(Appendix, Table 3 "Random seed").

Weights: every linear matrix and the embedding are N(0, 0.02^2) draws in fp32;
for bf16 shapes they are rounded to bf16 with round-to-nearest-even, so the
same values are exact in fp32 on the oracle side.  RMSNorm gains are 1 unless
``random_gains`` asks for N(1, 0.1^2) gains (used by tests to catch a gain
applied to the wrong index).
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .shapes import ModelShape, LAYER_TENSORS, tensor_names, tensor_shape

BASE_SEED = 42

# purposes of the random streams (second spawn-key element)
_P_WEIGHT = 1
_P_CONTEXT = 2
_P_DRAFT = 3
_P_TREE = 4
_P_MASK = 5
_P_GAIN = 6

_CHUNK_ELEMS = 1 << 22


def _rng(*key, seed=BASE_SEED) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=tuple(int(k) for k in key))))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of fp32 values rounded to bf16, round-to-nearest-even (finite inputs)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 values rounded to the nearest bf16 value (ties to even), returned as fp32."""
    return (bf16_bits(x).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _tensor_index(shape: ModelShape, name: str, layer: int) -> int:
    if name == "embed":
        return 0
    if name == "final_norm":
        return 1 + len(LAYER_TENSORS) * shape.n_layers
    if name == "lm_head":
        return 2 + len(LAYER_TENSORS) * shape.n_layers
    if not (0 <= layer < shape.n_layers):
        raise ValueError(f"layer {layer} out of range for {shape.name}")
    return 1 + len(LAYER_TENSORS) * layer + LAYER_TENSORS.index(name)


def weight_tensor(shape: ModelShape, name: str, layer: int = -1, seed: int = BASE_SEED,
                  random_gains: bool = False, threads: int | None = None,
                  as_bf16_bits: bool = False) -> np.ndarray:
    """One weight tensor of ``shape``, row-major [out][in] for matrices.

    Returns fp32 values (bf16-exact for bf16 shapes), or, with ``as_bf16_bits``,
    the uint16 bf16 bit patterns of the same values (bf16 shapes only).
    """
    ti = _tensor_index(shape, name, layer)
    dims = tensor_shape(shape, name)
    if len(dims) == 1:
        if random_gains:
            g = (1.0 + 0.1 * _rng(shape.shape_id, _P_GAIN, ti, seed=seed).standard_normal(dims[0])).astype(np.float32)
        else:
            g = np.ones(dims[0], dtype=np.float32)
        if shape.dtype == "bf16":
            g = bf16_round(g)
        return bf16_bits(g) if as_bf16_bits else g
    rows, cols = dims
    rows_per_chunk = max(1, _CHUNK_ELEMS // cols)
    chunks = [(c, r0, min(rows, r0 + rows_per_chunk)) for c, r0 in enumerate(range(0, rows, rows_per_chunk))]
    out = np.empty((rows, cols), dtype=np.uint16 if as_bf16_bits else np.float32)
    if as_bf16_bits and shape.dtype != "bf16":
        raise ValueError("bf16 bit patterns requested for an fp32 shape")

    def fill(ch):
        c, r0, r1 = ch
        buf = np.empty((r1 - r0, cols), dtype=np.float32)
        _rng(shape.shape_id, _P_WEIGHT, ti, c, seed=seed).standard_normal(out=buf, dtype=np.float32)
        buf *= np.float32(0.02)
        if shape.dtype == "bf16":
            if as_bf16_bits:
                out[r0:r1] = bf16_bits(buf)
                return
            buf = bf16_round(buf)
        out[r0:r1] = buf

    nthreads = threads or min(16, os.cpu_count() or 1)
    if nthreads <= 1 or len(chunks) == 1:
        for ch in chunks:
            fill(ch)
    else:
        with ThreadPoolExecutor(nthreads) as ex:
            list(ex.map(fill, chunks))
    return out


def context_tokens(vocab: int, n: int, seed: int = BASE_SEED, stream: int = 0) -> np.ndarray:
    """n uniform-random tokens in [0, vocab)."""
    return _rng(_P_CONTEXT, vocab, n, stream, seed=seed).integers(0, vocab, size=n, dtype=np.int64).astype(np.int32)


def _other_token(rng: np.random.Generator, vocab: int, avoid) -> int:
    avoid = set(int(a) for a in avoid)
    while True:
        t = int(rng.integers(0, vocab))
        if t not in avoid:
            return t


def chain_draft(greedy: np.ndarray, vocab: int, p_accept: float | None = None, n_greedy: int | None = None,
                seed: int = BASE_SEED, stream: int = 0) -> np.ndarray:
    """Draft chain d_1..d_k built from the target's greedy continuation g_1..g_k.

    Either each d_i equals g_i with probability ``p_accept`` (else a uniform
    token different from g_i), or the first ``n_greedy`` equal g_i and the rest
    are uniform tokens different from g_i.
    """
    greedy = np.asarray(greedy, dtype=np.int64)
    rng = _rng(_P_DRAFT, vocab, len(greedy), stream, seed=seed)
    out = np.empty(len(greedy), dtype=np.int32)
    for i, g in enumerate(greedy):
        if n_greedy is not None:
            take = i < n_greedy
        else:
            take = rng.random() < p_accept
        out[i] = g if take else _other_token(rng, vocab, [g])
    return out


def random_tree(n_nodes: int, seed: int = BASE_SEED, stream: int = 0, max_children: int | None = None) -> np.ndarray:
    """Random parent array with parent[0] = -1 and parent[i] < i."""
    rng = _rng(_P_TREE, n_nodes, stream, 1, seed=seed)
    parent = np.full(n_nodes, -1, dtype=np.int32)
    kids = np.zeros(n_nodes, dtype=np.int64)
    for i in range(1, n_nodes):
        while True:
            p = int(rng.integers(0, i))
            if max_children is None or kids[p] < max_children:
                break
        parent[i] = p
        kids[p] += 1
    return parent


def topk_tree_parents(branching, quotas) -> np.ndarray:
    """Breadth-first draft tree in the "top-k" style.

    ``branching[d]`` is the most children a node at depth d may have and
    ``quotas[d]`` the number of nodes at depth d+1.  Parents at one depth take
    children in rank order: the rank-0 parent fills its full branching first,
    then rank 1, and so on.  Node 0 is the root; ids are breadth-first, so
    parent[i] < i.
    """
    parent = [-1]
    level = [0]
    for bmax, q in zip(branching, quotas):
        nxt = []
        need = q
        for p in level:
            take = min(bmax, need)
            for _ in range(take):
                parent.append(p)
                nxt.append(len(parent) - 1)
            need -= take
            if need == 0:
                break
        if need:
            raise ValueError("quota exceeds the branching of the level above")
        level = nxt
    return np.asarray(parent, dtype=np.int32)


def tree_draft_tokens(parent: np.ndarray, root_token: int, greedy_of, vocab: int, p_accept: float,
                      seed: int = BASE_SEED, stream: int = 0) -> np.ndarray:
    """Tokens of a draft tree, level by level.

    ``greedy_of(tokens_so_far, node)`` must return the target's greedy token at
    ``node`` given the tokens assigned so far (it is only called for nodes whose
    children are being filled).  At each node with children, with probability
    ``p_accept`` the greedy token goes to one seeded child slot; the other
    children get uniform tokens, all siblings distinct.
    """
    parent = np.asarray(parent, dtype=np.int64)
    n = len(parent)
    rng = _rng(_P_TREE, n, stream, 2, seed=seed)
    tok = np.full(n, -1, dtype=np.int64)
    tok[0] = root_token
    children = [[] for _ in range(n)]
    for i in range(1, n):
        children[parent[i]].append(i)
    for node in range(n):
        kids = children[node]
        if not kids:
            continue
        g = int(greedy_of(tok.copy(), node))
        slot = int(rng.integers(0, len(kids))) if rng.random() < p_accept else -1
        used = set()
        for j, c in enumerate(kids):
            if j == slot:
                t = g
            else:
                t = _other_token(rng, vocab, used | {g})
            used.add(t)
            tok[c] = t
    return tok.astype(np.int32)


def mask_from_layers(n_layers: int, layers) -> np.ndarray:
    m = np.zeros(n_layers, dtype=np.uint8)
    for l in layers:
        m[int(l)] = 1
    return m


def nested_skip_masks(n_layers: int, lo: int, hi: int, counts, seed: int = BASE_SEED, stream: int = 0):
    """Nested skip masks: a seeded permutation of layers [lo, hi]; the mask with
    count c skips its first c layers, so a smaller mask is a subset of a larger one."""
    perm = _rng(_P_MASK, n_layers, lo, hi, stream, seed=seed).permutation(np.arange(lo, hi + 1))
    return {int(c): mask_from_layers(n_layers, perm[:c]) for c in counts}


def random_skip_mask(n_layers: int, lo: int, hi: int, count: int, seed: int = BASE_SEED, stream: int = 0) -> np.ndarray:
    rng = _rng(_P_MASK, n_layers, lo, hi, stream, count + 1000, seed=seed)
    layers = rng.choice(np.arange(lo, hi + 1), size=count, replace=False)
    return mask_from_layers(n_layers, layers)


def abi_tensor_loader(shape, seed: int = BASE_SEED, random_gains: bool = False):
    """get_tensor(index) for the library's load order: fp32 arrays, or bf16
    bit patterns (uint16) for bf16 shapes."""
    names = {i: (layer, nm) for i, layer, nm in tensor_names(shape.n_layers)}

    def get(index):
        layer, nm = names[index]
        return weight_tensor(shape, nm, layer, seed=seed, random_gains=random_gains,
                             as_bf16_bits=shape.dtype == "bf16")
    return get
