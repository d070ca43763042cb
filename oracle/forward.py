"""The oracle's forward pass, greedy verification and KV commit.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Everything is plain
numpy in the oracle's float type (fp32 by default), with one contiguous K and
one contiguous V array per layer and sequence, and explicit loops over nodes
and layers.  No tiling, paging, fusion or reordering.

Readings of points the paper leaves open (each one is a choice of this
oracle; the GPU library follows the same readings):

* Layers are numbered from 0 and a skip mask is one byte per layer (1 = skip).
  The paper's formula indexes blocks from 1, but the skip sets it reports read
  naturally as 0-based module indices.
* Node 0 of a draft is the root: the last committed token, whose K/V are not
  cached yet.  Row i's logits predict the children of node i.  A tree node's
  position is n_kv + depth; a node attends to every cached context row and to
  itself and its ancestors among the draft nodes.
* accept_len counts accepted draft tokens (the paper's accept length counts
  accepted draft tokens); the bonus token is extra, so a step commits
  accept_len + 1 tokens.
* Greedy argmax breaks ties toward the lowest vocabulary index; among accepted
  nodes of equal depth the lowest node index wins.
* RMSNorm epsilon is 1e-6 (not stated in the paper), computed in the oracle's
  float type.
* Rotary embedding is LLaMA rotate-half: dimension pairs (j, j + hd/2) rotate by
  pos * base^(-2j/hd), base 10000.  Angles are formed in float64.
* A skipped layer neither reads nor writes KV.  Prefill runs under the
  sequence's mask; a verify may only activate layers whose cached K/V cover
  the whole committed context.
* Commit keeps the K/V of the root and of the accepted path, moved to the
  slots right after the context, and grows n_kv by accept_len + 1.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return (x / np.sqrt(ms + x.dtype.type(eps))) * g


def rope(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """Rotate-half rotary embedding of x [M][H][hd] at integer positions pos [M]."""
    hd = x.shape[-1]
    half = hd // 2
    inv_freq = base ** (-(2.0 * np.arange(half, dtype=np.float64)) / hd)
    ang = pos.astype(np.float64)[:, None] * inv_freq[None, :]
    cos = np.cos(ang).astype(x.dtype)[:, None, :]
    sin = np.sin(ang).astype(x.dtype)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (x.dtype.type(1) + np.exp(-x))


def tree_meta(parent):
    """depth[i] and the visible set vis(i) = {i} + ancestors of i, from a parent array."""
    parent = [int(p) for p in parent]
    n = len(parent)
    if n == 0 or parent[0] != -1:
        raise ValueError("parent[0] must be -1")
    depth = [0] * n
    vis = [None] * n
    vis[0] = {0}
    for i in range(1, n):
        p = parent[i]
        if not (0 <= p < i):
            raise ValueError(f"parent[{i}]={p} must be in [0, {i})")
        depth[i] = depth[p] + 1
        vis[i] = vis[p] | {i}
    return np.asarray(depth, dtype=np.int64), vis


class OracleModel:
    """Weights of the target, fetched lazily per layer from ``get_tensor(name, layer)``.

    Only the layers that some call actually runs are ever fetched, so a model
    can be checked on a few active layers without materialising the rest.
    """

    def __init__(self, shape, get_tensor, dtype=np.float32):
        self.shape = shape
        self.dtype = np.dtype(dtype)
        self._get = get_tensor
        self._layers = {}
        self._glob = {}

    def _t(self, name, layer=-1):
        return np.ascontiguousarray(self._get(name, layer), dtype=self.dtype)

    def glob(self, name):
        if name not in self._glob:
            self._glob[name] = self._t(name)
        return self._glob[name]

    def layer(self, l):
        if l not in self._layers:
            self._layers[l] = {nm: self._t(nm, l) for nm in
                               ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")}
        return self._layers[l]


class OracleSequence:
    """One sequence's KV state: contiguous K_l, V_l of shape [n][H][hd] per layer."""

    def __init__(self, model: OracleModel, mask=None):
        s = model.shape
        self.model = model
        self.mask = np.zeros(s.n_layers, dtype=np.uint8) if mask is None else np.asarray(mask, dtype=np.uint8).copy()
        self.n_kv = 0
        empty = np.zeros((0, s.n_heads, s.head_dim), dtype=model.dtype)
        self.K = [empty.copy() for _ in range(s.n_layers)]
        self.V = [empty.copy() for _ in range(s.n_layers)]


@dataclass
class VerifyResult:
    logits: np.ndarray      # [M][V]
    greedy: np.ndarray      # [M] argmax per node (lowest index on ties)
    margin: np.ndarray      # [M] top-1 minus top-2 logit
    accept_len: int
    next_token: int
    best: int               # deepest accepted node
    path: list              # node ids root -> best


def _forward(model: OracleModel, seq: OracleSequence, tokens, parent, mask, with_logits: bool):
    """Run the sparse verifier over the nodes; returns (logits or None, per-layer new K/V rows)."""
    s = model.shape
    dt = model.dtype
    H, hd = s.n_heads, s.head_dim
    tokens = np.asarray(tokens, dtype=np.int64)
    M = len(tokens)
    depth, vis = tree_meta(parent)
    n_kv = seq.n_kv
    pos = n_kv + depth
    scale = dt.type(1.0 / np.sqrt(hd))
    # node i sees every cached context row, itself and its ancestors
    visible = np.zeros((M, n_kv + M), dtype=bool)
    visible[:, :n_kv] = True
    for i in range(M):
        visible[i, [n_kv + j for j in vis[i]]] = True

    h = model.glob("embed")[tokens].astype(dt)                  # [M][d]
    new_kv = {}
    for l in range(s.n_layers):
        if mask[l]:
            continue                                           # block bypass: h_{l+1} = h_l
        if seq.K[l].shape[0] != n_kv:
            raise ValueError(f"layer {l} has {seq.K[l].shape[0]} cached rows but n_kv is {n_kv}")
        w = model.layer(l)
        x = rmsnorm(h, w["attn_norm"], s.rms_eps)
        q = (x @ w["wq"].T).reshape(M, H, hd)
        k = (x @ w["wk"].T).reshape(M, H, hd)
        v = (x @ w["wv"].T).reshape(M, H, hd)
        q = rope(q, pos, s.rope_base)
        k = rope(k, pos, s.rope_base)
        new_kv[l] = (k, v)
        # masked attention: scores against every cached row and every node,
        # with the keys node i may not see set to -inf before the softmax
        Kall = np.concatenate([seq.K[l], k], axis=0)             # [n_kv + M][H][hd]
        Vall = np.concatenate([seq.V[l], v], axis=0)
        sc = np.matmul(q.transpose(1, 0, 2), Kall.transpose(1, 2, 0)) * scale   # [H][M][n_kv + M]
        sc = np.where(visible[None, :, :], sc, -np.inf)
        p = np.exp(sc - sc.max(axis=-1, keepdims=True))
        p = p / p.sum(axis=-1, keepdims=True)
        o = np.matmul(p, Vall.transpose(1, 0, 2)).transpose(1, 0, 2)           # [M][H][hd]
        h = h + o.reshape(M, H * hd) @ w["wo"].T
        x = rmsnorm(h, w["mlp_norm"], s.rms_eps)
        a = silu(x @ w["w_gate"].T) * (x @ w["w_up"].T)
        h = h + a @ w["w_down"].T
    logits = None
    if with_logits:
        logits = rmsnorm(h, model.glob("final_norm"), s.rms_eps) @ model.glob("lm_head").T
    return logits, new_kv, depth


def accept_scan(tokens, parent, greedy):
    """Greedy acceptance over a draft tree.

    A node is accepted when its parent is accepted and its token equals the
    greedy token at its parent; the root is always accepted.  The result is the
    deepest accepted node (lowest index on ties), its depth (= accept_len) and
    the greedy token there (= the bonus token).
    """
    depth, _ = tree_meta(parent)
    M = len(tokens)
    acc = [False] * M
    acc[0] = True
    for i in range(1, M):
        p = int(parent[i])
        acc[i] = acc[p] and int(tokens[i]) == int(greedy[p])
    best = 0
    for i in range(M):
        if acc[i] and depth[i] > depth[best]:
            best = i
    path = []
    j = best
    while j != -1:
        path.append(j)
        j = int(parent[j]) if j != 0 else -1
    path.reverse()
    return int(depth[best]), int(greedy[best]), best, path


def _commit(seq: OracleSequence, new_kv, nodes):
    for l, (k, v) in new_kv.items():
        seq.K[l] = np.concatenate([seq.K[l], k[nodes]], axis=0)
        seq.V[l] = np.concatenate([seq.V[l], v[nodes]], axis=0)
    seq.n_kv += len(nodes)


def prefill(model: OracleModel, seq: OracleSequence, tokens):
    """Append a chain of context tokens to the sequence under its own mask."""
    tokens = np.asarray(tokens, dtype=np.int64)
    if len(tokens) == 0:
        return
    parent = np.arange(-1, len(tokens) - 1)
    _, new_kv, _ = _forward(model, seq, tokens, parent, seq.mask, with_logits=False)
    _commit(seq, new_kv, list(range(len(tokens))))


def verify(model: OracleModel, seq: OracleSequence, tokens, parent=None, mask=None, commit: bool = False) -> VerifyResult:
    """One verification step over a chain (parent None) or a tree of draft nodes."""
    tokens = np.asarray(tokens, dtype=np.int64)
    M = len(tokens)
    if parent is None:
        parent = np.arange(-1, M - 1)
    parent = np.asarray(parent, dtype=np.int64)
    mask = seq.mask if mask is None else np.asarray(mask, dtype=np.uint8)
    logits, new_kv, depth = _forward(model, seq, tokens, parent, mask, with_logits=True)
    greedy = np.argmax(logits, axis=-1)                         # numpy returns the first maximum
    srt = np.sort(logits, axis=-1)
    margin = srt[:, -1] - srt[:, -2]
    accept_len, next_token, best, path = accept_scan(tokens, parent, greedy)
    if commit:
        _commit(seq, new_kv, path)
    return VerifyResult(logits=logits, greedy=greedy.astype(np.int64), margin=margin, accept_len=accept_len,
                        next_token=next_token, best=best, path=path)
