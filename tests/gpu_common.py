"""Shared helpers of the GPU tests: building a verifier and its oracle twin on
the same seeded weights, and the comparison rules.

Comparison rules (tolerances follow the arithmetic of each path):
* fp32 shapes (GPU all fp32, oracle fp32): logits max-abs <= 1e-4; greedy
  decisions must match wherever the oracle's top-2 margin exceeds 1e-3.
* bf16 shapes (GPU bf16 weights/KV/GEMM inputs with fp32 accumulation,
  residual and softmax; oracle fp32 on the same bf16-exact weights): logits
  max-abs <= 5e-2; accept_len and next_token must match wherever the smallest
  oracle margin over the accepted path and the bonus node exceeds 0.05.
"""
from __future__ import annotations

import numpy as np

import synth
from oracle import OracleModel, OracleSequence, prefill, verify

TOL = {"f32": (1e-4, 1e-3), "bf16": (5e-2, 5e-2)}


def log(msg):
    print(msg, flush=True)


def oracle_model(shape, random_gains=False, seed=synth.BASE_SEED):
    cache = {}

    def get(name, layer):
        key = (name, layer)
        if key not in cache:
            cache[key] = synth.weight_tensor(shape, name, layer, seed=seed, random_gains=random_gains)
        return cache[key]
    return OracleModel(shape, get)


def gpu_verifier(shape, random_gains=False, seed=synth.BASE_SEED, **kw):
    from paper_2609_26100_amd.verifier import Verifier
    v = Verifier(shape, **kw)
    v.load(synth.abi_tensor_loader(shape, seed=seed, random_gains=random_gains))
    return v


def check_decision(res, gpu_accept, gpu_next, margin_gate):
    """True if compared, False if excused by a small oracle margin."""
    nodes = list(res.path)
    if min(float(res.margin[i]) for i in nodes) <= margin_gate:
        return False
    assert (gpu_accept, gpu_next) == (res.accept_len, res.next_token)
    return True


def compare_step(shape, v, seq, m, oseq, tokens, parent=None, mask=None, commit=False):
    """Runs one verify on both sides and checks logits, greedy tokens and the decision."""
    tol, gate = TOL[shape.dtype]
    al, nt = v.verify(seq, tokens, parent, mask, commit)
    res = verify(m, oseq, tokens, parent, mask, commit)
    lg = v.logits(len(tokens))
    err = float(np.max(np.abs(lg - res.logits)))
    assert err <= tol, f"logits max-abs {err} > {tol}"
    g = v.greedy(len(tokens))
    sure = res.margin > gate
    np.testing.assert_array_equal(g[sure], res.greedy[sure])
    compared = check_decision(res, al, nt, gate)
    return res, (al, nt), err, compared


def prefill_chunked(m, oseq, tokens, chunk=512):
    """The oracle's prefill in pieces of `chunk` tokens (the same chain, bounded score arrays)."""
    tokens = np.asarray(tokens)
    for i in range(0, len(tokens), chunk):
        prefill(m, oseq, tokens[i:i + chunk])


def oracle_tree_tokens(m, oseq, parent, root, vocab, p_accept, stream, mask=None):
    """Draft-tree tokens whose accepted branches follow the oracle's greedy tokens (synth.tree_draft_tokens
    with the oracle as the target)."""
    parent = np.asarray(parent)

    def greedy_of(tok, node):
        path = [node]
        while parent[path[-1]] >= 0:
            path.append(int(parent[path[-1]]))
        return int(verify(m, oseq, tok[path[::-1]], None, mask).greedy[-1])
    return synth.tree_draft_tokens(parent, root, greedy_of, vocab, p_accept, stream=stream)


def assert_merged_split(v, rows, min_groups=2):
    """The last step's last attention launch divided every listed item's context pages among at least
    min_groups workgroups per head (the cross-workgroup merge path); rows = expected rows per item."""
    split = v.attn_split()
    log(f"attention split (workgroups per head, rows) per item: {split}")
    assert [r for _, r in split] == list(rows), split
    assert all(g >= min_groups for g, _ in split), split
    return split
