"""Pins of the CPU oracle against facts fixed outside it.

* Dense equivalence (Problem Formulation: the empty skip set is the dense
  verifier): with an all-zero mask the oracle's prefill + verify logits equal
  the logits of an independent LLaMA forward (Hugging Face Transformers) over
  context + drafts at the same positions (teacher forcing, i.e. the KV-cache
  identity).
* Skip identity (Domain-Aware Skip Controller, block bypass equation): mask
  {l} equals the independent forward of the model with block l deleted.
* Tree = per-path chains: each tree node's logits equal the independent
  forward over context + that node's root path.
* Acceptance (greedy verification, Appendix Evaluation Protocol, temperature
  0): brute-force enumeration of root-to-node paths on tiny trees, full
  acceptance of the target's own greedy continuation, and the closed form of
  the tiny workload (3 greedy then 2 non-greedy drafts accept exactly 3).
* Commit: after a committing step, the next step's logits equal the
  independent forward over context + accepted path + new drafts.
* Closed forms for RMSNorm and the rotary rotation, and for the top-2 margin
  that decides which parity cases are excused: with every block skipped and
  one-hot embeddings, each node's logits are one lm_head column scaled by the
  final norm, so the greedy token and the margin follow from that column.

The independent forward computes rotary angles in fp32, so agreement is
limited to about 1e-6; a dropped term, a wrong sign or a transposed operand
moves logits by orders of magnitude more.
"""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import OracleModel, OracleSequence, prefill, verify, accept_scan, rmsnorm, rope, tree_meta

from tests import llama_ref

SHAPE = synth.TINY
TOL = 1e-4


def _getter(random_gains=True, seed=7):
    cache = {}

    def get(name, layer):
        key = (name, layer)
        if key not in cache:
            cache[key] = synth.weight_tensor(SHAPE, name, layer, seed=seed, random_gains=random_gains)
        return cache[key]
    return get


@pytest.fixture(scope="module")
def get():
    return _getter()


@pytest.fixture(scope="module")
def hf_full(get):
    return llama_ref.build(SHAPE, get)


@pytest.fixture(scope="module")
def model64(get):
    return OracleModel(SHAPE, get, dtype=np.float64)


def _ctx(n, stream=0):
    return synth.context_tokens(SHAPE.vocab, n, seed=11, stream=stream)


def test_dense_chain_matches_independent_forward(model64, hf_full):
    ctx = _ctx(24)
    root = int(_ctx(25)[-1])
    drafts = synth.context_tokens(SHAPE.vocab, 5, seed=12)
    seq = OracleSequence(model64)
    prefill(model64, seq, ctx)
    res = verify(model64, seq, np.concatenate([[root], drafts]))
    ref = llama_ref.logits(hf_full, np.concatenate([ctx, [root], drafts]))[len(ctx):]
    assert res.logits.shape == ref.shape
    assert np.max(np.abs(res.logits - ref)) < TOL
    # logits are O(0.3) here; the comparison is not vacuous
    assert np.std(ref) > 0.05


@pytest.mark.parametrize("skip", [[2], [0], [1, 3]])
def test_skip_equals_deleted_block(model64, get, skip):
    hf = llama_ref.build(SHAPE, get, drop_layers=skip)
    mask = synth.mask_from_layers(SHAPE.n_layers, skip)
    ctx = _ctx(20, stream=1)
    tok = synth.context_tokens(SHAPE.vocab, 6, seed=13)
    seq = OracleSequence(model64, mask)
    prefill(model64, seq, ctx)
    res = verify(model64, seq, tok)
    ref = llama_ref.logits(hf, np.concatenate([ctx, tok]))[len(ctx):]
    assert np.max(np.abs(res.logits - ref)) < TOL
    # and the skipped layers got no KV
    for l in skip:
        assert seq.K[l].shape[0] == 0


def test_skipped_block_is_exact_identity(get):
    # Oracle-internal: mask {l} on a model equals the dense forward of a model
    # whose tensors for layers >= l are shifted by one (layer l removed).
    m = OracleModel(SHAPE, get)
    l = 1
    shifted = OracleModel(dataclasses.replace(SHAPE, n_layers=SHAPE.n_layers - 1),
                          lambda nm, ly: get(nm, ly if ly < l else ly + 1) if ly >= 0 else get(nm, ly))
    ctx = _ctx(16, stream=2)
    tok = synth.context_tokens(SHAPE.vocab, 4, seed=14)
    a = OracleSequence(m, synth.mask_from_layers(SHAPE.n_layers, [l]))
    prefill(m, a, ctx)
    b = OracleSequence(shifted)
    prefill(shifted, b, ctx)
    ra, rb = verify(m, a, tok), verify(shifted, b, tok)
    np.testing.assert_array_equal(ra.logits, rb.logits)


def test_tree_nodes_match_path_chains(model64, hf_full):
    ctx = _ctx(18, stream=3)
    parent = synth.random_tree(8, seed=15)
    tok = synth.context_tokens(SHAPE.vocab, 8, seed=16)
    seq = OracleSequence(model64)
    prefill(model64, seq, ctx)
    res = verify(model64, seq, tok, parent)
    depth, vis = tree_meta(parent)
    assert depth.max() >= 2
    for i in range(len(tok)):
        path = sorted(vis[i])
        ref = llama_ref.logits(hf_full, np.concatenate([ctx, tok[path]]))[-1]
        assert np.max(np.abs(res.logits[i] - ref)) < TOL, i


def _greedy_continuation(hf, prefix, k):
    seq = list(prefix)
    out = []
    for _ in range(k + 1):
        g = int(np.argmax(llama_ref.logits(hf, seq)[-1]))
        out.append(g)
        seq.append(g)
    return np.asarray(out)


def test_self_consistent_drafts_fully_accepted(model64, hf_full):
    ctx = _ctx(22, stream=4)
    root = int(_ctx(23, stream=4)[-1])
    g = _greedy_continuation(hf_full, np.concatenate([ctx, [root]]), 5)
    seq = OracleSequence(model64)
    prefill(model64, seq, ctx)
    res = verify(model64, seq, np.concatenate([[root], g[:5]]))
    assert res.accept_len == 5
    assert res.next_token == g[5]


def _bruteforce_accept(hf, ctx, tok, parent):
    """Enumerate root->node paths; a path is accepted when every token equals
    the independent forward's argmax at its predecessor on that path."""
    depth, vis = tree_meta(parent)
    best, best_depth = 0, 0
    for i in range(len(tok)):
        path = sorted(vis[i])
        lg = llama_ref.logits(hf, np.concatenate([ctx, tok[path]]))[len(ctx):]
        ok = all(int(np.argmax(lg[j])) == int(tok[path[j + 1]]) for j in range(len(path) - 1))
        if ok and depth[i] > best_depth:
            best, best_depth = i, int(depth[i])
    path = sorted(vis[best])
    nxt = int(np.argmax(llama_ref.logits(hf, np.concatenate([ctx, tok[path]]))[-1]))
    return best_depth, nxt


@pytest.mark.parametrize("stream", [0, 1, 2, 3])
def test_accept_matches_bruteforce(model64, hf_full, stream):
    ctx = _ctx(14, stream=10 + stream)
    parent = synth.random_tree(8, seed=17, stream=stream, max_children=3)

    def greedy_of(tokens, node):
        _, vis = tree_meta(parent)
        path = sorted(vis[node])
        return int(np.argmax(llama_ref.logits(hf_full, np.concatenate([ctx, tokens[path]]))[-1]))

    root = int(_ctx(15, stream=10 + stream)[-1])
    tok = synth.tree_draft_tokens(parent, root, greedy_of, SHAPE.vocab, p_accept=0.8, seed=18, stream=stream)
    seq = OracleSequence(model64)
    prefill(model64, seq, ctx)
    res = verify(model64, seq, tok, parent)
    assert np.min(res.margin) > 1e-6
    bl, bn = _bruteforce_accept(hf_full, ctx, tok, parent)
    assert (res.accept_len, res.next_token) == (bl, bn)


def test_tiny_workload_closed_form(get):
    """The tiny workload: 128 context tokens in KV, a root, a chain of k=5
    whose first 3 drafts are the masked target's greedy tokens and last 2 are
    other tokens, skip mask {2}: exactly 3 drafts are accepted."""
    m = OracleModel(SHAPE, get)
    mask = synth.mask_from_layers(SHAPE.n_layers, [2])
    toks = synth.context_tokens(SHAPE.vocab, 129)
    ctx, root = toks[:128], int(toks[128])
    seq = OracleSequence(m, mask)
    prefill(m, seq, ctx)
    # greedy continuation of the masked target, one token at a time
    g = []
    cur = [root]
    for _ in range(5):
        r = verify(m, seq, np.asarray(cur))
        g.append(int(r.greedy[-1]))
        cur.append(g[-1])
    drafts = synth.chain_draft(np.asarray(g), SHAPE.vocab, n_greedy=3)
    res = verify(m, seq, np.concatenate([[root], drafts]))
    assert res.accept_len == 3
    assert res.next_token == g[3]
    assert seq.n_kv == 128


def test_commit_then_verify_matches_long_forward(model64, hf_full):
    ctx = _ctx(12, stream=5)
    parent = np.array([-1, 0, 0, 1, 2, 2, 4], dtype=np.int32)

    def greedy_of(tokens, node):
        _, vis = tree_meta(parent)
        path = sorted(vis[node])
        return int(np.argmax(llama_ref.logits(hf_full, np.concatenate([ctx, tokens[path]]))[-1]))

    root = int(_ctx(13, stream=5)[-1])
    # force the accepted path through node 2 (not the first child) so commit must compact
    tok = np.full(7, -1, dtype=np.int64)
    tok[0] = root
    g0 = greedy_of(tok, 0)
    tok[1] = (g0 + 1) % SHAPE.vocab
    tok[2] = g0
    tok[3] = 5
    g2 = greedy_of(tok, 2)
    tok[4] = (g2 + 7) % SHAPE.vocab
    tok[5] = g2
    tok[6] = 9
    seq = OracleSequence(model64)
    prefill(model64, seq, ctx)
    r1 = verify(model64, seq, tok, parent, commit=True)
    assert r1.path == [0, 2, 5] and r1.accept_len == 2
    assert seq.n_kv == len(ctx) + 3
    nxt = synth.context_tokens(SHAPE.vocab, 3, seed=19)
    r2 = verify(model64, seq, np.concatenate([[r1.next_token], nxt]))
    ref = llama_ref.logits(hf_full, np.concatenate([ctx, tok[[0, 2, 5]], [r1.next_token], nxt]))[-4:]
    assert np.max(np.abs(r2.logits - ref)) < TOL


def test_verify_rejects_layers_without_kv(get):
    m = OracleModel(SHAPE, get)
    seq = OracleSequence(m, synth.mask_from_layers(SHAPE.n_layers, [1]))
    prefill(m, seq, _ctx(8))
    with pytest.raises(ValueError):
        verify(m, seq, np.array([1, 2]), mask=np.zeros(SHAPE.n_layers, dtype=np.uint8))


def test_fp32_oracle_close_to_fp64(get, model64):
    m32 = OracleModel(SHAPE, get, dtype=np.float32)
    ctx = _ctx(30, stream=6)
    tok = synth.context_tokens(SHAPE.vocab, 6, seed=20)
    s32, s64 = OracleSequence(m32), OracleSequence(model64)
    prefill(m32, s32, ctx)
    prefill(model64, s64, ctx)
    a, b = verify(m32, s32, tok), verify(model64, s64, tok)
    assert np.max(np.abs(a.logits - b.logits)) < 2e-5


def test_accept_scan_ties_and_duplicate_siblings():
    #        0
    #      /   \
    #     1     2      tokens 1 and 2 both equal greedy[0] (duplicate siblings)
    #     |     |
    #     3     4      3 matches greedy[1], 4 matches greedy[2]: equal depth, lowest index wins
    parent = [-1, 0, 0, 1, 2]
    greedy = [7, 8, 9, 10, 11]
    tokens = [0, 7, 7, 8, 9]
    al, nt, best, path = accept_scan(tokens, parent, greedy)
    assert (al, nt, best, path) == (2, 10, 3, [0, 1, 3])
    # nothing accepted
    al, nt, best, path = accept_scan([0, 5, 6], [-1, 0, 1], [1, 2, 3])
    assert (al, nt, best, path) == (0, 1, 0, [0])
    # a matching child under a rejected parent stays rejected
    al, nt, best, _ = accept_scan([0, 5, 2], [-1, 0, 1], [1, 2, 3])
    assert (al, nt, best) == (0, 1, 0)


def test_argmax_ties_take_lowest_index():
    # verify's greedy is numpy argmax, which returns the first maximum
    lg = np.array([[0.0, 3.0, 3.0, 1.0]])
    assert int(np.argmax(lg, axis=-1)[0]) == 1


def test_rmsnorm_closed_form():
    x = np.full((1, 8), 3.0)
    g = np.arange(1, 9, dtype=np.float64)
    y = rmsnorm(x, g, 1e-6)
    np.testing.assert_allclose(y[0], g * 3.0 / np.sqrt(9.0 + 1e-6), rtol=1e-14)


def test_rope_is_pairwise_rotation():
    rng = np.random.default_rng(0)
    hd, H = 16, 2
    x = rng.standard_normal((3, H, hd))
    pos = np.array([0, 5, 1000])
    y = rope(x, pos, 10000.0)
    for m in range(3):
        for j in range(hd // 2):
            th = pos[m] * 10000.0 ** (-2 * j / hd)
            R = np.array([[np.cos(th), -np.sin(th)], [np.sin(th), np.cos(th)]])
            for h in range(H):
                v = R @ np.array([x[m, h, j], x[m, h, j + hd // 2]])
                np.testing.assert_allclose([y[m, h, j], y[m, h, j + hd // 2]], v, rtol=1e-12, atol=1e-12)
    # position 0 is the identity, and rotation keeps the norm
    np.testing.assert_allclose(y[0], x[0])
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1))


def test_tree_meta_validation():
    d, vis = tree_meta([-1, 0, 0, 2])
    assert list(d) == [0, 1, 1, 2] and vis[3] == {0, 2, 3}
    for bad in ([0, 0], [-1, 1], [-1, 0, 3], []):
        with pytest.raises(ValueError):
            tree_meta(bad)


def test_margin_closed_form():
    """margin = largest minus second-largest logit of each row (0 on a tie,
    where the greedy token is the lowest tied index).  With every block
    skipped, node i's embedding c * e_i makes its logits s * W_lm[:, i] with
    s = sqrt(d) / sqrt(1 + eps * d / c^2) (final RMSNorm with unit gain), so
    the margin is s times the gap between the column's two largest values."""
    shape = dataclasses.replace(SHAPE, n_layers=1)
    d, V, c = shape.d_model, shape.vocab, 0.37
    rng = np.random.default_rng(3)
    lm = rng.uniform(-1.0, 0.9, size=(V, d))
    # column 0: a clear top-1 (index 17) over a runner-up (index 5)
    lm[17, 0], lm[5, 0] = 3.0, 2.5
    # column 1: a tie between indices 300 and 9 for the largest value
    lm[300, 1], lm[9, 1] = 2.0, 2.0
    # column 2: the largest value at the last index, every other value far below
    lm[:, 2] = rng.uniform(-2.0, -0.5, size=V)
    lm[V - 1, 2], lm[40, 2] = 1.25, -0.25
    emb = np.zeros((V, d))
    for i in range(3):
        emb[i, i] = c
    tensors = {"embed": emb, "lm_head": lm, "final_norm": np.ones(d)}
    m = OracleModel(shape, lambda name, layer: tensors[name], dtype=np.float64)
    seq = OracleSequence(m, np.ones(1, np.uint8))
    res = verify(m, seq, np.array([0, 1, 2]), parent=np.array([-1, 0, 0]))
    s = np.sqrt(d) / np.sqrt(1.0 + shape.rms_eps * d / c ** 2)
    np.testing.assert_allclose(res.margin, [s * 0.5, 0.0, s * 1.5], rtol=1e-12, atol=1e-12)
    assert list(res.greedy) == [17, 9, V - 1]
