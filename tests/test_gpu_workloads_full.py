"""GPU checks of the tree, batch and sweep workloads at their full sizes and in
the launch configurations the benchmark times.  The oracle cannot run these
sizes, so the checks are properties that hold at any size:

* the accept decision of a step equals the walk of the step's own greedy
  tokens down its draft tree (exact, no tolerance);
* a tree node sees exactly its root path, so the accepted path verified as a
  chain gives the same logits (bf16 tolerance) and, where the top-2 margins
  along it clear the gate, the same decision;
* a batched step gives each sequence the rows of its own single-sequence
  verify (bf16 tolerance; greedy tokens and decisions compared where the
  margins clear the gate);
* steps are bit-exact when repeated, also after other skip masks ran.

Workloads: 7B-shape, 2048-token context, 60-node top-k tree, 6 layers skipped;
13B-shape, 8 sequences with contexts 512-4096, chain k = 8, per-sequence masks;
33B-shape, 4096-token dense context, 32-node tree, three skip masks in a row.
"""
import gc

import numpy as np
import pytest

import synth
from tests.gpu_common import TOL, log

pytestmark = pytest.mark.gpu

TOL_BF16, GATE = TOL["bf16"]


def _load(shape, **kw):
    from tests.gpu_common import gpu_verifier
    log(f"loading {shape.name} with {kw}")
    return gpu_verifier(shape, **kw)


def _free(v):
    import torch
    v.close()
    del v.weights, v.workspace, v.kv_pool
    gc.collect()
    torch.cuda.empty_cache()


def _children(parent):
    kids = [[] for _ in range(len(parent))]
    for i in range(1, len(parent)):
        kids[parent[i]].append(i)
    return kids


def _greedy_walk(tokens, parent, greedy):
    """Nodes visited from the root following the child whose token is the
    current node's greedy token (siblings hold distinct tokens)."""
    kids = _children(parent)
    path = [0]
    while True:
        nxt = [c for c in kids[path[-1]] if tokens[c] == greedy[path[-1]]]
        if not nxt:
            return path
        path.append(nxt[0])


def _margins(lg):
    top2 = np.partition(lg, -2, axis=1)[:, -2:]
    return top2[:, 1] - top2[:, 0]


def _root_path(parent, node):
    path = [node]
    while parent[path[-1]] >= 0:
        path.append(int(parent[path[-1]]))
    return path[::-1]


def _tree_tokens(v, parent, root, mask, stream):
    """Draft tokens holding the target's greedy token (from chain dry runs
    along each root path) in one seeded child slot of every inner node."""
    def greedy_of(tok, node):
        chain = tok[_root_path(parent, node)]
        v.verify(0, chain, mask=mask)
        return int(v.greedy(len(chain))[-1])
    return synth.tree_draft_tokens(parent, root, greedy_of, v.shape.vocab, 1.0, stream=stream)


def _check_tree_step(v, tokens, parent, mask, what):
    """One dry-run tree verify: decision == greedy walk; the walked path as a
    chain matches; a greedy path through a greedy-filled tree ends at a leaf
    where the margins clear the gate.  Returns the step's logits."""
    n = len(parent)
    al, nt = v.verify(0, tokens, parent, mask=mask)
    lg, g = v.logits(n), v.greedy(n)
    np.testing.assert_array_equal(g, np.argmax(lg, axis=1))
    walk = _greedy_walk(tokens, parent, g)
    assert (al, nt) == (len(walk) - 1, int(g[walk[-1]])), what
    mg = _margins(lg)
    sure = float(mg[walk].min()) > GATE
    if sure:
        assert not _children(parent)[walk[-1]], f"{what}: greedy walk stopped at an inner node"
    ac, nc = v.verify(0, tokens[walk], mask=mask)
    err = float(np.max(np.abs(v.logits(len(walk)) - lg[walk])))
    log(f"{what}: accept {al} next {nt}, path {walk}, chain logits max-abs {err:.2e}, "
        f"min margin {float(mg[walk].min()):.3f}")
    assert err <= TOL_BF16
    if sure:
        assert (ac, nc) == (al, nt)
    return lg


def test_7b_tree_2048_ctx():
    shape = synth.LLAMA_7B
    ctx_n = 2048
    v = _load(shape, n_seqs=1, max_tokens=ctx_n + 64, max_nodes=64)
    mask = synth.random_skip_mask(shape.n_layers, 16, 31, 6, stream=3)
    toks = synth.context_tokens(shape.vocab, ctx_n + 1, stream=3)
    v.set_mask(0, mask)
    v.prefill(0, toks[:ctx_n])
    parent = synth.topk_tree_parents((4, 3, 2, 2, 1, 1), (4, 12, 20, 12, 8, 4))
    tokens = _tree_tokens(v, parent, int(toks[ctx_n]), None, stream=3)
    lg = _check_tree_step(v, tokens, parent, None, "7B tree")
    v.verify(0, tokens, parent)
    np.testing.assert_array_equal(v.logits(len(parent)), lg)
    assert v.length(0) == ctx_n
    _free(v)


def test_13b_batch_of_8_matches_single_verifies():
    shape = synth.LLAMA_13B
    B, k = 8, 8
    rng = np.random.default_rng(synth.BASE_SEED + 13)
    ctx_lens = [int(x) for x in rng.integers(512, 4097, size=B)]
    masks = [synth.random_skip_mask(shape.n_layers, 2, 39, int(rng.integers(0, 11)), stream=40 + i) for i in range(B)]
    v = _load(shape, n_seqs=B, max_tokens=4096 + k + 8, max_nodes=k + 1, max_batch=B)
    drafts, singles = [], []
    for i in range(B):
        toks = synth.context_tokens(shape.vocab, ctx_lens[i] + 1, stream=50 + i)
        v.set_mask(i, masks[i])
        v.prefill(i, toks[:-1])
        cur = [int(toks[-1])]
        for _ in range(k):
            v.verify(i, cur)
            cur.append(int(v.greedy(len(cur))[-1]))
        drafts.append(np.asarray(cur))
        al, nt = v.verify(i, drafts[-1])
        singles.append((al, nt, v.logits(k + 1), v.greedy(k + 1)))
    log(f"13B: contexts {ctx_lens}, single-sequence accepts {[s[0] for s in singles]}")
    al, nt = v.verify_batch(list(range(B)), drafts)
    lg, g = v.logits(B * (k + 1)), v.greedy(B * (k + 1))
    worst, rows_cmp, dec_cmp = 0.0, 0, 0
    for i in range(B):
        rows = slice(i * (k + 1), (i + 1) * (k + 1))
        s_al, s_nt, s_lg, s_g = singles[i]
        worst = max(worst, float(np.max(np.abs(lg[rows] - s_lg))))
        mg = _margins(s_lg)
        sure = mg > GATE
        np.testing.assert_array_equal(g[rows][sure], s_g[sure])
        rows_cmp += int(sure.sum())
        # exact: the batch decision is the scan of the batch's own greedy tokens
        n_acc = 0
        while n_acc < k and drafts[i][n_acc + 1] == g[rows][n_acc]:
            n_acc += 1
        assert (int(al[i]), int(nt[i])) == (n_acc, int(g[rows][n_acc]))
        if float(mg[: s_al + 1].min()) > GATE:
            assert (int(al[i]), int(nt[i])) == (s_al, s_nt)
            dec_cmp += 1
    log(f"13B batch of 8: accept {list(al)}, rows vs single verifies max-abs {worst:.2e}, "
        f"{rows_cmp}/{B * (k + 1)} greedy rows and {dec_cmp}/{B} decisions compared")
    assert worst <= TOL_BF16
    assert rows_cmp >= B * (k + 1) // 2
    for i in range(B):
        assert v.length(i) == ctx_lens[i]
    _free(v)


def test_33b_mask_sweep_4096_ctx():
    shape = synth.LLAMA_33B
    ctx_n = 4096
    v = _load(shape, n_seqs=1, max_tokens=ctx_n + 40, max_nodes=33)
    toks = synth.context_tokens(shape.vocab, ctx_n + 1, stream=5)
    v.prefill(0, toks[:ctx_n])
    parent = synth.topk_tree_parents((4, 3, 2, 1, 1), (4, 10, 10, 5, 3))
    rng = np.random.default_rng(synth.BASE_SEED + 33)
    masks = [synth.random_skip_mask(shape.n_layers, 2, 59, int(rng.integers(4, 17)), stream=100 + i)
             for i in range(3)]
    first = None
    for mi, mask in enumerate(masks):
        tokens = _tree_tokens(v, parent, int(toks[ctx_n]), mask, stream=5 + mi)
        lg = _check_tree_step(v, tokens, parent, mask, f"33B mask {mi} ({int(mask.sum())} skipped)")
        if first is None:
            first = (tokens, mask, lg)
    tokens, mask, lg = first
    v.verify(0, tokens, parent, mask=mask)
    np.testing.assert_array_equal(v.logits(len(parent)), lg)
    assert v.length(0) == ctx_n
    _free(v)
