"""GPU parity at 7B dimensions (d 4096, 32 heads x 128, FFN 11008, vocab
32000, bf16): every kernel at its full shape and launch configuration,
compared with the fp32 oracle on a few active layers, a 1024-token paged
context and chain drafts of k=5 with per-position accept probability 0.6,
and the 60-node draft tree at a 300-token context (one attention workgroup
per head) and at the 1024-token context (each head's pages split among
several workgroups whose four row tiles of partial states are merged across
workgroups, the path of the 2048-token tree workload)."""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import OracleSequence, prefill, verify
from tests.gpu_common import (assert_merged_split, compare_step, gpu_verifier, log, oracle_model,
                               oracle_tree_tokens)

pytestmark = pytest.mark.gpu

# The 7B block shapes with 4 layers: the skip masks below leave 1-3 of them active.
SHAPE = dataclasses.replace(synth.LLAMA_7B, name="llama-7b-dims-4L", n_layers=4)
CTX = 1024


@pytest.fixture(scope="module")
def pair():
    log("building 4-layer 7B-dims bf16 verifier")
    v = gpu_verifier(SHAPE, n_seqs=2, max_tokens=CTX + 80, max_nodes=64)
    m = oracle_model(SHAPE)
    yield v, m
    v.close()


@pytest.mark.parametrize("skip", [[1, 2, 3], [0, 2], [1]])
def test_chain_k5(pair, skip):
    v, m = pair
    mask = synth.mask_from_layers(SHAPE.n_layers, skip)
    toks = synth.context_tokens(SHAPE.vocab, CTX + 8, stream=len(skip))
    ctx = toks[:CTX]
    v.truncate(0, 0)
    v.set_mask(0, mask)
    v.prefill(0, ctx)
    o = OracleSequence(m, mask)
    prefill(m, o, ctx)
    compared = 0
    # several roots, so that some cases clear the 0.05 margin gate
    for r in range(4):
        root = int(toks[CTX + r])
        g, cur = [], [root]
        for _ in range(5):
            g.append(int(verify(m, o, np.asarray(cur)).greedy[-1]))
            cur.append(g[-1])
        for s in range(3):
            drafts = synth.chain_draft(np.asarray(g), SHAPE.vocab, p_accept=0.6, stream=4 * r + s)
            res, (al, nt), err, c = compare_step(SHAPE, v, 0, m, o, np.concatenate([[root], drafts]))
            compared += c
            log(f"skip {skip} root {r} draft {s}: accept {al}/{res.accept_len} next {nt}/{res.next_token} "
                f"err {err:.3e} path-margin {float(res.margin[res.path].min()):.3f}")
    assert compared >= 1


def test_tree_61_nodes(pair):
    v, m = pair
    mask = synth.mask_from_layers(SHAPE.n_layers, [0, 3])
    toks = synth.context_tokens(SHAPE.vocab, 301, stream=9)
    v.truncate(1, 0)
    v.set_mask(1, mask)
    v.prefill(1, toks[:300])
    o = OracleSequence(m, mask)
    prefill(m, o, toks[:300])
    parent = synth.topk_tree_parents((4, 3, 2, 2, 1, 1), (4, 12, 20, 12, 8, 4))
    tok = np.concatenate([[toks[300]], synth.context_tokens(SHAPE.vocab, 60, stream=10)])
    res, (al, nt), err, _ = compare_step(SHAPE, v, 1, m, o, tok, parent)
    log(f"tree 61: err {err:.3e}")


def test_tree_61_nodes_ctx1024_cross_workgroup_merge(pair):
    v, m = pair
    mask = synth.mask_from_layers(SHAPE.n_layers, [0, 3])
    toks = synth.context_tokens(SHAPE.vocab, CTX + 1, stream=19)
    v.truncate(1, 0)
    v.set_mask(1, mask)
    v.prefill(1, toks[:CTX])
    o = OracleSequence(m, mask)
    prefill(m, o, toks[:CTX])
    parent = synth.topk_tree_parents((4, 3, 2, 2, 1, 1), (4, 12, 20, 12, 8, 4))
    tok = oracle_tree_tokens(m, o, parent, int(toks[CTX]), SHAPE.vocab, 0.6, stream=19)
    res, (al, nt), err, compared = compare_step(SHAPE, v, 1, m, o, tok, parent)
    assert_merged_split(v, [61])
    log(f"tree 61 at 1024 tokens: accept {al}/{res.accept_len} next {nt}/{res.next_token} err {err:.3e} "
        f"decision compared: {compared}")
