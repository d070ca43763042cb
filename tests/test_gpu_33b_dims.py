"""GPU parity at 33B dimensions (d 6656, 52 heads x 128, FFN 17920, vocab
32000, bf16) on two layers: the widest projection blocks (ten-tile gate/up
blocks with 3 row tiles, six-tile Q/K/V blocks with 3-4 row tiles) against
the fp32 oracle, element by element, on the 33-node sweep tree and a 61-node
tree over a 256-token paged context (one attention workgroup per head), and
the 33-node tree over a 1024-token context, where each head's pages are split
among several workgroups and three row tiles of partial states are merged
across them (the path of the 4096-token sweep workload)."""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import OracleSequence, prefill
from tests.gpu_common import (assert_merged_split, compare_step, gpu_verifier, log, oracle_model,
                               oracle_tree_tokens)

pytestmark = pytest.mark.gpu

SHAPE = dataclasses.replace(synth.LLAMA_33B, name="llama-33b-dims-2L", n_layers=2)
CTX = 256
LONG_CTX = 1024


@pytest.fixture(scope="module")
def pair():
    log("building 2-layer 33B-dims bf16 verifier")
    v = gpu_verifier(SHAPE, n_seqs=1, max_tokens=LONG_CTX + 80, max_nodes=64)
    m = oracle_model(SHAPE)
    yield v, m
    v.close()


@pytest.mark.parametrize("skip,tree", [([], "sweep33"), ([0], "sweep33"), ([], "top61")])
def test_wide_blocks(pair, skip, tree):
    v, m = pair
    mask = synth.mask_from_layers(SHAPE.n_layers, skip)
    toks = synth.context_tokens(SHAPE.vocab, CTX + 1, stream=31 + len(skip))
    v.truncate(0, 0)
    v.set_mask(0, mask)
    v.prefill(0, toks[:CTX])
    o = OracleSequence(m, mask)
    prefill(m, o, toks[:CTX])
    if tree == "sweep33":
        parent = synth.topk_tree_parents((4, 3, 2, 1, 1), (4, 10, 10, 5, 3))
    else:
        parent = synth.topk_tree_parents((4, 3, 2, 2, 1, 1), (4, 12, 20, 12, 8, 4))
    n = len(parent)
    tok = np.concatenate([[toks[CTX]], synth.context_tokens(SHAPE.vocab, n - 1, stream=40 + n)])
    res, (al, nt), err, compared = compare_step(SHAPE, v, 0, m, o, tok, parent)
    log(f"33B dims, skip {skip}, {n}-node tree: logits err {err:.3e}, accept {al}/{res.accept_len}, "
        f"next {nt}/{res.next_token}, decision compared: {compared}")


def test_tree33_ctx1024_cross_workgroup_merge(pair):
    v, m = pair
    mask = synth.mask_from_layers(SHAPE.n_layers, [])
    toks = synth.context_tokens(SHAPE.vocab, LONG_CTX + 1, stream=35)
    v.truncate(0, 0)
    v.set_mask(0, mask)
    v.prefill(0, toks[:LONG_CTX])
    o = OracleSequence(m, mask)
    prefill(m, o, toks[:LONG_CTX])
    parent = synth.topk_tree_parents((4, 3, 2, 1, 1), (4, 10, 10, 5, 3))
    tok = oracle_tree_tokens(m, o, parent, int(toks[LONG_CTX]), SHAPE.vocab, 0.6, stream=35)
    res, (al, nt), err, compared = compare_step(SHAPE, v, 0, m, o, tok, parent)
    assert_merged_split(v, [33])
    log(f"33B dims, 33-node tree at 1024 tokens: logits err {err:.3e}, accept {al}/{res.accept_len}, "
        f"next {nt}/{res.next_token}, decision compared: {compared}")
