"""GPU parity at 33B dimensions (d 6656, 52 heads x 128, FFN 17920, vocab
32000, bf16) on two layers: the widest projection blocks (ten-tile gate/up
blocks with 3 row tiles, six-tile Q/K/V blocks with 3-4 row tiles) against
the fp32 oracle, element by element, on the 33-node sweep tree and a 61-node
tree over a 256-token paged context."""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import OracleSequence, prefill
from tests.gpu_common import compare_step, gpu_verifier, log, oracle_model

pytestmark = pytest.mark.gpu

SHAPE = dataclasses.replace(synth.LLAMA_33B, name="llama-33b-dims-2L", n_layers=2)
CTX = 256


@pytest.fixture(scope="module")
def pair():
    log("building 2-layer 33B-dims bf16 verifier")
    v = gpu_verifier(SHAPE, n_seqs=1, max_tokens=CTX + 80, max_nodes=64)
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
