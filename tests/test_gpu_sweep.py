"""GPU parity of tss_verify_sweep: one draft tree of one sequence verified
under many skip masks, the masks packed as segments of shared steps.

Each mask's decision and greedy tokens must equal the oracle's verify of the
tree under that mask alone (decisions and greedy tokens compared where the
oracle's top-2 margins clear the gate); the last step's logits rows are
compared element by element.  Steps hold several segments (one context, each
segment with its own draft slots after it), attention items span segments,
and the row and KV-slot limits split the masks into several steps.
"""
import dataclasses
import itertools

import numpy as np
import pytest

import synth
from oracle import OracleSequence, prefill, verify
from tests.gpu_common import TOL, gpu_verifier, log, oracle_model

pytestmark = pytest.mark.gpu

TINY = synth.TINY


def _all_masks(n_layers):
    return np.array(list(itertools.product([0, 1], repeat=n_layers)), dtype=np.uint8)


def _compare_sweep(shape, v, m, o, tokens, parent, masks, per_step):
    """Sweep on the GPU, one oracle verify per mask; returns the number of
    decisions compared."""
    tol, gate = TOL[shape.dtype]
    n = len(tokens)
    al, nt, g = v.verify_sweep(0, tokens, masks, parent, want_greedy=True, reuse_prefix=False)
    last = len(masks) - (len(masks) - 1) % per_step - 1  # first mask of the last step (caller order)
    lg = v.logits((len(masks) - last) * n)
    compared = rows = 0
    for k, mk in enumerate(masks):
        res = verify(m, o, np.asarray(tokens), parent, mk)
        sure = res.margin > gate
        np.testing.assert_array_equal(g[k][sure], res.greedy[sure], err_msg=f"mask {k}")
        rows += int(sure.sum())
        path = list(res.path)
        if min(float(res.margin[i]) for i in path) > gate:
            assert (int(al[k]), int(nt[k])) == (res.accept_len, res.next_token), f"mask {k}"
            compared += 1
        if k >= last:
            i = k - last
            err = float(np.max(np.abs(lg[i * n:(i + 1) * n] - res.logits)))
            assert err <= tol, f"mask {k}: logits max-abs {err} > {tol}"
    log(f"sweep of {len(masks)} masks: {compared} decisions and {rows}/{len(masks) * n} greedy tokens compared")
    return compared


@pytest.fixture(scope="module")
def tiny():
    log("building tiny fp32 sweep verifier (rows 64: up to 9 segments of 7 nodes)")
    v = gpu_verifier(TINY, random_gains=True, n_seqs=2, max_tokens=300, max_nodes=8, max_batch=8)
    m = oracle_model(TINY, random_gains=True)
    ctx = synth.context_tokens(TINY.vocab, 150, stream=2000)
    v.prefill(0, ctx)
    o = OracleSequence(m, np.zeros(TINY.n_layers, np.uint8))
    prefill(m, o, ctx)
    yield v, m, o
    v.close()


def test_tiny_sweep_all_masks_vs_oracle(tiny):
    v, m, o = tiny
    masks = _all_masks(TINY.n_layers)[[0, 1, 2, 4, 8, 3, 5, 6, 9, 10, 12, 15]]  # dense first, all skipped last
    tokens = synth.context_tokens(TINY.vocab, 7, stream=2001)
    parent = synth.random_tree(7, stream=2002, max_children=3)
    comp = _compare_sweep(TINY, v, m, o, tokens, parent, masks, per_step=9)
    assert comp >= 8
    assert v.length(0) == 150


def test_tiny_sweep_chain_and_single_node(tiny):
    v, m, o = tiny
    masks = _all_masks(TINY.n_layers)
    chain = synth.context_tokens(TINY.vocab, 5, stream=2003)
    _compare_sweep(TINY, v, m, o, chain, None, masks, per_step=12)
    one = synth.context_tokens(TINY.vocab, 1, stream=2004)
    _compare_sweep(TINY, v, m, o, one, None, masks[:5], per_step=32)


def test_tiny_sweep_limited_by_free_kv_slots():
    """A sequence with 20 free slots takes 2 segments of 8 nodes per step."""
    v = gpu_verifier(TINY, random_gains=True, n_seqs=1, max_tokens=100, max_nodes=8, max_batch=8)
    m = oracle_model(TINY, random_gains=True)
    ctx = synth.context_tokens(TINY.vocab, 80, stream=2010)
    v.prefill(0, ctx)
    o = OracleSequence(m, np.zeros(TINY.n_layers, np.uint8))
    prefill(m, o, ctx)
    masks = _all_masks(TINY.n_layers)[::3]
    tokens = synth.context_tokens(TINY.vocab, 8, stream=2011)
    parent = synth.random_tree(8, stream=2012)
    _compare_sweep(TINY, v, m, o, tokens, parent, masks, per_step=2)
    assert v.length(0) == 80
    v.close()


def test_tiny_sweep_matches_single_verifies_and_repeats(tiny):
    v, m, o = tiny
    masks = _all_masks(TINY.n_layers)[1:12]
    tokens = synth.context_tokens(TINY.vocab, 6, stream=2020)
    parent = synth.random_tree(6, stream=2021)
    al, nt, g = v.verify_sweep(0, tokens, masks, parent, want_greedy=True)
    again = v.verify_sweep(0, tokens, masks, parent, want_greedy=True)
    for a, b in zip((al, nt, g), again):
        np.testing.assert_array_equal(a, b)
    for k, mk in enumerate(masks):
        a1, n1 = v.verify(0, tokens, parent, mask=mk)
        lg = v.logits(6)
        top2 = np.sort(lg, axis=1)[:, -2:]
        sure = top2[:, 1] - top2[:, 0] > 1e-3
        np.testing.assert_array_equal(v.greedy(6)[sure], g[k][sure])
        if sure.all():
            assert (a1, n1) == (int(al[k]), int(nt[k]))


def test_sweep_errors_leave_state_unchanged(tiny):
    from paper_2609_26100_amd import tss as abi
    v, m, o = tiny
    L = TINY.n_layers
    tok = synth.context_tokens(TINY.vocab, 4, stream=2030)
    # sequence 1 prefilled with layer 2 skipped: a mask that runs layer 2 lacks its K/V
    v.set_mask(1, synth.mask_from_layers(L, [2]))
    v.prefill(1, synth.context_tokens(TINY.vocab, 30, stream=2031))
    bad = [
        ((1, tok, np.zeros((2, L), np.uint8)), abi.TSS_ESTATE),
        ((0, tok, np.zeros((0, L), np.uint8)), abi.TSS_EINVAL),                  # no masks
        ((0, tok, np.full((1, L), 2, np.uint8)), abi.TSS_EINVAL),                # mask byte not 0/1
        ((0, np.array([1, TINY.vocab]), np.zeros((1, L), np.uint8)), abi.TSS_EINVAL),  # token outside the vocabulary
        ((0, np.arange(9), np.zeros((1, L), np.uint8)), abi.TSS_EINVAL),         # more nodes than max_nodes
        ((5, tok, np.zeros((1, L), np.uint8)), abi.TSS_EINVAL),                  # unknown sequence
    ]
    for args, status in bad:
        with pytest.raises(abi.TSSError) as e:
            v.verify_sweep(*args)
        assert e.value.status == status, args
    with pytest.raises(abi.TSSError) as e:
        v.verify_sweep(0, tok, np.zeros((1, L), np.uint8), parent=np.array([-1, 0, 3, 1]))
    assert e.value.status == abi.TSS_EINVAL
    assert (v.length(0), v.length(1)) == (150, 30)
    al, nt = v.verify_sweep(1, tok, synth.mask_from_layers(L, [2])[None])   # the sequence's own mask works
    assert v.length(1) == 30


# 4 blocks with 13B dimensions (d 5120, 40 heads x 128, FFN 13824), bf16
SHAPE13 = dataclasses.replace(synth.LLAMA_13B, n_layers=4, name="llama13b-4l")


def test_13b_dims_sweep_of_16_masks_vs_oracle():
    """17-node tree under all 16 masks of 4 blocks: steps of 7 segments
    (119 rows, two attention items of 64 and 55 rows), 7, then 2."""
    log("building the 4-layer 13B-dimension bf16 model (sweep of 16 masks x 17 nodes)")
    v = gpu_verifier(SHAPE13, n_seqs=1, max_tokens=600, max_nodes=17, max_batch=8)
    m = oracle_model(SHAPE13)
    ctx = synth.context_tokens(SHAPE13.vocab, 333, stream=2100)
    v.prefill(0, ctx)
    o = OracleSequence(m, np.zeros(4, np.uint8))
    prefill(m, o, ctx)
    parent = synth.topk_tree_parents((3, 2, 2, 1), (3, 5, 5, 3))
    masks = _all_masks(4)
    root = int(synth.context_tokens(SHAPE13.vocab, 1, stream=2101)[0])

    def greedy_of(tok, node):
        path = [node]
        while parent[path[-1]] >= 0:
            path.append(int(parent[path[-1]]))
        return int(verify(m, o, tok[path[::-1]]).greedy[-1])
    tokens = synth.tree_draft_tokens(parent, root, greedy_of, SHAPE13.vocab, 0.7, stream=2102)
    comp = _compare_sweep(SHAPE13, v, m, o, tokens, parent, masks, per_step=7)
    assert comp >= 4
    assert v.length(0) == 333
    v.close()


def _late_masks(n_layers):
    """The dense mask and every mask that runs layer 0 (first skip >= 1)."""
    return np.array([m for m in _all_masks(n_layers) if m[0] == 0], dtype=np.uint8)


def _prefix_case(shape, v, m, ctx_n, n, stream, random_gains):
    o = OracleSequence(m, np.zeros(shape.n_layers, np.uint8))
    ctx = synth.context_tokens(shape.vocab, ctx_n, stream=stream)
    v.prefill(0, ctx)
    prefill(m, o, ctx)
    tokens = synth.context_tokens(shape.vocab, n, stream=stream + 1)
    parent = synth.random_tree(n, stream=stream + 2, max_children=3)
    return o, tokens, parent


def _sweep_vs_oracle(shape, v, m, o, tokens, parent, masks, reuse):
    """Every mask's greedy tokens and decision against the oracle; the last
    step's logits (one or more masks, the last in first-skip order) too."""
    tol, gate = TOL[shape.dtype]
    n = len(tokens)
    al, nt, g = v.verify_sweep(0, tokens, masks, parent, want_greedy=True, reuse_prefix=reuse)
    res = [verify(m, o, np.asarray(tokens), parent, mk) for mk in masks]
    compared = 0
    for k, r in enumerate(res):
        sure = r.margin > gate
        np.testing.assert_array_equal(g[k][sure], r.greedy[sure], err_msg=f"mask {k}")
        if min(float(r.margin[i]) for i in r.path) > gate:
            assert (int(al[k]), int(nt[k])) == (r.accept_len, r.next_token), f"mask {k}"
            compared += 1
    return al, nt, g, res, compared


def test_tiny_sweep_prefix_reuse_one_mask_per_step():
    """8 free slots for an 8-node tree: one mask per step, so every step after
    the dense pass resumes at its mask's first skipped layer."""
    v = gpu_verifier(TINY, random_gains=True, n_seqs=1, max_tokens=88, max_nodes=8, max_batch=8)
    m = oracle_model(TINY, random_gains=True)
    o, tokens, parent = _prefix_case(TINY, v, m, 80, 8, 2200, True)
    masks = _late_masks(TINY.n_layers)          # dense, 0001, 0010, ..., 0111
    al, nt, g, res, comp = _sweep_vs_oracle(TINY, v, m, o, tokens, parent, masks, reuse=True)
    # the last step is mask 0100 or later in first-skip order: a step resumed at layer 1
    last = [k for k in range(len(masks)) if masks[k][1] == 1][-1]
    err = float(np.max(np.abs(v.logits(8) - res[last].logits)))
    log(f"tiny prefix reuse: {comp}/{len(masks)} decisions compared, resumed step logits max-abs {err:.2e}")
    assert err <= TOL["f32"][0]
    assert comp >= 6
    al2, nt2, g2 = v.verify_sweep(0, tokens, masks, parent, want_greedy=True, reuse_prefix=False)
    np.testing.assert_array_equal(al2, al)
    np.testing.assert_array_equal(nt2, nt)
    assert (g2 == g).mean() > 0.99
    assert v.length(0) == 80
    v.close()


def test_13b_dims_sweep_prefix_reuse_vs_oracle():
    """Two masks per step (rows 34), masks that all run layer 0: after the
    dense pass, steps {0001, 0010}, {0011, 0100}, {0101, 0110}, {0111}
    resume at layers 2, 1, 1 and 1 from its saved residual."""
    log("building the 4-layer 13B-dimension bf16 model (prefix reuse, 17-node tree)")
    v = gpu_verifier(SHAPE13, n_seqs=1, max_tokens=400, max_nodes=17, max_batch=2)
    m = oracle_model(SHAPE13)
    o, tokens, parent = _prefix_case(SHAPE13, v, m, 257, 17, 2300, False)
    masks = _late_masks(4)
    al, nt, g, res, comp = _sweep_vs_oracle(SHAPE13, v, m, o, tokens, parent, masks, reuse=True)
    err = float(np.max(np.abs(v.logits(17) - res[7].logits)))   # the last step: mask 0111 alone
    log(f"13B dims prefix reuse: {comp}/8 decisions compared, resumed step logits max-abs {err:.2e}")
    assert err <= TOL["bf16"][0]
    assert comp >= 3
    assert v.length(0) == 257
    v.close()
