"""GPU parity of tss_verify_batch: several sequences with their own contexts,
skip masks and draft trees verified in one step.

Each sequence's rows must equal the oracle's verify of that sequence alone
(the batch is independent sequences sharing weight reads); rows of a sequence
that skips a block stay untouched inside a launched block; a block every
sequence skips is not launched; commit and tree-path compaction work per
sequence.  The tiny fp32 decoder checks this element by element; a 4-layer
decoder with 13B dimensions checks the 72-row bf16 case of the batched
workload (8 sequences x 9 nodes).
"""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import OracleSequence, prefill, verify
from tests.gpu_common import TOL, check_decision, gpu_verifier, log, oracle_model, prefill_chunked

pytestmark = pytest.mark.gpu

TINY = synth.TINY


def _setup(v, m, shape, seqs, masks, ctx_lens, stream0):
    """Prefills each sequence under its own mask on both sides."""
    oseqs = []
    for sq, mask, n in zip(seqs, masks, ctx_lens):
        ctx = synth.context_tokens(shape.vocab, n, stream=stream0 + sq)
        v.truncate(sq, 0)
        v.set_mask(sq, mask)
        v.prefill(sq, ctx)
        o = OracleSequence(m, mask)
        prefill_chunked(m, o, ctx)
        oseqs.append(o)
    return oseqs


def _compare_batch(shape, v, m, seqs, oseqs, drafts, parents, masks=None, commit=False):
    """One batch step on the GPU, each sequence's verify on the oracle; returns
    (worst logits error, decisions compared)."""
    tol, gate = TOL[shape.dtype]
    al, nt = v.verify_batch(seqs, drafts, parents, masks, commit)
    n = sum(len(t) for t in drafts)
    lg, g = v.logits(n), v.greedy(n)
    off, worst, compared = 0, 0.0, 0
    for i, (o, tok) in enumerate(zip(oseqs, drafts)):
        par = None if parents is None else parents[i]
        mk = None if masks is None else masks[i]
        res = verify(m, o, np.asarray(tok), par, mk, commit)
        rows = slice(off, off + len(tok))
        err = float(np.max(np.abs(lg[rows] - res.logits)))
        assert err <= tol, f"sequence {i}: logits max-abs {err} > {tol}"
        sure = res.margin > gate
        np.testing.assert_array_equal(g[rows][sure], res.greedy[sure])
        compared += check_decision(res, int(al[i]), int(nt[i]), gate)
        worst = max(worst, err)
        off += len(tok)
    return worst, compared, (al, nt)


@pytest.fixture(scope="module")
def tiny():
    log("building tiny fp32 batch verifier (8 sequences x 8 nodes)")
    v = gpu_verifier(TINY, random_gains=True, n_seqs=8, max_tokens=400, max_nodes=8, max_batch=8)
    m = oracle_model(TINY, random_gains=True)
    yield v, m
    v.close()


TINY_MASKS = [[], [0], [3], [1, 2], [0, 1, 3], [0, 1, 2, 3], [2], []]


def _tiny_drafts(n_nodes, stream):
    drafts, parents = [], []
    for i, n in enumerate(n_nodes):
        drafts.append(synth.context_tokens(TINY.vocab, n, stream=stream + i))
        parents.append(synth.random_tree(n, stream=stream + 50 + i, max_children=3) if i % 2 else None)
    return drafts, parents


def test_batch_vs_oracle_mixed_masks_and_trees(tiny):
    v, m = tiny
    seqs = list(range(8))
    masks = [synth.mask_from_layers(TINY.n_layers, s) for s in TINY_MASKS]
    oseqs = _setup(v, m, TINY, seqs, masks, [5, 16, 17, 60, 130, 33, 250, 1], 300)
    drafts, parents = _tiny_drafts([6, 8, 1, 7, 3, 8, 5, 8], 400)
    err, comp, _ = _compare_batch(TINY, v, m, seqs, oseqs, drafts, parents)
    log(f"tiny batch of 8: worst logits err {err:.2e}, {comp} decisions compared")


def test_batch_block_skipped_by_all(tiny):
    """Layer 1 skipped by every sequence (never launched), layer 3 by some; a
    sequence order other than the id order; explicit per-call masks."""
    v, m = tiny
    seqs = [5, 2, 7]
    masks = [synth.mask_from_layers(TINY.n_layers, s) for s in ([1], [1, 3], [0, 1])]
    oseqs = _setup(v, m, TINY, seqs, masks, [40, 9, 77], 500)
    drafts, parents = _tiny_drafts([4, 8, 2], 600)
    err, comp, _ = _compare_batch(TINY, v, m, seqs, oseqs, drafts, parents, masks=masks)
    log(f"block skipped by all: worst logits err {err:.2e}, {comp} compared")


def test_batch_commit_then_next_step(tiny):
    """Committing batch (tree paths compacted per sequence), then a second batch
    step on the grown contexts, both against the oracle doing the same."""
    v, m = tiny
    seqs = [0, 1, 2, 3]
    masks = [synth.mask_from_layers(TINY.n_layers, s) for s in ([], [2], [0, 3], [1])]
    oseqs = _setup(v, m, TINY, seqs, masks, [20, 35, 50, 65], 700)
    # drafts that follow the oracle's greedy tokens along a non-first branch,
    # so the accepted paths are not prefixes and compaction has work to do
    drafts, parents = [], []
    for i, o in enumerate(oseqs):
        parent = np.array([-1, 0, 0, 2, 2, 4], dtype=np.int32)
        tok = np.zeros(6, dtype=np.int64)
        tok[0] = int(synth.context_tokens(TINY.vocab, 1, stream=800 + i)[0])
        g0 = int(verify(m, o, tok[:1]).greedy[0])
        tok[1], tok[2] = (g0 + 1) % TINY.vocab, g0
        r = verify(m, o, tok[:3], parent[:3])
        tok[3], tok[4] = (int(r.greedy[2]) + 5) % TINY.vocab, int(r.greedy[2])
        r = verify(m, o, tok[:5], parent[:5])
        tok[5] = int(r.greedy[4])
        drafts.append(tok)
        parents.append(parent)
    err, comp, (al, nt) = _compare_batch(TINY, v, m, seqs, oseqs, drafts, parents, commit=True)
    for sq, o in zip(seqs, oseqs):
        assert v.length(sq) == o.n_kv
    drafts2 = [np.concatenate([[nt[i]], synth.context_tokens(TINY.vocab, 4, stream=900 + i)]) for i in range(4)]
    err2, comp2, _ = _compare_batch(TINY, v, m, seqs, oseqs, drafts2, None, commit=True)
    for sq, o in zip(seqs, oseqs):
        assert v.length(sq) == o.n_kv
    log(f"batch commit: accept {list(al)}, errs {err:.2e} {err2:.2e}, compared {comp}+{comp2}")
    assert comp >= 2


def test_batch_of_one_is_bit_exact_with_verify(tiny):
    v, m = tiny
    masks = [synth.mask_from_layers(TINY.n_layers, [2])]
    _setup(v, m, TINY, [4], masks, [45], 1000)
    tok = synth.context_tokens(TINY.vocab, 7, stream=1001)
    parent = synth.random_tree(7, stream=1002)
    a = v.verify(4, tok, parent)
    la = v.logits(7)
    al, nt = v.verify_batch([4], [tok], [parent])
    assert (int(al[0]), int(nt[0])) == a
    np.testing.assert_array_equal(v.logits(7), la)


def test_batch_graph_replays_match_direct(tiny):
    from paper_2609_26100_amd import tss as abi
    v, m = tiny
    seqs = [6, 3, 0]
    masks = [synth.mask_from_layers(TINY.n_layers, s) for s in ([0], [], [2, 3])]
    _setup(v, m, TINY, seqs, masks, [70, 18, 100], 1100)
    drafts, parents = _tiny_drafts([5, 8, 3], 1200)
    v.set_launch_mode(abi.TSS_LAUNCH_DIRECT)
    ref = v.verify_batch(seqs, drafts, parents)
    ref_lg = v.logits(16)
    v.set_launch_mode(abi.TSS_LAUNCH_GRAPH)
    for _ in range(3):
        out = v.verify_batch(seqs, drafts, parents)
        np.testing.assert_array_equal(out[0], ref[0])
        np.testing.assert_array_equal(out[1], ref[1])
        np.testing.assert_array_equal(v.logits(16), ref_lg)
        v.verify(3, drafts[1][:2])   # an eager single-sequence step in between


def test_batch_errors_leave_state_unchanged(tiny):
    from paper_2609_26100_amd import tss as abi
    v, m = tiny
    masks = [synth.mask_from_layers(TINY.n_layers, s) for s in ([], [1])]
    _setup(v, m, TINY, [0, 1], masks, [12, 13], 1300)
    t = [np.array([1, 2, 3]), np.array([4, 5])]
    bad_calls = [
        (([0, 0], t), abi.TSS_EINVAL),                                   # same sequence twice
        (([0, 8], t), abi.TSS_EINVAL),                                   # unknown sequence
        (([0, 1], [np.arange(9), t[1]]), abi.TSS_EINVAL),                # more nodes than max_nodes
        (([0, 1], [t[0], np.array([4, TINY.vocab])]), abi.TSS_EINVAL),   # token outside the vocabulary
        (([0, 1], t, [np.array([-1, 0, 2]), None]), abi.TSS_EINVAL),     # parent not before the node
        (([0, 1], t, None, [None, np.zeros(TINY.n_layers)]), abi.TSS_ESTATE),  # layer 1 has no KV for seq 1
    ]
    for args, status in bad_calls:
        with pytest.raises(abi.TSSError) as e:
            v.verify_batch(*args, commit=True)
        assert e.value.status == status, args
    with pytest.raises(abi.TSSError) as e:
        v.verify_batch(list(range(8)) + [0], [np.array([1])] * 9)        # more sequences than max_batch
    assert e.value.status == abi.TSS_EINVAL
    assert (v.length(0), v.length(1)) == (12, 13)
    al, nt = v.verify_batch([0, 1], t, commit=True)
    assert v.length(0) == 12 + al[0] + 1 and v.length(1) == 13 + al[1] + 1


# 4 blocks with 13B dimensions (d 5120, 40 heads x 128, FFN 13824), bf16
SHAPE13 = dataclasses.replace(synth.LLAMA_13B, n_layers=4, name="llama13b-4l")


def test_13b_dims_batch_of_8_vs_oracle():
    log("building the 4-layer 13B-dimension bf16 model (batch of 8 x 9 nodes)")
    v = gpu_verifier(SHAPE13, n_seqs=8, max_tokens=400, max_nodes=9, max_batch=8)
    m = oracle_model(SHAPE13)
    seqs = list(range(8))
    rng = np.random.default_rng(7)
    masks = [synth.random_skip_mask(4, 0, 3, int(rng.integers(0, 3)), stream=20 + i) for i in seqs]
    ctx_lens = [int(x) for x in rng.integers(40, 300, size=8)]
    log(f"contexts {ctx_lens}, masks {[list(np.nonzero(mk)[0]) for mk in masks]}")
    oseqs = _setup(v, m, SHAPE13, seqs, masks, ctx_lens, 1400)
    worst, comp = 0.0, 0
    for rep in range(2):
        drafts = []
        for i, o in enumerate(oseqs):
            root = int(synth.context_tokens(SHAPE13.vocab, 1, stream=1500 + 10 * rep + i)[0])
            g, cur = [], [root]
            for _ in range(8):
                g.append(int(verify(m, o, np.asarray(cur)).greedy[-1]))
                cur.append(g[-1])
            drafts.append(np.concatenate([[root], synth.chain_draft(np.asarray(g), SHAPE13.vocab, p_accept=0.6,
                                                                    stream=1600 + 10 * rep + i)]))
        err, c, (al, nt) = _compare_batch(SHAPE13, v, m, seqs, oseqs, drafts, None)
        worst, comp = max(worst, err), comp + c
        log(f"13B dims batch rep {rep}: accept {list(al)}, logits err {err:.3e}, compared {c}/8")
    v.close()
    assert comp >= 8


# 2 blocks with 13B dimensions and room for 4160 tokens per sequence: a batch
# whose contexts exceed 1024 tokens takes one attention workgroup per 64 pages
# of each sequence, merged across workgroups (the path of the 13B batch
# workload, contexts 512-4096)
SHAPE13_2 = dataclasses.replace(synth.LLAMA_13B, n_layers=2, name="llama13b-2l")


def test_13b_dims_batch_long_contexts_vs_oracle():
    log("building the 2-layer 13B-dimension bf16 model (batch of 8 x 9 nodes, 4160 tokens per sequence)")
    v = gpu_verifier(SHAPE13_2, n_seqs=8, max_tokens=4160, max_nodes=9, max_batch=8)
    m = oracle_model(SHAPE13_2)
    seqs = list(range(8))
    ctx_lens = [1100, 2100, 64, 300, 1300, 40, 200, 520]
    # the long contexts run both blocks; the others skip one block or none
    skips = [[], [], [0], [1], [], [1], [0], []]
    masks = [synth.mask_from_layers(2, sk) for sk in skips]
    log(f"contexts {ctx_lens}, skipped blocks {skips}")
    oseqs = _setup(v, m, SHAPE13_2, seqs, masks, ctx_lens, 1700)
    drafts = []
    for i, o in enumerate(oseqs):
        root = int(synth.context_tokens(SHAPE13_2.vocab, 1, stream=1800 + i)[0])
        g, cur = [], [root]
        for _ in range(8):
            g.append(int(verify(m, o, np.asarray(cur)).greedy[-1]))
            cur.append(g[-1])
        drafts.append(np.concatenate([[root], synth.chain_draft(np.asarray(g), SHAPE13_2.vocab, p_accept=0.6,
                                                                stream=1900 + i)]))
    err, comp, (al, nt) = _compare_batch(SHAPE13_2, v, m, seqs, oseqs, drafts, None)
    # the last launched block (1) serves the sequences that run it, one item each
    split = v.attn_split()
    log(f"13B dims long batch: accept {list(al)}, logits err {err:.3e}, compared {comp}/8; split {split}")
    runs1 = [i for i in seqs if 1 not in skips[i]]
    assert [r for _, r in split] == [9] * len(runs1)
    groups = dict(zip(runs1, [gr for gr, _ in split]))
    assert all(groups[i] >= 2 for i in (0, 1, 4)), groups
    assert groups[1] > groups[0], groups
    v.check_kv()
    v.close()
    assert comp >= 4
