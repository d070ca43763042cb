"""The seeded input generators: determinism, bf16 rounding, and the structure
of drafts, trees and masks they promise."""
import numpy as np
import torch

import synth


def test_weights_deterministic_and_distributed():
    a = synth.weight_tensor(synth.TINY, "wq", 1)
    b = synth.weight_tensor(synth.TINY, "wq", 1, threads=1)
    np.testing.assert_array_equal(a, b)
    c = synth.weight_tensor(synth.TINY, "wq", 2)
    assert not np.array_equal(a, c)
    assert a.shape == (256, 256) and a.dtype == np.float32
    assert abs(float(a.std()) - 0.02) < 0.001 and abs(float(a.mean())) < 0.001
    g = synth.weight_tensor(synth.TINY, "attn_norm", 0)
    np.testing.assert_array_equal(g, np.ones(256, np.float32))


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 3
    x[:4] = [1.00390625, 1.01171875, -2.5, 0.0]   # exact ties and exact values
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(synth.bf16_bits(x), ref)
    r = synth.bf16_round(x)
    np.testing.assert_array_equal(torch.from_numpy(x).to(torch.bfloat16).float().numpy(), r)


def test_bf16_shape_weights_are_bf16_exact():
    import dataclasses
    sh = dataclasses.replace(synth.TINY, dtype="bf16")
    w = synth.weight_tensor(sh, "w_up", 0)
    np.testing.assert_array_equal(w, synth.bf16_round(w))
    bits = synth.weight_tensor(sh, "w_up", 0, as_bf16_bits=True)
    np.testing.assert_array_equal((bits.astype(np.uint32) << 16).view(np.float32), w)


def test_chain_draft_structure():
    g = np.arange(100, 105)
    d = synth.chain_draft(g, 4096, n_greedy=3)
    assert list(d[:3]) == [100, 101, 102] and d[3] != 103 and d[4] != 104
    hits = []
    for s in range(400):
        d = synth.chain_draft(np.arange(5), 32000, p_accept=0.6, stream=s)
        hits.extend(d == np.arange(5))
    assert abs(np.mean(hits) - 0.6) < 0.03


def test_topk_tree_shape():
    p = synth.topk_tree_parents((4, 3, 2, 2, 1, 1), (4, 12, 20, 12, 8, 4))
    assert len(p) == 61 and p[0] == -1 and all(0 <= p[i] < i for i in range(1, 61))
    depth = np.zeros(61, int)
    for i in range(1, 61):
        depth[i] = depth[p[i]] + 1
    assert depth.max() == 6
    assert [int((depth == k).sum()) for k in range(1, 7)] == [4, 12, 20, 12, 8, 4]
    kids = np.bincount(p[1:], minlength=61)
    for i in range(61):
        assert kids[i] <= (4, 3, 2, 2, 1, 1, 0)[depth[i]]


def test_tree_tokens_distinct_siblings():
    p = synth.topk_tree_parents((3, 2), (3, 4))
    tok = synth.tree_draft_tokens(p, 5, lambda t, n: 7, 100, p_accept=1.0)
    for node in range(len(p)):
        kids = [i for i in range(1, len(p)) if p[i] == node]
        assert len(set(tok[kids])) == len(kids)
        if kids:
            assert 7 in set(tok[kids])


def test_masks_nested_and_in_range():
    ms = synth.nested_skip_masks(32, 16, 31, (0, 4, 8))
    assert ms[0].sum() == 0 and ms[4].sum() == 4 and ms[8].sum() == 8
    assert np.all(ms[8][:16] == 0)
    assert np.all(ms[8] >= ms[4])
    r = synth.random_skip_mask(60, 2, 59, 10)
    assert r.sum() == 10 and r[:2].sum() == 0


def test_context_tokens_range():
    t = synth.context_tokens(32000, 5000)
    assert t.min() >= 0 and t.max() < 32000 and t.dtype == np.int32
    np.testing.assert_array_equal(t, synth.context_tokens(32000, 5000))
