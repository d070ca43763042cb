"""tss_verify_static, the entry point that allocates nothing (the step's
workspace lives in the library's static device scratch), against
tss_verify with the context's own workspace: identical decisions, greedy
tokens, logits and commits, on two calls in a row (the second with fewer
nodes), across two models of different shapes that share the scratch (the
7B-dimension one at a 1024-token context, where attention merges partial
states across workgroups through counters in the scratch), interleaved with
graph replays of tss_verify, and a model too large for the scratch is
refused before any device work."""
import dataclasses

import numpy as np
import pytest

import synth
from paper_2609_26100_amd import tss as abi
from tests.gpu_common import gpu_verifier, log

pytestmark = pytest.mark.gpu

TINY = synth.TINY
SHAPE7 = dataclasses.replace(synth.LLAMA_7B, name="llama-7b-dims-2L", n_layers=2)


def _both(v, seq, tok, parent=None, mask=None, commit=False):
    """(decision, logits, greedy) of tss_verify, then of tss_verify_static, on the same sequence state."""
    n = len(tok)
    flags = abi.TSS_COMMIT if commit else 0
    ref = v.verify(seq, tok, parent, mask)
    ref_lg, ref_g = v.logits(n), v.greedy(n)
    st = abi.tss_verify_static(v.ctx, seq, tok, parent, mask, flags)
    st_lg, st_g = v.logits(n), v.greedy(n)
    return (ref, ref_lg, ref_g), (st, st_lg, st_g)


def _check(pair, n):
    (ref, ref_lg, ref_g), (st, st_lg, st_g) = pair
    assert st == ref
    np.testing.assert_array_equal(st_g, ref_g)
    np.testing.assert_array_equal(st_lg, ref_lg)
    assert st_lg.shape[0] == n


def test_static_verify_equals_verify_on_consecutive_calls():
    v = gpu_verifier(TINY, random_gains=True, n_seqs=2, max_tokens=300, max_nodes=16)
    for sq in (0, 1):
        v.prefill(sq, synth.context_tokens(TINY.vocab, 100, stream=80))
    tree = synth.random_tree(12, stream=81, max_children=3)
    tok12 = synth.context_tokens(TINY.vocab, 12, stream=82)
    tok3 = synth.context_tokens(TINY.vocab, 3, stream=83)
    mask = synth.mask_from_layers(TINY.n_layers, [1])
    first = _both(v, 0, tok12, tree, mask)
    _check(first, 12)
    _check(_both(v, 0, tok3), 3)                       # the second call: fewer nodes
    # the context's graph replays still use its own workspace afterwards
    assert v.verify(0, tok12, tree, mask) == first[0][0]
    np.testing.assert_array_equal(v.logits(12), first[0][1])
    # committing: the static call on sequence 1 grows it as tss_verify grows sequence 0
    a = v.verify(0, tok12, tree, commit=True)
    b = abi.tss_verify_static(v.ctx, 1, tok12, tree, None, abi.TSS_COMMIT)
    assert a == b and v.length(0) == v.length(1) == 100 + a[0] + 1
    _check(_both(v, 1, tok3), 3)
    np.testing.assert_array_equal(v.logits(3), abi.tss_get_logits(v.ctx, 3, TINY.vocab))
    v.check_kv()
    v.close()


def test_static_verify_shared_by_two_models():
    t = gpu_verifier(TINY, random_gains=True, n_seqs=1, max_tokens=200, max_nodes=16)
    w = gpu_verifier(SHAPE7, n_seqs=1, max_tokens=1100, max_nodes=64)
    ctx = synth.context_tokens(SHAPE7.vocab, 1025, stream=84)
    w.prefill(0, ctx[:1024])
    t.prefill(0, synth.context_tokens(TINY.vocab, 60, stream=85))
    parent = synth.topk_tree_parents((4, 3, 2, 2, 1, 1), (4, 12, 20, 12, 8, 4))
    tok61 = np.concatenate([[ctx[1024]], synth.context_tokens(SHAPE7.vocab, 60, stream=86)])
    tok6 = np.concatenate([[ctx[1024]], synth.context_tokens(SHAPE7.vocab, 5, stream=87)])
    tiny_tok = synth.context_tokens(TINY.vocab, 9, stream=88)
    for rep in range(2):
        pw = _both(w, 0, tok61, parent)
        split = w.attn_split()
        log(f"7B dims, 61-node tree at 1024 tokens, static call {rep}: split {split}")
        assert split and all(g >= 2 for g, _ in split)
        _check(pw, 61)
        _check(_both(t, 0, tiny_tok), 9)
        _check(_both(w, 0, tok6), 6)                     # a smaller input on the larger model
    t.close()
    w.close()


def test_static_verify_refuses_models_beyond_the_scratch():
    import torch
    big = synth.ModelShape("d8192-v64000", 90, n_layers=1, d_model=8192, n_heads=64, head_dim=128, ffn_dim=64,
                           vocab=64000)
    cfg = abi.make_cfg(big, 64, 1)
    need = abi.tss_static_workspace_bytes(cfg)
    assert need > abi.TSS_STATIC_SCRATCH_BYTES
    wb, sb, kb = abi.tss_weights_bytes(cfg), abi.tss_workspace_bytes(cfg), abi.tss_kv_bytes(cfg, 1, 64)
    wt = torch.empty(wb, dtype=torch.uint8, device="cuda:0")
    ws = torch.zeros(sb, dtype=torch.uint8, device="cuda:0")
    kv = torch.zeros(kb, dtype=torch.uint8, device="cuda:0")
    torch.cuda.synchronize()
    ctx = abi.tss_create(cfg, torch.cuda.current_stream().cuda_stream, wt.data_ptr(), wb, ws.data_ptr(), sb)
    try:
        abi.tss_kv_alloc(ctx, 1, 64, kv.data_ptr(), kb)
        with pytest.raises(abi.TSSError) as e:
            abi.tss_verify_static(ctx, 0, np.array([1, 2, 3]))
        assert e.value.status == abi.TSS_ENOSPACE and "static scratch" in str(e.value)
        assert abi.tss_seq_length(ctx, 0) == 0
    finally:
        abi.tss_destroy(ctx)
