"""GPU parity on the tiny fp32 decoder (4 layers, d 256, 4 heads x 64, FFN 704,
vocab 4096): every kernel of the verify path against the oracle, element by
element, plus the properties that must hold bit-exactly on the GPU."""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import OracleSequence, prefill, verify
from tests.gpu_common import compare_step, gpu_verifier, log, oracle_model

pytestmark = pytest.mark.gpu

SHAPE = synth.TINY
L = SHAPE.n_layers


@pytest.fixture(scope="module")
def pair():
    log("building tiny fp32 verifier (random gains)")
    v = gpu_verifier(SHAPE, random_gains=True, n_seqs=4, max_tokens=600, max_nodes=64)
    m = oracle_model(SHAPE, random_gains=True)
    yield v, m
    v.close()


def _fresh(v, m, seq, mask, ctx):
    v.truncate(seq, 0)
    v.set_mask(seq, mask)
    v.prefill(seq, ctx)
    o = OracleSequence(m, mask)
    prefill(m, o, ctx)
    assert v.length(seq) == o.n_kv == len(ctx)
    return o


def test_all_blocks_skipped(pair):
    v, m = pair
    mask = np.ones(L, np.uint8)
    ctx = synth.context_tokens(SHAPE.vocab, 20, stream=1)
    o = _fresh(v, m, 0, mask, ctx)
    tok = synth.context_tokens(SHAPE.vocab, 6, stream=2)
    _, _, err, _ = compare_step(SHAPE, v, 0, m, o, tok)
    log(f"all skipped: logits err {err:.2e}")


@pytest.mark.parametrize("skip", [[], [0], [3], [1, 2], [0, 1, 3]])
def test_masks_chain(pair, skip):
    v, m = pair
    mask = synth.mask_from_layers(L, skip)
    ctx = synth.context_tokens(SHAPE.vocab, 57, stream=3)
    o = _fresh(v, m, 1, mask, ctx)
    tok = synth.context_tokens(SHAPE.vocab, 6, stream=4)
    _, _, err, _ = compare_step(SHAPE, v, 1, m, o, tok)
    log(f"mask {skip}: logits err {err:.2e}")


def test_tiny_workload(pair):
    """128 context tokens in KV, root, chain k=5 (3 greedy then 2 other tokens), mask {2}."""
    v, m = pair
    mask = synth.mask_from_layers(L, [2])
    toks = synth.context_tokens(SHAPE.vocab, 129)
    ctx, root = toks[:128], int(toks[128])
    o = _fresh(v, m, 0, mask, ctx)
    g, cur = [], [root]
    for _ in range(5):
        g.append(int(verify(m, o, np.asarray(cur)).greedy[-1]))
        cur.append(g[-1])
    drafts = synth.chain_draft(np.asarray(g), SHAPE.vocab, n_greedy=3)
    res, (al, nt), err, compared = compare_step(SHAPE, v, 0, m, o, np.concatenate([[root], drafts]))
    log(f"tiny workload: accept {al} next {nt} (oracle {res.accept_len} {res.next_token}) err {err:.2e}")
    assert res.accept_len == 3 and compared


@pytest.mark.parametrize("n_nodes", [1, 2, 8, 17, 33, 64])
def test_trees(pair, n_nodes):
    v, m = pair
    mask = synth.mask_from_layers(L, [1])
    ctx = synth.context_tokens(SHAPE.vocab, 45, stream=5)
    o = _fresh(v, m, 2, mask, ctx)
    parent = synth.random_tree(n_nodes, stream=n_nodes, max_children=4)
    tok = synth.context_tokens(SHAPE.vocab, n_nodes, stream=6 + n_nodes)
    _, _, err, _ = compare_step(SHAPE, v, 2, m, o, tok, parent)
    log(f"tree {n_nodes}: logits err {err:.2e}")


def test_prefill_chunks_and_context_lengths(pair):
    """Contexts that end inside and at page edges, prefilled in several chunks."""
    v, m = pair
    for n in (1, 15, 16, 17, 64, 65, 200):
        ctx = synth.context_tokens(SHAPE.vocab, n, stream=100 + n)
        o = _fresh(v, m, 3, np.zeros(L, np.uint8), ctx)
        tok = synth.context_tokens(SHAPE.vocab, 3, stream=200 + n)
        _, _, err, _ = compare_step(SHAPE, v, 3, m, o, tok)
        log(f"context {n}: logits err {err:.2e}")


def test_tree_commit_then_chain(pair):
    v, m = pair
    mask = synth.mask_from_layers(L, [3])
    ctx = synth.context_tokens(SHAPE.vocab, 31, stream=7)
    o = _fresh(v, m, 1, mask, ctx)
    parent = np.array([-1, 0, 0, 1, 2, 2, 4, 4, 6], dtype=np.int32)
    # tokens along 0 -> 2 -> 5 follow the oracle's greedy choices so the accepted path is not a prefix
    tok = np.array([int(synth.context_tokens(SHAPE.vocab, 1, stream=8)[0])] + [0] * 8, dtype=np.int64)
    g = verify(m, o, tok[:1]).greedy
    tok[1], tok[2] = (g[0] + 1) % SHAPE.vocab, g[0]
    res = verify(m, o, tok[:3], parent[:3])
    tok[3], tok[4] = 11, (res.greedy[2] + 3) % SHAPE.vocab
    tok[5] = res.greedy[2]
    res = verify(m, o, tok[:6], parent[:6])
    tok[6], tok[7], tok[8] = res.greedy[4], 12, 13
    res, (al, nt), err, compared = compare_step(SHAPE, v, 1, m, o, tok, parent, commit=True)
    assert compared and res.path == [0, 2, 5] and al == 2
    assert v.length(1) == o.n_kv == 31 + 3
    nxt = np.concatenate([[nt], synth.context_tokens(SHAPE.vocab, 4, stream=9)])
    _, _, err2, _ = compare_step(SHAPE, v, 1, m, o, nxt)
    log(f"tree commit: errs {err:.2e} {err2:.2e}")


def test_chain_as_tree_is_bit_exact(pair):
    v, m = pair
    ctx = synth.context_tokens(SHAPE.vocab, 40, stream=10)
    _fresh(v, m, 0, np.zeros(L, np.uint8), ctx)
    tok = synth.context_tokens(SHAPE.vocab, 7, stream=11)
    a = v.verify(0, tok)
    la = v.logits(7)
    b = v.verify(0, tok, np.arange(-1, 6, dtype=np.int32))
    lb = v.logits(7)
    assert a == b
    np.testing.assert_array_equal(la, lb)


def test_run_to_run_bit_exact(pair):
    v, m = pair
    ctx = synth.context_tokens(SHAPE.vocab, 70, stream=12)
    _fresh(v, m, 0, synth.mask_from_layers(L, [0]), ctx)
    tok = synth.context_tokens(SHAPE.vocab, 20, stream=13)
    parent = synth.random_tree(20, stream=14)
    outs = []
    for _ in range(3):
        v.verify(0, tok, parent)
        outs.append(v.logits(20))
    np.testing.assert_array_equal(outs[0], outs[1])
    np.testing.assert_array_equal(outs[0], outs[2])


def test_page_permutation_is_bit_exact(pair):
    v, m = pair
    ctx = synth.context_tokens(SHAPE.vocab, 90, stream=15)
    tok = synth.context_tokens(SHAPE.vocab, 6, stream=16)
    _fresh(v, m, 0, np.zeros(L, np.uint8), ctx)
    v.verify(0, tok)
    ref = v.logits(6)
    n_pages = 4 * ((600 + 15) // 16)
    order = np.random.default_rng(3).permutation(n_pages).astype(np.int32)
    w = gpu_verifier(SHAPE, random_gains=True, n_seqs=4, max_tokens=600, max_nodes=64, page_order=order)
    w.prefill(0, ctx)
    w.verify(0, tok)
    np.testing.assert_array_equal(w.logits(6), ref)
    w.close()


def test_skip_equals_deleted_block_bit_exact(pair):
    """GPU with mask {l} is bit-identical to the GPU on the model with block l deleted."""
    v, m = pair
    l = 2
    short = dataclasses.replace(SHAPE, n_layers=L - 1)
    short_names = {i: (ly, nm) for i, ly, nm in synth.tensor_names(L - 1)}

    def get_short(idx):
        ly, nm = short_names[idx]
        return synth.weight_tensor(SHAPE, nm, ly + 1 if ly >= l else ly, random_gains=True)
    from paper_2609_26100_amd.verifier import Verifier
    w = Verifier(short, n_seqs=1, max_tokens=600, max_nodes=64)
    w.load(get_short)
    ctx = synth.context_tokens(SHAPE.vocab, 50, stream=17)
    tok = synth.context_tokens(SHAPE.vocab, 9, stream=18)
    parent = synth.random_tree(9, stream=19)
    _fresh(v, m, 0, synth.mask_from_layers(L, [l]), ctx)
    a = v.verify(0, tok, parent)
    w.prefill(0, ctx)
    b = w.verify(0, tok, parent)
    assert a == b
    np.testing.assert_array_equal(v.logits(9), w.logits(9))
    w.close()


def test_own_greedy_drafts_fully_accepted(pair):
    v, m = pair
    ctx = synth.context_tokens(SHAPE.vocab, 33, stream=20)
    _fresh(v, m, 0, synth.mask_from_layers(L, [1]), ctx)
    cur = [int(synth.context_tokens(SHAPE.vocab, 1, stream=21)[0])]
    for _ in range(6):
        v.verify(0, cur)
        cur.append(int(v.greedy(len(cur))[-1]))
    al, nt = v.verify(0, cur[:6])
    assert al == 5 and nt == cur[6]


def test_errors_leave_state_unchanged(pair):
    from paper_2609_26100_amd import tss as abi
    v, m = pair
    ctx = synth.context_tokens(SHAPE.vocab, 10, stream=22)
    _fresh(v, m, 0, synth.mask_from_layers(L, [2]), ctx)
    with pytest.raises(abi.TSSError) as e:   # layer 2 has no KV for the context
        v.verify(0, [1, 2], mask=np.zeros(L, np.uint8))
    assert e.value.status == abi.TSS_ESTATE
    with pytest.raises(abi.TSSError) as e:
        v.verify(0, [1, SHAPE.vocab])
    assert e.value.status == abi.TSS_EINVAL
    with pytest.raises(abi.TSSError) as e:
        v.verify(0, [1, 2, 3], [-1, 0, 2])
    assert e.value.status == abi.TSS_EINVAL
    with pytest.raises(abi.TSSError) as e:
        v.verify(0, list(range(65)))
    assert e.value.status == abi.TSS_EINVAL
    with pytest.raises(abi.TSSError) as e:
        v.prefill(0, np.zeros(600, np.int32))
    assert e.value.status == abi.TSS_ECAPACITY
    assert v.length(0) == 10
    # still usable
    v.verify(0, [1, 2], commit=True)
    assert v.length(0) in (11, 12)


def test_graph_replays_match_direct_launches(pair):
    """Captured steps, replayed several times with eager steps in between, are
    bit-identical to direct launches (chain, tree, two masks)."""
    from paper_2609_26100_amd import tss as abi
    v, m = pair
    ctx = synth.context_tokens(SHAPE.vocab, 77, stream=50)
    _fresh(v, m, 0, synth.mask_from_layers(L, [1]), ctx)
    cases = [
        (synth.context_tokens(SHAPE.vocab, 6, stream=51), None, None),
        (synth.context_tokens(SHAPE.vocab, 9, stream=52), synth.random_tree(9, stream=53), None),
        (synth.context_tokens(SHAPE.vocab, 3, stream=54), None, synth.mask_from_layers(L, [1, 3])),
    ]
    v.set_launch_mode(abi.TSS_LAUNCH_DIRECT)
    ref = []
    for tok, par, mask in cases:
        ref.append((v.verify(0, tok, par, mask), v.logits(len(tok))))
    for rep in range(3):
        v.set_launch_mode(abi.TSS_LAUNCH_GRAPH)
        for (tok, par, mask), (r, lg) in zip(cases, ref):
            assert v.verify(0, tok, par, mask) == r
            np.testing.assert_array_equal(v.logits(len(tok)), lg)
        v.set_launch_mode(abi.TSS_LAUNCH_DIRECT)
        assert v.verify(0, *cases[0][:2]) == ref[0][0]
    v.set_launch_mode(abi.TSS_LAUNCH_GRAPH)


@pytest.mark.parametrize("mode", [0, 1])
def test_committing_decode_loop(pair, mode):
    """Committing steps in a row (in graph mode the same captured graph is
    replayed at a growing context length) against the oracle doing the same
    steps.  Each step uses a draft whose decision the oracle takes with margin;
    when the root itself has no margin the loop moves to a fresh context."""
    from paper_2609_26100_amd import tss as abi
    v, m = pair
    v.set_launch_mode(mode)
    mask = synth.mask_from_layers(L, [2])
    gate = 1e-3
    steps = 0
    for ctx_stream in range(60, 66):
        ctx = synth.context_tokens(SHAPE.vocab, 90, stream=ctx_stream)
        o = _fresh(v, m, 1, mask, ctx)
        root = int(synth.context_tokens(SHAPE.vocab, 1, stream=ctx_stream + 100)[0])
        for step in range(5):
            g, cur = [], [root]
            for _ in range(4):
                g.append(int(verify(m, o, np.asarray(cur)).greedy[-1]))
                cur.append(g[-1])
            tok = None
            for attempt in range(8):
                drafts = synth.chain_draft(np.asarray(g), SHAPE.vocab, p_accept=0.7,
                                           stream=1000 * ctx_stream + 100 * step + attempt)
                cand = np.concatenate([[root], drafts])
                r = verify(m, o, cand)
                if float(r.margin[r.path].min()) > gate:
                    tok = cand
                    break
            if tok is None:
                break
            res, (al, nt), err, compared = compare_step(SHAPE, v, 1, m, o, tok, commit=True)
            assert compared and v.length(1) == o.n_kv
            root = nt
            steps += 1
        if steps >= 6:
            break
    assert steps >= 6
    v.set_launch_mode(abi.TSS_LAUNCH_GRAPH)


def test_nan_logits_pick_the_first_nan():
    """Degenerate logits: lm_head rows 17 and 3000 hold NaN, so those two
    logits are NaN for every node.  The greedy token is then the first NaN
    index, as in the oracle's (numpy's) argmax, and never an out-of-range
    index: every node's greedy token is 17, a chain of 17s is fully
    accepted and the bonus token is 17."""
    from paper_2609_26100_amd.verifier import Verifier

    names = {i: (layer, nm) for i, layer, nm in synth.tensor_names(L)}
    base = synth.abi_tensor_loader(SHAPE)

    def poisoned(a):
        a = np.array(a, copy=True)
        a[[17, 3000]] = np.nan
        return a

    def get(index):
        a = base(index)
        return poisoned(a) if names[index][1] == "lm_head" else a

    ocache = {}

    def oget(name, layer):
        if (name, layer) not in ocache:
            t = synth.weight_tensor(SHAPE, name, layer)
            ocache[(name, layer)] = poisoned(t) if name == "lm_head" else t
        return ocache[(name, layer)]

    from oracle import OracleModel
    v = Verifier(SHAPE, n_seqs=1, max_tokens=128, max_nodes=16)
    try:
        v.load(get)
        m = OracleModel(SHAPE, oget)
        ctx = synth.context_tokens(SHAPE.vocab, 30, stream=77)
        v.prefill(0, ctx)
        o = OracleSequence(m, None)
        prefill(m, o, ctx)
        tok = np.array([5, 17, 17, 17, 17, 17], np.int32)
        res = verify(m, o, tok)
        al, nt = v.verify(0, tok)
        g = v.greedy(len(tok))
        lg = v.logits(len(tok))
        assert np.isnan(lg[:, [17, 3000]]).all() and np.isnan(res.logits[:, [17, 3000]]).all()
        np.testing.assert_array_equal(res.greedy, np.full(len(tok), 17))
        np.testing.assert_array_equal(g, np.full(len(tok), 17))
        assert (al, nt) == (res.accept_len, res.next_token) == (5, 17)
        finite = np.isfinite(res.logits)
        assert float(np.max(np.abs(lg[finite] - res.logits[finite]))) <= 1e-4
    finally:
        v.close()


def test_kv_rebind_drops_captured_steps():
    """Steps captured for one KV binding must not survive a rebind: after
    verifies have been captured and replayed, the context is rebound to a new
    pool (another size, permuted pages) and the old pool is filled with a
    sentinel.  Prefill and verify (chain and tree) on the new pool must equal
    a fresh context bit for bit, and the old pool must stay untouched."""
    import torch
    v = gpu_verifier(SHAPE, random_gains=True, n_seqs=2, max_tokens=200, max_nodes=16)
    w = gpu_verifier(SHAPE, random_gains=True, n_seqs=3, max_tokens=300, max_nodes=16)
    ctx = synth.context_tokens(SHAPE.vocab, 90, stream=61)
    chain = synth.context_tokens(SHAPE.vocab, 6, stream=62)
    tree = synth.random_tree(9, stream=63, max_children=3)
    tree_tok = synth.context_tokens(SHAPE.vocab, 9, stream=64)
    for sq in (0, 1):
        v.prefill(sq, ctx[: 40 + 20 * sq])
    for _ in range(3):  # capture, then replay, both step shapes on both sequences
        for sq in (0, 1):
            v.verify(sq, chain)
            v.verify(sq, tree_tok, tree)
    n_pages = 3 * ((300 + 15) // 16)
    perm = np.random.default_rng(65).permutation(n_pages).astype(np.int32)
    old = v.bind_kv(3, 300, perm)
    old.fill_(0x7F)
    torch.cuda.synchronize()
    results = {}
    for name, x in (("rebound", v), ("fresh", w)):
        out = []
        for sq in (2, 1):
            x.prefill(sq, ctx[: 50 + 20 * sq])
            out.append((x.verify(sq, chain), x.logits(6)))
            out.append((x.verify(sq, tree_tok, tree, commit=True), x.logits(9)))
            out.append((x.verify(sq, chain), x.logits(6)))
        results[name] = out
    for (da, la), (db, lb) in zip(results["rebound"], results["fresh"]):
        assert da == db
        np.testing.assert_array_equal(la, lb)
    assert v.length(1) == w.length(1) and v.length(2) == w.length(2)
    assert bool((old == 0x7F).all()), "a step wrote into the KV pool of the previous binding"
    v.check_kv()
    w.check_kv()
    v.close()
    w.close()


def test_logits_device_copy_and_split_report(pair):
    """tss_get_logits_device gives the host copy's values; the attention split
    report names one workgroup per head at a short context and no item when
    every block is skipped."""
    v, m = pair
    mask = synth.mask_from_layers(L, [2])
    ctx = synth.context_tokens(SHAPE.vocab, 30, stream=66)
    o = _fresh(v, m, 2, mask, ctx)
    tok = synth.context_tokens(SHAPE.vocab, 6, stream=67)
    v.verify(2, tok)
    host = v.logits(6)
    dev = v.logits_device(6)
    np.testing.assert_array_equal(dev.cpu().numpy(), host)
    assert v.attn_split() == [(1, 6)]
    v.verify(2, tok, mask=np.ones(L, np.uint8))
    assert v.attn_split() == []
    res = verify(m, o, tok, mask=np.ones(L, np.uint8))
    assert float(np.max(np.abs(v.logits(6) - res.logits))) <= 1e-4


def test_context_past_the_argument_pages():
    """A single sequence whose context outgrows the page ids passed in the kernel arguments (4500 tokens:
    282 pages, 256 of them in the arguments): the pages past the list come from the page table, read once
    per wave before its walk.  Chain and tree steps against the oracle, and a committing step followed by
    another verify."""
    from tests.gpu_common import prefill_chunked
    n = 4500
    v = gpu_verifier(SHAPE, random_gains=True, n_seqs=1, max_tokens=n + 80, max_nodes=64)
    m = oracle_model(SHAPE, random_gains=True)
    try:
        mask = synth.mask_from_layers(L, [1])
        toks = synth.context_tokens(SHAPE.vocab, n + 20, stream=61)
        v.set_mask(0, mask)
        v.prefill(0, toks[:n])
        o = OracleSequence(m, mask)
        prefill_chunked(m, o, toks[:n])
        tok = np.concatenate([[toks[n]], synth.context_tokens(SHAPE.vocab, 5, stream=62)])
        _, _, err, _ = compare_step(SHAPE, v, 0, m, o, tok)
        log(f"{n}-token context, chain: logits err {err:.2e}")
        parent = synth.random_tree(16, stream=63)
        tok = np.concatenate([[toks[n]], synth.context_tokens(SHAPE.vocab, 15, stream=64)])
        _, _, err, _ = compare_step(SHAPE, v, 0, m, o, tok, parent)
        log(f"{n}-token context, 16-node tree: logits err {err:.2e}")
        tok = np.concatenate([[toks[n]], synth.context_tokens(SHAPE.vocab, 5, stream=65)])
        res, (al, nt), err, _ = compare_step(SHAPE, v, 0, m, o, tok, commit=True)
        assert v.length(0) == o.n_kv == n + al + 1
        tok = np.concatenate([[nt], synth.context_tokens(SHAPE.vocab, 5, stream=66)])
        _, _, err2, _ = compare_step(SHAPE, v, 0, m, o, tok)
        log(f"after a commit (n_kv {o.n_kv}): logits err {err:.2e} / {err2:.2e}")
    finally:
        v.close()
