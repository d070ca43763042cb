"""Evidence that the oracle pins are sharp: plant a plausible mistake in the
oracle (on the CPU, through monkeypatching) and check that the pins fail.

Each planted mistake is one a hand-written LLaMA verifier commonly makes: a
rotary sign flip, a dropped norm gain, epsilon added in the wrong place, the
tree mask leaking sibling nodes, tree positions taken from the node index, an
accept scan that ignores the parent, the bonus token read from the wrong node
and the skip mask applied to the wrong layer.
"""
import numpy as np
import pytest

import oracle.forward as ov
from tests import test_oracle_pins as pins


def _fails(fn, *args):
    try:
        fn(*args)
    except AssertionError:
        return True
    return False


@pytest.fixture(scope="module")
def env():
    get = pins._getter()
    return get, pins.llama_ref.build(pins.SHAPE, get)


def _model64(get):
    return ov.OracleModel(pins.SHAPE, get, dtype=np.float64)


def test_rope_sign_flip_is_caught(env, monkeypatch):
    get, hf = env
    real = ov.rope

    def bad(x, pos, base):
        return real(x, -pos, base)
    monkeypatch.setattr(ov, "rope", bad)
    assert _fails(pins.test_dense_chain_matches_independent_forward, _model64(get), hf)


def test_missing_norm_gain_is_caught(env, monkeypatch):
    get, hf = env
    real = ov.rmsnorm
    monkeypatch.setattr(ov, "rmsnorm", lambda x, g, eps: real(x, np.ones_like(g), eps))
    assert _fails(pins.test_dense_chain_matches_independent_forward, _model64(get), hf)


def test_wrong_rms_eps_placement_is_caught(env, monkeypatch):
    get, hf = env
    monkeypatch.setattr(ov, "rmsnorm", lambda x, g, eps: x / np.sqrt(np.mean(x * x, -1, keepdims=True)) * g + 1e-3)
    assert _fails(pins.test_dense_chain_matches_independent_forward, _model64(get), hf)


def test_tree_mask_leak_is_caught(env, monkeypatch):
    get, hf = env

    def leaky(parent):
        depth, vis = real(parent)
        n = len(parent)
        return depth, [set(range(i + 1)) for i in range(n)]   # causal over node ids instead of ancestors
    real = ov.tree_meta
    monkeypatch.setattr(ov, "tree_meta", leaky)
    assert _fails(pins.test_tree_nodes_match_path_chains, _model64(get), hf)


def test_tree_positions_by_index_is_caught(env, monkeypatch):
    get, hf = env
    real = ov.tree_meta

    def by_index(parent):
        _, vis = real(parent)
        return np.arange(len(parent)), vis
    monkeypatch.setattr(ov, "tree_meta", by_index)
    assert _fails(pins.test_tree_nodes_match_path_chains, _model64(get), hf)


def test_accept_scan_ignoring_parent_is_caught(monkeypatch):
    def bad(tokens, parent, greedy):
        # compares each node with the greedy token of node i-1
        n = len(tokens)
        best = 0
        for i in range(1, n):
            if int(tokens[i]) == int(greedy[i - 1]):
                best = i
            else:
                break
        return best, int(greedy[best]), best, list(range(best + 1))
    monkeypatch.setattr(ov, "accept_scan", bad)
    monkeypatch.setattr(pins, "accept_scan", bad)
    assert _fails(pins.test_accept_scan_ties_and_duplicate_siblings)


def test_bonus_from_wrong_node_is_caught(env, monkeypatch):
    get, hf = env
    real = ov.accept_scan

    def bad(tokens, parent, greedy):
        al, nt, best, path = real(tokens, parent, greedy)
        return al, int(greedy[path[-2]]) if len(path) > 1 else nt, best, path
    monkeypatch.setattr(ov, "accept_scan", bad)
    assert _fails(pins.test_self_consistent_drafts_fully_accepted, _model64(get), hf)


def test_skip_applied_to_wrong_layer_is_caught(env, monkeypatch):
    get, _ = env
    real = ov._forward

    def shifted(model, seq, tokens, parent, mask, with_logits):
        return real(model, seq, tokens, parent, np.roll(mask, 1), with_logits)
    monkeypatch.setattr(ov, "_forward", shifted)
    assert _fails(pins.test_skip_equals_deleted_block, _model64(get), get, [2])


@pytest.mark.parametrize("kind", ["distinct_runner_up", "gap_to_mean"])
def test_wrong_margin_is_caught(monkeypatch, kind):
    """A margin taken against the second-largest distinct value (a tie then
    looks decided) or against the row mean fails the closed-form margin pin."""
    real = pins.verify

    def bad(*args, **kw):
        res = real(*args, **kw)
        lg = res.logits
        if kind == "distinct_runner_up":
            res.margin = np.array([np.unique(r)[-1] - np.unique(r)[-2] for r in lg])
        else:
            res.margin = lg.max(axis=-1) - lg.mean(axis=-1)
        return res
    monkeypatch.setattr(pins, "verify", bad)
    assert _fails(pins.test_margin_closed_form)
