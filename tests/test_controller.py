"""Host logic of the domain controller: the configuration map (JSON round
trip, dense fallback for unknown domains, R_d = |S| / L), admission of
requests on a verifier, and the batch planner's cost on cases worked by hand
and against exhaustive search on small instances."""
import itertools
import json

import numpy as np
import pytest

from paper_2609_26100_amd.controller import (ConfigMap, DomainConfig, SkipController, launched_blocks,
                                              plan_batches, plan_cost)
from paper_2609_26100_amd.search import breadth_search
from tests.test_search_pins import WORKED, _t, table_eval


def test_map_round_trip_and_fallback(tmp_path):
    phi = ConfigMap(32, {"translation": {"skip": [30, 17, 25]}, "qa": DomainConfig([20], 3.1, 0.7)})
    assert phi.domains["translation"].skip == [17, 25, 30]
    assert phi.domains["translation"].ratio == 3 / 32
    p = tmp_path / "phi.json"
    phi.save(p)
    doc = json.loads(p.read_text())
    assert doc["n_layers"] == 32 and set(doc["domains"]) == {"translation", "qa"}
    back = ConfigMap.load(p)
    assert back.skip_set("translation") == (17, 25, 30)
    assert back.domains["qa"].accept == 3.1 and back.domains["qa"].ratio == 1 / 32
    assert back.skip_set("unseen") == () and not back.mask("unseen").any()
    assert back.mask(None).sum() == 0
    m = back.mask("translation")
    assert m.dtype == np.uint8 and m.sum() == 3 and m[[17, 25, 30]].all()


def test_map_rejects_bad_skip_sets():
    with pytest.raises(ValueError):
        ConfigMap(8, {"x": {"skip": [8]}})
    with pytest.raises(ValueError):
        ConfigMap(8, {"x": {"skip": [1, 1]}})


class _Rec:
    """Stands in for a Verifier: records the masks set on sequences."""
    class shape:
        n_layers = 5

    def __init__(self):
        self.masks = {}

    def set_mask(self, seq, mask):
        self.masks[seq] = np.asarray(mask).copy()


def test_search_result_into_map_and_controller():
    res = breadth_search(5, 3, _Quality(), _Cost(), eps_A=0.2, eps_M=0.05, tau_A=0.3, tau_M=0.02)
    phi = ConfigMap(5)
    phi.add_search_result("legal", res)
    g = phi.domains["legal"]
    assert g.skip == [0, 3] and g.accept == 2.85 and g.metric == 0.8 and g.ratio == 0.4
    assert [a["skip"] for a in g.alternatives] == [[], [4]]
    v = _Rec()
    ctl = SkipController(v, phi)
    assert ctl.admit(3, "legal").tolist() == [1, 0, 0, 1, 0]
    assert ctl.admit(4, "poetry").tolist() == [0] * 5       # unknown domain: dense
    assert v.masks[3].tolist() == [1, 0, 0, 1, 0] and not v.masks[4].any()
    assert ctl.plan([3, 4], 8) == [[3, 4]]


class _Quality:
    def __call__(self, sets):
        t = table_eval(_t(WORKED))
        v = [t(S) for S in sets]
        return np.array([x[0] for x in v]), np.array([x[1] for x in v])


class _Cost:
    def __call__(self, sets):
        t = table_eval(_t(WORKED))
        return np.array([t(S)[2] for S in sets])


L = 32
A = tuple(range(24, 32))       # domain A skips 8 late layers
B = tuple(range(16, 24))       # domain B skips 8 others


def test_full_domain_groups_get_pure_batches():
    # arrival order interleaves the domains
    skip_of = {s: (A if s % 2 == 0 else B) for s in range(16)}
    plan = plan_batches(skip_of, L, 8)
    assert sorted(map(sorted, plan)) == [list(range(0, 16, 2)), list(range(1, 16, 2))]
    assert plan_cost(plan, skip_of, L) == 24 + 24
    naive = [list(range(0, 8)), list(range(8, 16))]        # arrival order
    assert plan_cost(naive, skip_of, L) == 32 + 32


def test_leftovers_share_a_batch():
    skip_of = {0: A, 1: A, 2: B, 3: B, 4: ()}
    plan = plan_batches(skip_of, L, 8)
    assert [sorted(b) for b in plan] == [[0, 1, 2, 3, 4]]        # one step of 32 blocks beats three steps
    assert plan_cost(plan, skip_of, L) == 32


def test_batches_respect_the_size_limit_and_cover_every_sequence():
    rng = np.random.default_rng(0)
    for trial in range(50):
        n = int(rng.integers(1, 30))
        pool = [tuple(sorted(rng.choice(L, size=int(rng.integers(0, 9)), replace=False))) for _ in range(4)]
        skip_of = {s: pool[int(rng.integers(0, 4))] for s in range(n)}
        B = int(rng.integers(1, 9))
        plan = plan_batches(skip_of, L, B)
        assert sorted(s for b in plan for s in b) == list(range(n))
        assert all(1 <= len(b) <= B for b in plan)


def _optimum(skip_of, n_layers, B):
    """Exhaustive minimum of the plan cost (set partitions into blocks of <= B)."""
    seqs = sorted(skip_of)
    best = None

    def rec(i, parts):
        nonlocal best
        if i == len(seqs):
            c = plan_cost(parts, skip_of, n_layers)
            best = c if best is None else min(best, c)
            return
        for p in parts:
            if len(p) < B:
                p.append(seqs[i])
                rec(i + 1, parts)
                p.pop()
        parts.append([seqs[i]])
        rec(i + 1, parts)
        parts.pop()
    rec(0, [])
    return best


@pytest.mark.parametrize("seed", range(8))
def test_plan_cost_close_to_exhaustive_optimum(seed):
    """Small instances (6 sequences, 12 layers, 3 domains): the plan is never
    worse than arrival order in chunks, and within 1.5x of the optimum."""
    rng = np.random.default_rng(seed)
    nl = 12
    doms = [tuple(sorted(rng.choice(nl, size=int(rng.integers(1, 6)), replace=False))) for _ in range(3)]
    skip_of = {s: doms[int(rng.integers(0, 3))] for s in range(6)}
    B = int(rng.integers(2, 4))
    plan = plan_batches(skip_of, nl, B)
    cost = plan_cost(plan, skip_of, nl)
    naive = plan_cost([list(range(i, min(6, i + B))) for i in range(0, 6, B)], skip_of, nl)
    opt = _optimum(skip_of, nl, B)
    assert opt <= cost <= naive
    assert cost <= 1.5 * opt
