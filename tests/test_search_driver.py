"""The product search driver (batched, memoised Algorithm 1) against the
search oracle on seeded evaluation tables: same pool, feasible sets, Pareto
set and selection; each skip set evaluated once; quality asked once per
depth; cost asked only for the baseline and the feasible sets."""
import itertools

import numpy as np
import pytest

from oracle.search import breadth_search as oracle_search
from paper_2609_26100_amd.search import breadth_search
from tests.test_search_pins import WORKED, _t, table_eval


class Table:
    """A deterministic evaluation table shared by both sides, counting calls."""

    def __init__(self, fn):
        self.fn = fn
        self.quality_calls = 0
        self.quality_sets = 0
        self.cost_sets = []

    def E(self, S):
        return self.fn(frozenset(S))

    def quality(self, sets):
        self.quality_calls += 1
        self.quality_sets += len(sets)
        v = [self.fn(frozenset(S)) for S in sets]
        return np.array([x[0] for x in v]), np.array([x[1] for x in v])

    def cost(self, sets):
        self.cost_sets.extend(sets)
        return np.array([self.fn(frozenset(S))[2] for S in sets])


def random_table(seed, L):
    """Acceptance and metric fall with each skipped layer by a per-layer
    amount plus an interaction term; cost falls per skipped layer."""
    rng = np.random.default_rng(seed)
    dA = rng.uniform(-0.05, 0.25, L)
    dM = rng.uniform(-0.01, 0.04, L)
    dC = rng.uniform(0.5, 1.5, L)
    cache = {}

    def fn(S):
        if S not in cache:
            s = sorted(S)
            inter = rng.normal(0, 0.05) if len(s) > 1 else 0.0
            cache[S] = (3.0 - dA[s].sum() + inter, 0.8 - dM[s].sum() + inter / 5, 20.0 - dC[s].sum())
        return cache[S]
    return fn


def _same(out, res):
    assert res.pool == out.pool
    assert res.feasible == [tuple(sorted(S)) for S in out.feasible]
    assert res.best == tuple(sorted(out.best))
    assert [e.skip for e in res.pareto] == [tuple(sorted(p[0])) for p in out.pareto]
    assert [(e.A, e.M, e.C) for e in res.pareto] == [p[1:] for p in out.pareto]
    assert res.per_depth == out.per_depth and res.depth_reached == out.depth_reached


def test_worked_case_matches_oracle():
    t = Table(table_eval(_t(WORKED)))
    args = dict(eps_A=0.2, eps_M=0.05, tau_A=0.3, tau_M=0.02)
    out = oracle_search(5, 3, t.E, **args)
    res = breadth_search(5, 3, t.quality, t.cost, **args)
    _same(out, res)
    # each set once: dense, 5 singles, 6 pairs, 4 triples (the oracle asks 20 times)
    assert res.evaluations == 16
    assert t.quality_calls == 1 + 1 + 2     # dense, singles, depth 2, depth 3 (depth 1 is memoised)
    assert sorted(t.cost_sets) == sorted([(), (3,), (4,), (0, 3), (3, 4)])
    assert res.config(5) == {"skip": [0, 3], "accept": 2.85, "metric": 0.8, "ratio": 0.4, "cost_ms": 6.0}


@pytest.mark.parametrize("seed", range(12))
def test_random_tables_match_oracle(seed):
    L = 8
    fn = random_table(seed, L)
    rng = np.random.default_rng(100 + seed)
    args = dict(eps_A=float(rng.uniform(0.1, 0.6)), eps_M=float(rng.uniform(0.02, 0.1)),
                tau_A=float(rng.uniform(0.0, 0.2)), tau_M=float(rng.uniform(0.0, 0.03)))
    K = int(rng.integers(1, 5))
    t = Table(fn)
    out = oracle_search(L, K, t.E, **args)
    res = breadth_search(L, K, t.quality, t.cost, **args)
    _same(out, res)
    distinct = {frozenset()} | {frozenset((l,)) for l in range(L)}
    for k in range(1, len(out.per_depth) + 1):
        distinct |= {frozenset(S) for S in itertools.combinations(out.pool, k)}
    assert res.evaluations == len(distinct)
    assert len(t.cost_sets) == len(set(t.cost_sets)) == len(res.feasible)


def test_relative_tolerances_equal_absolute_ones():
    L = 7
    fn = random_table(3, L)
    A0, M0, _ = fn(frozenset())
    t = Table(fn)
    rel = breadth_search(L, 3, t.quality, t.cost, eps_A=0.05, eps_M=0.05, tau_A=0.02, tau_M=0.02, relative=True)
    out = oracle_search(L, 3, Table(fn).E, eps_A=0.05 * A0, eps_M=0.05 * M0, tau_A=0.02 * A0, tau_M=0.02 * M0)
    _same(out, rel)


def test_candidate_layers_restrict_the_pool():
    L = 8
    fn = random_table(5, L)
    t = Table(fn)
    res = breadth_search(L, 2, t.quality, t.cost, eps_A=1.0, eps_M=1.0, tau_A=1.0, tau_M=1.0, layers=[6, 2, 7])
    assert res.pool == [2, 6, 7]
    assert all(set(S) <= {2, 6, 7} for S in res.feasible)


# ------------------------------------------------------------ the beam variant

from paper_2609_26100_amd.search import beam_search  # noqa: E402


def test_beam_worked_case():
    """6 layers, barriers 2 / 0 (candidates 5, 4, 3, 2), beam 2.  Dense A 3.0,
    M 0.80, C 10.  Depth 1 keeps {5} (3.2), {4} (3.0), {3} (3.1), {2} fails
    A; beam {5}, {3}.  Depth 2 children of {5}: {4,5}, {3,5}, {2,5}; of {3}:
    {3,4}, {2,3}: kept {3,5} (3.4), {4,5} (3.0; M 0.77 is within 5 %); beam
    {3,5}, {4,5}.  Depth 3: {3,4,5} fails M, {2,3,5} fails A, {2,4,5} fails A:
    stop.  Triple wins (M >= 0.80, A >= 3.0, A/C >= 0.3): {5}, {3}, {4},
    {3,5}; {4,5} has M 0.77.  Largest kept set 2, so sets of >= 2 skips are
    preferred: {3,5}."""
    T = {(): (3.0, 0.80, 10.0), (5,): (3.2, 0.80, 9.0), (3,): (3.1, 0.81, 9.0), (4,): (3.0, 0.85, 9.0),
         (2,): (2.9, 0.90, 9.0), (0,): (9.0, 0.90, 1.0), (1,): (9.0, 0.90, 1.0),
         (4, 5): (3.0, 0.77, 8.0), (3, 5): (3.4, 0.80, 8.0), (2, 5): (2.0, 0.80, 8.0), (3, 4): (2.5, 0.80, 8.0),
         (2, 3): (2.5, 0.80, 8.0), (3, 4, 5): (3.5, 0.70, 7.0), (2, 3, 5): (2.0, 0.80, 7.0),
         (2, 4, 5): (2.0, 0.80, 7.0)}
    t = Table(table_eval(_t(T)))
    res = beam_search(6, t.quality, t.cost, beam_width=2, early_barrier=2, latter_barrier=0, score_tol=0.05)
    assert res.pool == [5, 4, 3, 2]
    assert res.per_depth == [3, 2, 0]
    assert res.feasible == [(5,), (4,), (3,), (4, 5), (3, 5)]     # in the order met
    assert res.best == (3, 5)
    assert [e.skip for e in res.pareto] == [(3, 5), ]
    assert all(0 not in S and 1 not in S for S in res.entries)   # the early barrier is never skipped
    assert res.evaluations == 1 + 4 + 5 + 3


def test_beam_without_a_triple_win_returns_dense():
    T = {(): (3.0, 0.80, 10.0), (3,): (3.0, 0.79, 10.5)}     # kept (within 5 %) but neither M nor tok/s wins
    t = Table(table_eval(_t(T)))
    res = beam_search(4, t.quality, t.cost)
    assert res.feasible == [(3,)] and res.best == () and res.pareto == []
