"""Pins of the search oracle (Algorithm 1): hand-worked cases whose answers
follow from the algorithm's text, not from the code under test.

Case W (worked by hand, 5 layers, K = 3; thresholds tau_A = 0.3, tau_M = 0.02,
eps_A = 0.2, eps_M = 0.05):

  dense: A 3.00  M 0.80  C 10.0
  single skips        A     M     OR filter (A >= 2.7 or M >= 0.78)
    {0}             2.00  0.80    in  (metric only: the permissive OR)
    {1}             3.10  0.70    in  (acceptance only)
    {2}             2.50  0.60    out
    {3}             2.95  0.79    in
    {4}             2.90  0.81    in
  pool L = [0, 1, 3, 4]
  depth 1 (AND: A >= 2.8 and M >= 0.75): {3} C 8.0 and {4} C 8.2 feasible;
    {0} fails A, {1} fails M
  depth 2: {0,3} (2.85, 0.80, C 6.0) and {3,4} (2.85, 0.77, C 6.1) feasible
    ({0} alone was not: the OR pool keeps it for combinations);
    {1,4} (3.20, 0.74) fails M; the rest use the default (1.0, 0.5, C 5.0)
  depth 3: nothing feasible -> stop
  evaluations: 1 + 5 + 4 + 6 + 4 = 20
  best = argmin C over {{}, {3}, {4}, {0,3}, {3,4}} = {0,3} (6.0)
  Pareto (dominance in A and M only): {} (3.00, 0.80) dominates {3},
    {0,3} and {3,4}; {4} has the highest M and stays -> [{}, {4}]
"""
import itertools

import numpy as np
import pytest

from oracle.search import breadth_search

DEFAULT = (1.0, 0.5, 5.0)


def table_eval(table, default=DEFAULT):
    def E(S):
        return table.get(frozenset(S), default)
    return E


WORKED = {
    (): (3.0, 0.80, 10.0),
    (0,): (2.0, 0.80, 9.0), (1,): (3.1, 0.70, 9.0), (2,): (2.5, 0.60, 9.0),
    (3,): (2.95, 0.79, 8.0), (4,): (2.9, 0.81, 8.2),
    (0, 3): (2.85, 0.80, 6.0), (3, 4): (2.85, 0.77, 6.1), (1, 4): (3.2, 0.74, 5.5),
}


def _t(d):
    return {frozenset(k): v for k, v in d.items()}


def test_worked_case():
    out = breadth_search(5, 3, table_eval(_t(WORKED)), eps_A=0.2, eps_M=0.05, tau_A=0.3, tau_M=0.02)
    assert out.pool == [0, 1, 3, 4]
    assert out.feasible == [frozenset(), frozenset({3}), frozenset({4}), frozenset({0, 3}), frozenset({3, 4})]
    assert out.per_depth == [2, 2, 0]
    assert out.depth_reached == 2
    assert out.evaluations == 20
    assert out.best == frozenset({0, 3})
    assert [p[0] for p in out.pareto] == [frozenset(), frozenset({4})]


def test_stops_at_first_empty_depth_even_if_deeper_sets_qualify():
    """Skipping is not additive: {0,1,2} is feasible here, but depth 2 has no
    feasible set, so the search never reaches depth 3."""
    t = _t({(): (3.0, 0.8, 10.0), (0,): (3.0, 0.8, 9.0), (1,): (3.0, 0.8, 9.0), (2,): (3.0, 0.8, 9.0),
            (0, 1, 2): (3.0, 0.8, 1.0)})
    # depth 2 subsets fall to the default (infeasible)
    out = breadth_search(3, 3, table_eval(t), eps_A=0.1, eps_M=0.1, tau_A=0.1, tau_M=0.1)
    assert out.depth_reached == 1
    assert out.per_depth == [3, 0]
    assert frozenset({0, 1, 2}) not in out.feasible
    assert out.best in (frozenset({0}), frozenset({1}), frozenset({2}))
    assert out.best == frozenset({0})            # equal costs: the first met
    assert out.evaluations == 1 + 3 + 3 + 3


def test_empty_pool_returns_dense():
    t = _t({(): (3.0, 0.8, 10.0)})               # every skip gets the default (1.0, 0.5)
    out = breadth_search(6, 4, table_eval(t), eps_A=0.1, eps_M=0.1, tau_A=0.1, tau_M=0.1)
    assert out.pool == []
    assert out.best == frozenset()
    assert out.feasible == [frozenset()]
    assert out.evaluations == 1 + 6
    assert out.per_depth == [0]
    assert [p[0] for p in out.pareto] == [frozenset()]


def test_depth_cap_K():
    """Every set feasible and cheaper with more skips: K bounds the depth."""
    def E(S):
        return (3.0, 0.8, 10.0 - len(S))
    out = breadth_search(4, 2, E, eps_A=0.0, eps_M=0.0, tau_A=0.0, tau_M=0.0)
    assert out.depth_reached == 2
    assert len(out.feasible) == 1 + 4 + 6
    assert out.best == frozenset({0, 1})         # cost 8, first among the six pairs
    assert out.evaluations == 1 + 4 + 4 + 6


def test_pareto_keeps_ties_and_incomparable_entries():
    t = _t({(): (3.0, 0.80, 10.0), (0,): (3.0, 0.80, 9.0), (1,): (3.2, 0.70, 9.0), (2,): (2.9, 0.90, 9.0),
            (3,): (2.9, 0.70, 9.0)})
    out = breadth_search(4, 1, table_eval(t), eps_A=1.0, eps_M=1.0, tau_A=1.0, tau_M=1.0)
    names = [p[0] for p in out.pareto]
    # {} and {0} tie in (A, M): both stay; {1} and {2} are incomparable with them; {3} is dominated by {}
    assert names == [frozenset(), frozenset({0}), frozenset({1}), frozenset({2})]
    assert out.best == frozenset({0})


def test_thresholds_are_inclusive():
    t = _t({(): (3.0, 0.8, 10.0), (0,): (2.7, 0.75, 9.0)})
    out = breadth_search(1, 1, table_eval(t), eps_A=0.3, eps_M=0.05, tau_A=0.3, tau_M=0.05)
    assert out.pool == [0] and out.best == frozenset({0})
    out = breadth_search(1, 1, table_eval(t), eps_A=0.29, eps_M=0.05, tau_A=0.3, tau_M=0.05)
    assert out.pool == [0] and out.best == frozenset()


@pytest.mark.parametrize("seed", range(5))
def test_feasible_sets_obey_both_bounds_and_subsets_of_pool(seed):
    """Invariants on random tables: every feasible set lies in the pool,
    meets both bounds, depths are contiguous, and the best is the cheapest of
    them."""
    rng = np.random.default_rng(seed)
    L, K = 6, 3
    cache = {}

    def E(S):
        if S not in cache:
            cache[S] = (3.0 - 0.1 * len(S) + rng.normal(0, 0.1), 0.8 - 0.02 * len(S) + rng.normal(0, 0.02),
                        10.0 - len(S) + rng.normal(0, 0.3))
        return cache[S]
    E(frozenset())
    out = breadth_search(L, K, E, eps_A=0.25, eps_M=0.05, tau_A=0.1, tau_M=0.01)
    A0, M0, _ = cache[frozenset()]
    depths = sorted({len(S) for S in out.feasible})
    assert depths == list(range(len(depths)))
    for S in out.feasible[1:]:
        assert S <= set(out.pool)
        A, M, _ = cache[S]
        assert A >= A0 - 0.25 and M >= M0 - 0.05
    assert cache[out.best][2] == min(cache[S][2] for S in out.feasible)
    for S, A, M, _ in out.pareto:
        assert not any(A2 >= A and M2 >= M and (A2 > A or M2 > M) for _, A2, M2, _ in out.pareto)
