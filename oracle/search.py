"""Oracle of the offline skip-set search: the Acceptance- and Metric-Aware
Breadth Search (Algorithm 1 and the section that explains it), written as the
algorithm's steps in the paper's order and notation.

TEST INFRASTRUCTURE ONLY (see the package docstring): the product's search
driver is checked against this function on seeded evaluation tables.

The evaluation E(S) -> (A_d(S), M_d(S), C_d(S)) is passed in: acceptance,
downstream metric and verification cost of skip set S on the calibration set
(Problem Formulation).  Layers are numbered 0 .. L-1 here (the paper counts
from 1).  Readings where the paper leaves room:

* The single-layer skips are evaluated in the candidate-pool loop and again
  as the depth-1 configurations; E is deterministic, so both give one value.
  This function calls E as often as the algorithm says (a memoising caller
  evaluates each set once).
* The depth-k configurations are every k-subset of the pool, in increasing
  lexicographic order of their sorted layers (the order does not change the
  result).
* "Dominated in both acceptance and downstream metric": S leaves the Pareto
  set when another entry has A >= A(S) and M >= M(S) with at least one of the
  two strictly greater; cost plays no part (as the sentence says).  Entries
  with equal (A, M) all stay.
* argmin C runs over the union of the feasible sets of every depth, the empty
  set included (the dense verifier is feasible by definition); ties go to the
  configuration met first (empty set, then depth by depth in enumeration
  order).
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass, field


@dataclass
class SearchOutcome:
    best: frozenset                       # S_d^*
    pareto: list                          # [(S, A, M, C)] after removing dominated entries
    feasible: list                        # F_d: every feasible S, empty set first, depth by depth
    pool: list                            # L_d, increasing layer order
    evaluations: int                      # calls of E
    depth_reached: int                    # last depth whose feasible set was non-empty (0: none)
    per_depth: list = field(default_factory=list)  # |F_d^(k)| for each depth evaluated


def breadth_search(n_layers, K, evaluate, eps_A, eps_M, tau_A, tau_M):
    """Algorithm 1.  evaluate(frozenset) -> (A, M, C); thresholds absolute."""
    calls = 0

    def E(S):
        nonlocal calls
        calls += 1
        A, M, C = evaluate(frozenset(S))
        return float(A), float(M), float(C)

    # dense baseline
    A0, M0, C0 = E(())
    # candidate pool: the permissive OR filter on single-layer skips
    pool = []
    for l in range(n_layers):
        A, M, C = E((l,))
        if A >= A0 - tau_A or M >= M0 - tau_M:
            pool.append(l)
    feasible = [frozenset()]
    pareto = [(frozenset(), A0, M0, C0)]
    costs = {frozenset(): C0}
    per_depth = []
    depth_reached = 0
    for k in range(1, K + 1):
        level = []
        for S in itertools.combinations(pool, k):
            A, M, C = E(S)
            # the strict AND feasibility on both objectives
            if A >= A0 - eps_A and M >= M0 - eps_M:
                level.append(frozenset(S))
                pareto.append((frozenset(S), A, M, C))
                costs[frozenset(S)] = C
        per_depth.append(len(level))
        if not level:
            break
        feasible.extend(level)
        depth_reached = k
    # drop entries dominated in acceptance and metric
    kept = []
    for i, (S, A, M, C) in enumerate(pareto):
        dominated = any(A2 >= A and M2 >= M and (A2 > A or M2 > M)
                        for j, (_, A2, M2, _) in enumerate(pareto) if j != i)
        if not dominated:
            kept.append((S, A, M, C))
    # the cheapest feasible configuration
    best = feasible[0]
    for S in feasible[1:]:
        if costs[S] < costs[best]:
            best = S
    return SearchOutcome(best, kept, feasible, pool, calls, depth_reached, per_depth)
