"""Oracle of the offline skip-set search (the Acceptance- and Metric-Aware
Breadth Search of the paper's search section, Algorithm 1), written from the
quantities that section defines, each as a set:

* the dense baseline (A_d^0, M_d^0, C_d^0) = E(empty set);
* the candidate pool L_d: the layers whose single-layer skip keeps acceptance
  within tau_A OR the metric within tau_M of the baseline (the permissive
  filter);
* the feasible configurations of depth k, F_d^(k): the k-subsets of L_d whose
  acceptance is within eps_A AND whose metric is within eps_M of the baseline;
* the stop rule: depths are explored in increasing k up to K, and the search
  ends at the first depth whose F_d^(k) is empty (skipping is not additive,
  so a deeper feasible set is never reached past an empty depth);
* the Pareto set P_d: the baseline and every feasible configuration of the
  explored depths, minus those another entry dominates in both acceptance and
  metric;
* the selection S_d^* = argmin C over the same configurations.

TEST INFRASTRUCTURE ONLY (see the package docstring): the product's search
driver is checked against this function on seeded evaluation tables.

The evaluation E(S) -> (A_d(S), M_d(S), C_d(S)) is passed in: acceptance,
downstream metric and verification cost of skip set S on the calibration set
(Problem Formulation).  Layers are numbered 0 .. L-1 here (the paper counts
from 1).  Readings where the paper leaves room:

* `evaluations` counts what the algorithm evaluates: the baseline, the L
  single-layer skips of the pool filter, and every k-subset of the pool at
  each explored depth (the empty depth that stops the search included).  The
  depth-1 subsets are single-layer skips again; E is deterministic, so both
  evaluations give one value, but both are counted.
* F_d^(k) lists its sets in increasing lexicographic order of their sorted
  layers (the order does not change the result, only which set is "first"
  among equal costs).
* "Dominated in both acceptance and downstream metric": S leaves the Pareto
  set when another entry has A >= A(S) and M >= M(S) with at least one of the
  two strictly greater; cost plays no part.  Entries with equal (A, M) all
  stay.
* argmin C runs over the baseline and every feasible configuration (the
  dense verifier is feasible by definition); ties go to the configuration met
  first (the baseline, then depth by depth).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from itertools import combinations
from math import comb


@dataclass
class SearchOutcome:
    best: frozenset                       # S_d^*
    pareto: list                          # P_d as [(S, A, M, C)]
    feasible: list                        # the baseline, then F_d^(1), F_d^(2), ... of the explored depths
    pool: list                            # L_d, increasing layer order
    evaluations: int                      # evaluations the algorithm makes
    depth_reached: int                    # deepest depth with a non-empty F_d^(k) (0: none)
    per_depth: list = field(default_factory=list)  # |F_d^(k)| of each explored depth


def breadth_search(n_layers, K, evaluate, eps_A, eps_M, tau_A, tau_M):
    """S_d^* and the sets around it.  evaluate(frozenset) -> (A, M, C); thresholds absolute."""
    known = {}

    def E(S):
        S = frozenset(S)
        if S not in known:
            A, M, C = evaluate(S)
            known[S] = (float(A), float(M), float(C))
        return known[S]

    A0, M0, _ = E(())
    L_d = sorted({l for l in range(n_layers)
                  if E((l,))[0] >= A0 - tau_A or E((l,))[1] >= M0 - tau_M})

    def F(k):
        """F_d^(k): the k-subsets of the pool meeting both tolerances."""
        return [frozenset(S) for S in combinations(L_d, k)
                if E(S)[0] >= A0 - eps_A and E(S)[1] >= M0 - eps_M]

    # explored depths: 1 .. K, up to and including the first empty F_d^(k)
    levels = []
    for k in range(1, K + 1):
        levels.append(F(k))
        if not levels[-1]:
            break
    reached = [Fk for Fk in levels if Fk]          # every explored depth before the empty one
    configs = [frozenset()] + [S for Fk in reached for S in Fk]

    def dominated(S):
        A, M, _ = E(S)
        return any(E(T)[0] >= A and E(T)[1] >= M and (E(T)[0] > A or E(T)[1] > M) for T in configs if T != S)

    pareto = [(S, *E(S)) for S in configs if not dominated(S)]
    best = min(configs, key=lambda S: E(S)[2])      # min keeps the first of equal costs
    evaluations = 1 + n_layers + sum(comb(len(L_d), k) for k in range(1, len(levels) + 1))
    return SearchOutcome(best, pareto, configs, L_d, evaluations, len(reached), [len(Fk) for Fk in levels])
