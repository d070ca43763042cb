"""Offline skip-set search: the Acceptance- and Metric-Aware Breadth Search
(Algorithm 1), driven by batched evaluations on the GPU.

The search itself is host logic: dense baseline, every single-layer skip, a
candidate pool kept by the permissive OR filter, then depth by depth every
subset of the pool of that size, kept by the strict AND feasibility test,
stopping at the first depth with nothing feasible; dominated entries leave
the Pareto set and the cheapest feasible configuration is selected.  What
differs from a literal loop is only how evaluations are issued:

* quality (A_d, M_d) is asked for a whole depth at once, so a GPU evaluator
  can verify all of that depth's masks in a few shared sweep steps
  (tss_verify_sweep);
* every skip set is evaluated once (the single-layer skips of the pool filter
  are the depth-1 sets);
* the cost C_d is only measured for the dense baseline and the feasible sets,
  the only ones whose cost the algorithm reads (the argmin and the Pareto
  entries).

Tolerances are absolute, as in the algorithm, or relative to the dense
baseline (relative=True; the paper's tolerance study quotes -5 %).
Dominance is taken in acceptance and metric only, as the search section
states; entries with equal (A, M) all stay.
"""
from __future__ import annotations

import itertools
import time
from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Entry:
    skip: tuple    # skipped layers, increasing
    A: float       # acceptance (mean tokens per verify step on the calibration set)
    M: float       # downstream metric
    C: float       # verification cost (ms per verify step)


@dataclass
class SearchResult:
    best: tuple                  # S_d^*
    baseline: Entry              # the dense verifier
    pareto: list                 # [Entry], non-dominated in (A, M)
    feasible: list               # [tuple]: the empty set, then each depth's feasible sets
    pool: list                   # candidate layers L_d
    per_depth: list              # |F_d^(k)| for each depth evaluated
    depth_reached: int
    evaluations: int             # distinct skip sets whose quality was evaluated
    cost_evaluations: int
    entries: dict = field(default_factory=dict)  # skip -> (A, M) of every evaluated set
    costs: dict = field(default_factory=dict)    # skip -> C of every costed set
    seconds: float = 0.0

    def config(self, n_layers):
        """The configuration record G_d = (S_d^*, A_d(S_d^*), M_d(S_d^*), R_d) of
        the Domain-to-Configuration Mapping, R_d = |S_d^*| / L."""
        A, M = self.entries[self.best]
        return {"skip": list(self.best), "accept": A, "metric": M, "ratio": len(self.best) / n_layers,
                "cost_ms": self.costs.get(self.best)}


def _dominated(A, M):
    """dominated[i]: some j has A_j >= A_i and M_j >= M_i, one of them strictly."""
    A = np.asarray(A, float)
    M = np.asarray(M, float)
    ge = (A[:, None] >= A[None, :]) & (M[:, None] >= M[None, :])
    gt = (A[:, None] > A[None, :]) | (M[:, None] > M[None, :])
    return (ge & gt).any(axis=0)


def breadth_search(n_layers, max_depth, quality, cost, eps_A, eps_M, tau_A, tau_M, relative=False,
                   layers=None, log=None):
    """Algorithm 1.

    quality(list of skip tuples) -> (A, M) arrays; cost(list of skip tuples)
    -> C array.  layers: candidate layers (default all); relative: tolerances
    are fractions of the dense values.  log(str) receives progress lines.
    """
    t0 = time.perf_counter()
    entries, costs = {}, {}

    def q(sets):
        todo = [S for S in sets if S not in entries]
        if todo:
            A, M = quality(todo)
            for S, a, m in zip(todo, A, M):
                entries[S] = (float(a), float(m))
        return [entries[S] for S in sets]

    def c(sets):
        todo = [S for S in sets if S not in costs]
        if todo:
            for S, v in zip(todo, cost(todo)):
                costs[S] = float(v)
        return [costs[S] for S in sets]

    cand = list(range(n_layers)) if layers is None else sorted(int(l) for l in layers)
    dense = ()
    (A0, M0), = q([dense])
    (C0,) = c([dense])
    scale_A, scale_M = (abs(A0), abs(M0)) if relative else (1.0, 1.0)
    eA, eM, tA, tM = eps_A * scale_A, eps_M * scale_M, tau_A * scale_A, tau_M * scale_M
    singles = [(l,) for l in cand]
    pool = [l for (l,), (A, M) in zip(singles, q(singles)) if A >= A0 - tA or M >= M0 - tM]
    if log:
        log(f"dense A {A0:.3f} M {M0:.3f} C {C0:.3f}; pool {pool}")
    feasible = [dense]
    per_depth = []
    depth_reached = 0
    for k in range(1, max_depth + 1):
        level = list(itertools.combinations(pool, k))
        ok = [S for S, (A, M) in zip(level, q(level)) if A >= A0 - eA and M >= M0 - eM]
        per_depth.append(len(ok))
        if log:
            log(f"depth {k}: {len(level)} sets, {len(ok)} feasible")
        if not ok:
            break
        feasible.extend(ok)
        depth_reached = k
    C = c(feasible)
    A = [entries[S][0] for S in feasible]
    M = [entries[S][1] for S in feasible]
    dom = _dominated(A, M)
    pareto = [Entry(S, a, m, cc) for S, a, m, cc, d in zip(feasible, A, M, C, dom) if not d]
    best = feasible[int(np.argmin(C))]  # first minimum: the order the sets were met
    return SearchResult(best, Entry(dense, A0, M0, C0), pareto, feasible, pool, per_depth, depth_reached,
                        len(entries), len(costs), entries, costs, time.perf_counter() - t0)


def beam_search(n_layers, quality, cost, beam_width=3, early_barrier=2, latter_barrier=0, score_tol=0.05,
                min_skips=3, max_depth=None, log=None):
    """The beam-style search of the paper's hyperparameter table (Table 3), an
    alternative to Algorithm 1's exhaustive depths.  Reading of its settings:

    * candidates: layers [early_barrier, n_layers - latter_barrier), tried
      latter to early;
    * depth by depth, every beam entry grows by one candidate layer; a child
      is kept only if A >= A_dense (hard acceptance constraint) and
      M >= (1 - score_tol) M_dense (relative score tolerance);
    * the kept children are ranked by acceptance, then number of skipped
      layers, then tok/s = A / C (all descending, first met on ties) and the
      best beam_width form the next beam; the search stops when none is kept;
    * selection: among every kept configuration, the "triple wins" (metric,
      acceptance and tok/s all >= the dense verifier's), preferring those with
      at least min(min_skips, largest |S| kept) skipped layers, ranked as
      above; the dense verifier when there is none.

    Returns a SearchResult (pool = candidate layers, feasible = kept sets in
    the order met, pareto = the selection ranking of the triple wins)."""
    t0 = time.perf_counter()
    entries, costs = {}, {}

    def q(sets):
        todo = [S for S in sets if S not in entries]
        if todo:
            A, M = quality(todo)
            for S, a, m in zip(todo, A, M):
                entries[S] = (float(a), float(m))
        return [entries[S] for S in sets]

    def c(sets):
        todo = [S for S in sets if S not in costs]
        if todo:
            for S, v in zip(todo, cost(todo)):
                costs[S] = float(v)
        return [costs[S] for S in sets]

    (A0, M0), = q([()])
    (C0,) = c([()])
    tps0 = A0 / C0
    cand = list(range(n_layers - latter_barrier - 1, early_barrier - 1, -1))
    rank = lambda S: (-entries[S][0], -len(S), -entries[S][0] / costs[S])  # noqa: E731
    beam, kept, per_depth = [()], [], []
    while beam and (max_depth is None or len(per_depth) < max_depth):
        children, seen = [], set()
        for S in beam:
            for l in cand:
                if l in S:
                    continue
                ch = tuple(sorted(S + (l,)))
                if ch not in seen:
                    seen.add(ch)
                    children.append(ch)
        ok = [S for S, (A, M) in zip(children, q(children)) if A >= A0 and M >= (1 - score_tol) * M0]
        per_depth.append(len(ok))
        if log:
            log(f"beam depth {len(per_depth)}: {len(children)} children, {len(ok)} kept")
        if not ok:
            break
        c(ok)
        kept.extend(ok)
        beam = sorted(ok, key=rank)[:beam_width]
    wins = [S for S in kept if entries[S][1] >= M0 and entries[S][0] >= A0 and entries[S][0] / costs[S] >= tps0]
    need = min(min_skips, max((len(S) for S in kept), default=0))
    pref = [S for S in wins if len(S) >= need] or wins
    ranked = sorted(pref, key=rank)
    best = ranked[0] if ranked else ()
    pareto = [Entry(S, entries[S][0], entries[S][1], costs[S]) for S in ranked]
    return SearchResult(best, Entry((), A0, M0, C0), pareto, kept, cand, per_depth,
                        sum(1 for k in per_depth if k), len(entries), len(costs), entries, costs,
                        time.perf_counter() - t0)


# ---------------------------------------------------------------- GPU evaluators

class SweepQuality:
    """A_d and M_d of skip sets on a calibration set, through tss_verify_sweep.

    items: [(seq, draft_tokens, tree_parent or None)], each sequence prefilled
    dense (every layer holds the context's K/V).  A(S) = mean over the items of
    accept_len + 1 (tokens produced per verify step).  The downstream metric
    needs task data the method's calibration sets provide; in its place M(S)
    is the fraction of draft nodes whose greedy token under S equals the
    dense verifier's (how closely the sparse verifier reproduces the dense
    one's output), 1 for the dense set.
    """

    def __init__(self, verifier, items):
        self.v = verifier
        self.items = items
        self.L = verifier.shape.n_layers
        self.dense_greedy = None
        self.sweeps = 0

    def masks(self, sets):
        m = np.zeros((len(sets), self.L), np.uint8)
        for i, S in enumerate(sets):
            m[i, list(S)] = 1
        return m

    def __call__(self, sets):
        m = self.masks(sets)
        if self.dense_greedy is None:
            self.dense_greedy = [self.v.verify_sweep(seq, tok, np.zeros((1, self.L), np.uint8), par,
                                                     want_greedy=True)[2][0] for seq, tok, par in self.items]
        acc = np.zeros(len(sets))
        agree = np.zeros(len(sets))
        nodes = 0
        for (seq, tok, par), g0 in zip(self.items, self.dense_greedy):
            al, _, g = self.v.verify_sweep(seq, tok, m, par, want_greedy=True)
            self.sweeps += 1
            acc += al + 1
            agree += (g == g0[None, :]).sum(axis=1)
            nodes += len(tok)
        return acc / len(self.items), agree / nodes


class MeasuredCost:
    """C_d(S): median wall time (ms) of one blocking dry-run verify of a
    calibration item under S, in the runtime's launch mode (a captured step
    per mask), after one warm-up call."""

    def __init__(self, verifier, item, reps=5):
        self.v = verifier
        self.item = item
        self.reps = reps
        self.L = verifier.shape.n_layers

    def __call__(self, sets):
        seq, tok, par = self.item
        out = []
        for S in sets:
            mask = np.zeros(self.L, np.uint8)
            mask[list(S)] = 1
            self.v.verify(seq, tok, par, mask=mask)
            t = []
            for _ in range(self.reps):
                a = time.perf_counter()
                self.v.verify(seq, tok, par, mask=mask)
                t.append(time.perf_counter() - a)
            out.append(float(np.median(t)) * 1e3)
        return np.asarray(out)
