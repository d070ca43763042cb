"""Domain-to-Configuration Mapping and the Domain-Aware Skip Controller.

Phi maps each supported domain d to its configuration record
G_d = (S_d^*, A_d(S_d^*), M_d(S_d^*), R_d) with R_d = |S_d^*| / L, the skip
set the offline search selected plus its calibrated acceptance, metric and
sparsity ratio; alternative operating points from the search's Pareto set may
be kept beside it.  The map lives in a small local JSON file.  At run time
the controller looks up the request's domain and fixes that skip set for the
whole request; a domain outside the map gets the empty set (the dense
verifier).  One model serves every domain: nothing is pruned or copied.

Batching.  A batched verify step launches each block that any of its
sequences runs, so its weight bytes follow the union of the sequences' active
layers; mixing domains with different skip sets gives back part of what each
one skips.  plan_batches groups the sequences of a scheduling round so as to
keep the total number of launched blocks (summed over the round's steps)
low: a domain with at least max_batch sequences gets full batches of its own
(each launching only its active layers), and the remaining sequences are
packed one by one (largest skip set first) into the open batch whose union of
active layers grows least, or into a new batch when even the best fit would
add more blocks than a batch of its own launches (on a tie it joins: one step
fewer saves the embedding, lm_head and accept work and the launches).
"""
from __future__ import annotations

import json
from dataclasses import asdict, dataclass, field

import numpy as np


@dataclass
class DomainConfig:
    skip: list                 # S_d^*, 0-based layer indices
    accept: float = float("nan")   # A_d(S_d^*)
    metric: float = float("nan")   # M_d(S_d^*)
    ratio: float = 0.0         # R_d = |S_d^*| / L
    alternatives: list = field(default_factory=list)  # other Pareto points: [{"skip", "accept", "metric", "cost_ms"}]


class ConfigMap:
    """Phi: domain -> G_d for a model with n_layers blocks."""

    def __init__(self, n_layers, domains=None):
        self.n_layers = int(n_layers)
        self.domains = {}
        for name, cfg in (domains or {}).items():
            self.set(name, cfg if isinstance(cfg, DomainConfig) else DomainConfig(**cfg))

    def set(self, domain, cfg: DomainConfig):
        skip = sorted(int(l) for l in cfg.skip)
        if len(set(skip)) != len(skip) or any(l < 0 or l >= self.n_layers for l in skip):
            raise ValueError(f"domain {domain!r}: skip set {cfg.skip} outside 0..{self.n_layers - 1}")
        cfg.skip = skip
        cfg.ratio = len(skip) / self.n_layers
        self.domains[str(domain)] = cfg

    def add_search_result(self, domain, result, keep_alternatives=True):
        """Stores the outcome of the offline search (search.breadth_search)."""
        c = result.config(self.n_layers)
        alts = []
        if keep_alternatives:
            alts = [{"skip": list(e.skip), "accept": e.A, "metric": e.M, "cost_ms": e.C}
                    for e in result.pareto if tuple(e.skip) != tuple(result.best)]
        self.set(domain, DomainConfig(c["skip"], c["accept"], c["metric"], c["ratio"], alts))

    def skip_set(self, domain):
        """S(x) = Phi(d(x)) for a supported domain, else the empty set."""
        cfg = self.domains.get(domain)
        return tuple(cfg.skip) if cfg else ()

    def mask(self, domain):
        m = np.zeros(self.n_layers, np.uint8)
        m[list(self.skip_set(domain))] = 1
        return m

    def save(self, path):
        with open(path, "w") as f:
            json.dump({"n_layers": self.n_layers, "domains": {d: asdict(c) for d, c in self.domains.items()}},
                      f, indent=1, sort_keys=True)

    @classmethod
    def load(cls, path):
        with open(path) as f:
            doc = json.load(f)
        return cls(doc["n_layers"], doc.get("domains", {}))


class SkipController:
    """Routes requests to their domain's skip set on a verifier: the mask is set
    on the sequence when the request is admitted (before its prefill) and stays
    for the whole request."""

    def __init__(self, verifier, config_map: ConfigMap):
        if config_map.n_layers != verifier.shape.n_layers:
            raise ValueError("the config map was made for another depth")
        self.v = verifier
        self.phi = config_map
        self.domain_of = {}

    def admit(self, seq, domain):
        mask = self.phi.mask(domain)
        self.v.set_mask(seq, mask)
        self.domain_of[seq] = domain
        return mask

    def release(self, seq):
        self.domain_of.pop(seq, None)

    def plan(self, seqs, max_batch):
        return plan_batches({s: self.phi.skip_set(self.domain_of.get(s)) for s in seqs}, self.phi.n_layers,
                            max_batch)


def launched_blocks(skip_sets, n_layers):
    """Blocks a batched step launches: those some sequence of the batch runs."""
    run = np.zeros(n_layers, bool)
    for S in skip_sets:
        m = np.ones(n_layers, bool)
        m[list(S)] = False
        run |= m
    return int(run.sum())


def plan_batches(skip_of, n_layers, max_batch):
    """skip_of: {seq: skip set}.  Returns a list of batches (lists of seqs),
    each of at most max_batch sequences; see the module docstring."""
    groups = {}
    for s in sorted(skip_of):
        groups.setdefault(tuple(sorted(skip_of[s])), []).append(s)
    batches, rest = [], []
    for S, members in sorted(groups.items(), key=lambda kv: (-len(kv[1]), kv[0])):
        full = len(members) // max_batch * max_batch
        batches += [members[i:i + max_batch] for i in range(0, full, max_batch)]
        rest += [(S, s) for s in members[full:]]
    # leftovers: most skipped layers first, into the batch whose union grows least
    rest.sort(key=lambda x: (-len(x[0]), x[0], x[1]))
    open_b = []  # [members, skip sets]
    for S, s in rest:
        alone = launched_blocks([S], n_layers)
        best, best_add = None, None
        for b in open_b:
            if len(b[0]) >= max_batch:
                continue
            add = launched_blocks(b[1] + [S], n_layers) - launched_blocks(b[1], n_layers)
            if best is None or add < best_add:
                best, best_add = b, add
        if best is not None and best_add <= alone:  # on a tie, joining saves a step's fixed work
            best[0].append(s)
            best[1].append(S)
        else:
            open_b.append([[s], [S]])
    return batches + [b[0] for b in open_b]


def plan_cost(batches, skip_of, n_layers):
    """Total blocks launched by the steps of a plan."""
    return sum(launched_blocks([skip_of[s] for s in b], n_layers) for b in batches)
