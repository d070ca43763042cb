"""A synthetic drafter for decode loops: proposes draft trees from a known
reference continuation (the target's own greedy tokens, computed beforehand
and passed in), so acceptance is controlled by one probability p.

At every draft node that lies on the reference path (its root path spells
the reference tokens), with probability p the next reference token goes to
one of its child slots, slot r (children in rank order, rank 0 first, the
one a top-k tree expands most) drawn with weight 2^-r; every other child,
and every child of an off-path node, gets a uniform token, siblings
distinct.  A chain is the tree whose
node i has parent i - 1.  Holds no model arithmetic: the reference tokens
come from the caller.
"""
from __future__ import annotations

import numpy as np

from .gen import BASE_SEED, _P_DRAFT, _rng


class ReferenceDrafter:
    def __init__(self, reference, vocab, p, parent=None, k=None, seed=BASE_SEED, stream=0):
        """reference: the tokens that follow the root of the first step;
        parent: tree shape (parent[0] = -1), or k for a chain of k drafts."""
        if parent is None:
            parent = np.arange(-1, k, dtype=np.int32)
        self.ref = np.asarray(reference, dtype=np.int64)
        self.parent = np.asarray(parent, dtype=np.int32)
        self.vocab = int(vocab)
        self.p = float(p)
        self.rng = _rng(_P_DRAFT, 7, len(self.parent), stream, seed=seed)
        n = len(self.parent)
        self.children = [[] for _ in range(n)]
        for i in range(1, n):
            self.children[self.parent[i]].append(i)

    def _other(self, avoid):
        while True:
            t = int(self.rng.integers(0, self.vocab))
            if t not in avoid:
                return t

    def __call__(self, root, pos):
        """Draft for the step whose root is the token after `pos` generated
        tokens (reference[pos] is the true next token).  Returns (tokens, parent)."""
        n = len(self.parent)
        tok = np.empty(n, dtype=np.int32)
        tok[0] = root
        on = np.zeros(n, dtype=bool)
        on[0] = True
        depth = np.zeros(n, dtype=np.int64)
        for node in range(n):
            kids = self.children[node]
            if not kids:
                continue
            r = pos + depth[node]
            truth = int(self.ref[r]) if on[node] and r < len(self.ref) else -1
            slot = -1
            if truth >= 0 and self.rng.random() < self.p:
                w = 0.5 ** np.arange(len(kids))
                slot = int(self.rng.choice(len(kids), p=w / w.sum()))
            used = {truth}
            for j, c in enumerate(kids):
                depth[c] = depth[node] + 1
                if j == slot:
                    tok[c] = truth
                    on[c] = True
                else:
                    tok[c] = self._other(used)
                used.add(int(tok[c]))
        return tok, self.parent.copy()
