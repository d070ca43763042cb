"""Decode loops around the sparse verifier.

speculative_decode: greedy speculative decoding of one sequence (Problem
Formulation): a drafter proposes a chain or tree after the last committed
token, one verify step under the request's skip mask accepts the longest root
path that matches the verifier's greedy tokens and commits it with the bonus
token, and the bonus token becomes the next root.  With greedy acceptance
the output is exactly what plain greedy decoding with the same verifier
produces, however good the drafts are; only the number of verify steps
changes.

autoregressive_decode: the plain greedy loop, one token per verify step (a
one-node draft: the root alone), the baseline both for the output and for
throughput.

A drafter is any callable drafter(root, pos) -> (tokens, parent) with
tokens[0] == root, parent[0] == -1 (parent None = chain), where pos counts
the tokens generated so far.  The loop's own host work per step is a
verify call, reading the accepted path, and list appends.
"""
from __future__ import annotations

import time
from dataclasses import dataclass, field

import numpy as np


@dataclass
class DecodeResult:
    tokens: np.ndarray             # the first max_new generated tokens
    steps: int                     # verify steps
    accept_lens: list = field(default_factory=list)  # accepted draft tokens per step
    seconds: float = 0.0           # wall time of the loop
    draft_seconds: float = 0.0     # of which in the drafter

    @property
    def tokens_per_step(self):
        return (sum(self.accept_lens) + len(self.accept_lens)) / max(1, self.steps)

    @property
    def tokens_per_second(self):
        return len(self.tokens) / self.seconds if self.seconds > 0 else float("nan")


def speculative_decode(verifier, seq, root, max_new, drafter, mask=None):
    """Generates at least max_new tokens after `root` (the last prompt token,
    whose K/V are not cached yet) and returns the first max_new.  Every step
    commits, so the sequence grows by accept_len + 1 per step (up to one
    step's worth beyond max_new)."""
    out, acc = [], []
    t_draft = 0.0
    t0 = time.perf_counter()
    while len(out) < max_new:
        a = time.perf_counter()
        tokens, parent = drafter(root, len(out))
        t_draft += time.perf_counter() - a
        al, nt = verifier.verify(seq, tokens, parent, mask=mask, commit=True)
        if al:
            if parent is None:
                out.extend(int(t) for t in tokens[1:al + 1])
            else:
                out.extend(int(tokens[j]) for j in verifier.path(0)[1:])
        out.append(int(nt))
        acc.append(int(al))
        root = int(nt)
    return DecodeResult(np.asarray(out[:max_new], dtype=np.int32), len(acc), acc, time.perf_counter() - t0, t_draft)


def autoregressive_decode(verifier, seq, root, max_new, mask=None):
    """Plain greedy decoding: one committing verify of the root alone per token."""
    out = []
    one = np.zeros(1, dtype=np.int32)
    t0 = time.perf_counter()
    for _ in range(max_new):
        one[0] = root
        _, nt = verifier.verify(seq, one, None, mask=mask, commit=True)
        out.append(int(nt))
        root = int(nt)
    return DecodeResult(np.asarray(out, dtype=np.int32), max_new, [0] * max_new, time.perf_counter() - t0)
