"""Plain, slow CPU oracle of the sparse-depth verification step.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
baseline leg of the benchmark may import or run anything in this package; the
library's product path never does, and this package shares no code with it
(it imports nothing from the HIP package).

What it computes, and from where:

* The sparse verifier T_S of the paper's Problem Formulation: the target with
  the blocks in the skip set S bypassed; S empty is the dense verifier.
* The block rule of the Domain-Aware Skip Controller section: before block l
  the forward checks l against S and either applies the block (attention and
  feed-forward) or passes the hidden state through unchanged.
* Parallel verification of the drafted tokens by one target pass (Problem
  Formulation) with greedy decoding (Appendix, Evaluation Protocol and Table 3:
  temperature 0) and the underlying method's accept/reject rule kept as is
  (Experiments, Models and speculative decoding methods): the accepted length
  is the depth of the deepest draft node whose whole root path matches the
  target's greedy tokens, and the bonus token is the greedy token there.
* The target is a LLaMA decoder (Appendix, Models): pre-norm residual blocks
  with RMSNorm, rotate-half rotary position embedding, multi-head causal
  attention and a SwiGLU MLP, then a final RMSNorm and an untied lm_head.

Readings where the paper is silent are listed in the module docstrings of
``oracle.forward``.  Numeric values beyond the invariants pinned by the tests
(dense equivalence with an independent LLaMA forward, skip identity, tree =
per-path chains, brute-force acceptance, self-consistency) are not printed by
the paper; no worked example of the verify step exists.
"""
from .forward import (
    OracleModel,
    OracleSequence,
    rmsnorm,
    rope,
    tree_meta,
    prefill,
    verify,
    accept_scan,
    VerifyResult,
)

__all__ = ["OracleModel", "OracleSequence", "rmsnorm", "rope", "tree_meta", "prefill", "verify",
           "accept_scan", "VerifyResult"]
