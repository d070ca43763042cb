"""GPU checks of the host components around the step: the domain controller
(requests admitted with their domain's skip set, batches planned by skip set,
each sequence's result against the oracle's verify of that sequence) and the
search's sweep evaluator (acceptance and metric stand-in from tss_verify_sweep
equal to those computed from one verify per mask)."""
import numpy as np
import pytest

import synth
from oracle import OracleSequence, prefill, verify
from paper_2609_26100_amd.controller import ConfigMap, SkipController, plan_cost
from paper_2609_26100_amd.search import MeasuredCost, SweepQuality, breadth_search
from tests.gpu_common import TOL, check_decision, gpu_verifier, log, oracle_model

pytestmark = pytest.mark.gpu

TINY = synth.TINY


@pytest.fixture(scope="module")
def pair():
    v = gpu_verifier(TINY, random_gains=True, n_seqs=8, max_tokens=200, max_nodes=8, max_batch=4)
    m = oracle_model(TINY, random_gains=True)
    yield v, m
    v.close()


def test_controller_routes_plans_and_verifies(pair):
    v, m = pair
    phi = ConfigMap(TINY.n_layers, {"translation": {"skip": [3]}, "qa": {"skip": [1, 2]}})
    ctl = SkipController(v, phi)
    domains = ["translation", "qa", "qa", "translation", "unknown", "qa", "translation", "translation"]
    tol, gate = TOL["f32"]
    oseqs = {}
    for s, dom in enumerate(domains):
        v.truncate(s, 0)
        mask = ctl.admit(s, dom)
        ctx = synth.context_tokens(TINY.vocab, 30 + 7 * s, stream=4000 + s)
        v.prefill(s, ctx)
        o = OracleSequence(m, mask)
        prefill(m, o, ctx)
        oseqs[s] = o
    assert not ctl.phi.mask("unknown").any()
    plan = ctl.plan(range(8), 4)
    skip_of = {s: phi.skip_set(domains[s]) for s in range(8)}
    # four translation requests fill one batch of their own
    assert sorted([0, 3, 6, 7]) in [sorted(b) for b in plan]
    assert plan_cost(plan, skip_of, TINY.n_layers) <= plan_cost([[0, 1, 2, 3], [4, 5, 6, 7]], skip_of, TINY.n_layers)
    compared = 0
    for b in plan:
        drafts = [synth.context_tokens(TINY.vocab, 5, stream=4100 + s) for s in b]
        al, nt = v.verify_batch(b, drafts, commit=True)
        lg = v.logits(5 * len(b))
        for i, s in enumerate(b):
            res = verify(m, oseqs[s], drafts[i], None, None, commit=True)
            err = float(np.max(np.abs(lg[5 * i:5 * (i + 1)] - res.logits)))
            assert err <= tol, f"sequence {s}: logits max-abs {err}"
            compared += check_decision(res, int(al[i]), int(nt[i]), gate)
            assert v.length(s) == oseqs[s].n_kv
    log(f"controller: plan {plan}, {compared} decisions compared")


def test_sweep_quality_equals_single_verifies(pair):
    v, m = pair
    L = TINY.n_layers
    items = []
    for s in range(3):
        v.truncate(s, 0)
        v.set_mask(s, None)
        v.prefill(s, synth.context_tokens(TINY.vocab, 40 + 5 * s, stream=4200 + s))
        # a chain of the dense verifier's own greedy tokens (fully accepted when dense)
        cur = [int(synth.context_tokens(TINY.vocab, 1, stream=4300 + s)[0])]
        for _ in range(5):
            v.verify(s, cur, mask=np.zeros(L, np.uint8))
            cur.append(int(v.greedy(len(cur))[-1]))
        items.append((s, np.asarray(cur, dtype=np.int32), None))
    sets = [(), (0,), (3,), (1, 2), (0, 1, 2, 3), (2,)]
    q = SweepQuality(v, items)
    A, M = q(sets)
    # the same quantities from one dry-run verify per (item, mask)
    A1 = np.zeros(len(sets))
    M1 = np.zeros(len(sets))
    dense = []
    for seq, tok, par in items:
        v.verify(seq, tok, par, mask=np.zeros(L, np.uint8))
        dense.append(v.greedy(6))
    for k, S in enumerate(sets):
        mk = np.zeros(L, np.uint8)
        mk[list(S)] = 1
        agree = 0
        for (seq, tok, par), g0 in zip(items, dense):
            al, _ = v.verify(seq, tok, par, mask=mk)
            A1[k] += al + 1
            agree += int((v.greedy(6) == g0).sum())
        A1[k] /= len(items)
        M1[k] = agree / (6 * len(items))
    log(f"sweep quality A {A.tolist()} M {np.round(M, 3).tolist()}")
    np.testing.assert_allclose(A, A1)
    np.testing.assert_allclose(M, M1)
    assert M[0] == 1.0 and A[0] == 6.0
    # a short search end to end on the GPU evaluators
    res = breadth_search(L, 2, q, MeasuredCost(v, items[0], reps=2), eps_A=10.0, eps_M=1.0, tau_A=10.0, tau_M=1.0)
    assert res.pool == list(range(L)) and res.per_depth[0] == L
    assert res.best in res.feasible and res.evaluations == 1 + L + L * (L - 1) // 2
