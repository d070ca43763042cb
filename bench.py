"""Benchmark of the sparse-depth verification step on one MI355X.

Workload: 7B-shape decoder (32 layers, d 4096, 32 heads x 128, FFN 11008,
vocab 32000), bf16 random-init N(0, 0.02) weights, one sequence with a
1024-token uniform-random context in paged KV (16-token pages), chain drafts
of k=5 where each drafted token equals the target's greedy token with
probability 0.6, skip masks of 0, 4 and 8 layers drawn from layers 16-31
(nested).  One step is one blocking tss_verify (embedding, every active block,
lm_head, argmax and accept scan) with commit, followed by a rewind of the
sequence to its 1024-token context.

The chain drafts of each mask are a fixed pool of 200 (seeded, drawn whatever
--steps is); warm-up and timed steps cycle through it.

Prints one compact JSON line.  value = accepted tokens/s of the dense
verifier over the timed steps (sum(accept_len + 1) / sum(step latency));
tok_s_at_E divides the expected tokens per step of this draft distribution
(E[accept_len + 1] = 2.383) by the median latency.  The skip-4 and skip-8
figures are in "by_skip", other workloads in "workloads" (one summary each);
--detail-out writes the full records to a file.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import synth  # noqa: E402

METRIC = "verify-step latency (µs) & accepted tok/s, 7B-shape k=5, dense vs 4/8 skipped"
PEAK_HBM = 8.0e12
CTX, K_DRAFT, P_ACCEPT = 1024, 5, 0.6
SKIPS = (0, 4, 8)
# chain drafts per mask, drawn once whatever --steps is; warm-up and timed
# steps cycle through them
DRAFT_POOL = 200
# expected tokens committed per step with chain drafts of k=5 at p=0.6:
# E[accept_len + 1] = sum_{j=0..5} 0.6^j
EXPECTED_TOKENS = sum(P_ACCEPT ** j for j in range(K_DRAFT + 1))


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(shape, active, n_ctx, M):
    """Bytes one verify must move: active blocks' bf16 weights, their KV read
    and write, norm gains; lm_head, embedding rows, final norm and logits."""
    d, f, v = shape.d_model, shape.ffn_dim, shape.vocab
    per_layer = 2 * (4 * d * d + 3 * d * f) + 4 * d * n_ctx + 4 * d * M + 4 * d
    return active * per_layer + 2 * v * d + 2 * M * d + 2 * d + 4 * M * v


def batch_bytes(shape, seqs):
    """Algorithmic bytes of one step over several sequences, each given as
    (skip mask, context length, nodes): the weights and norm gains of every
    block some sequence runs (read once for the batch), each sequence's KV read
    and write for the blocks it runs, lm_head, embedding rows, final norm and
    the logits of all rows."""
    d, f, v = shape.d_model, shape.ffn_dim, shape.vocab
    union = np.zeros(shape.n_layers, bool)
    kv = 0
    for mask, n_ctx, m in seqs:
        act = np.asarray(mask) == 0
        union |= act
        kv += int(act.sum()) * (4 * d * n_ctx + 4 * d * m)
    M = sum(m for _, _, m in seqs)
    return int(union.sum()) * (2 * (4 * d * d + 3 * d * f) + 4 * d) + kv + 2 * v * d + 2 * M * d + 2 * d + 4 * M * v


# HBM traffic of one gate/up launch (7B shape, 6 rows), from two rocprofv3
# --pmc passes (FETCH_SIZE, then WRITE_SIZE) over
#   bench.py --steps 5 --warmup 1 --no-cpu-baseline --skips 0 --workloads none --calib-copy 1
# KiB per dispatch, mean of the last 32 gate/up dispatches.  The same counters
# read 524319.2 KiB (FETCH) and 1048576.0 KiB (WRITE) for the 1 GiB device copy
# that run makes, so FETCH_SIZE is scaled by 2.0 and WRITE_SIZE by 1.0.  The
# figures hold for the kernel sources hashed here; any change to them voids
# the traffic field until the counters are taken again.
GATEUP_COUNTERS = {"fetch_kib": 88389.5, "write_kib": 129.0, "fetch_scale": 2.0, "write_scale": 1.0,
                   "sources": ("paper_2609_26100_amd/csrc/k_gemm.hip", "paper_2609_26100_amd/csrc/tss_internal.h"),
                   "sha256": "4491eeb3952547523949bd68985d968d5278dad93cb1cdcb0afcd43bc396b1dc"}


def gateup_traffic():
    """Measured HBM bytes per gate/up launch, or None if the kernel changed since."""
    import hashlib
    h = hashlib.sha256()
    for f in GATEUP_COUNTERS["sources"]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    if h.hexdigest() != GATEUP_COUNTERS["sha256"]:
        return None
    c = GATEUP_COUNTERS
    return (c["fetch_kib"] * c["fetch_scale"] + c["write_kib"] * c["write_scale"]) * 1024


def gateup_bytes(shape, M):
    """Algorithmic bytes of one gate/up launch: W_gate and W_up (bf16), the
    normalised input rows, the SwiGLU output rows."""
    d, f = shape.d_model, shape.ffn_dim
    return 2 * 2 * f * d + 2 * M * d + 2 * M * f


def run_gpu(args):
    import torch
    from paper_2609_26100_amd import tss as abi
    from paper_2609_26100_amd.verifier import Verifier

    shape = synth.LLAMA_7B
    M = K_DRAFT + 1
    t0 = time.time()
    # room for the 2048-token tree workload, which reuses these weights
    v = Verifier(shape, n_seqs=1, max_tokens=2048 + 64, max_nodes=64, device="cuda:0")
    gen = synth.abi_tensor_loader(shape)
    t_gen = [0.0]

    def get(idx):
        a = time.time()
        arr = gen(idx)
        t_gen[0] += time.time() - a
        return arr
    v.load(get)
    log(f"weights generated ({t_gen[0]:.1f}s) and loaded ({time.time() - t0 - t_gen[0]:.1f}s)")
    toks = synth.context_tokens(shape.vocab, CTX + 1)
    ctx, root = toks[:CTX], int(toks[CTX])
    masks = synth.nested_skip_masks(shape.n_layers, 16, 31, SKIPS)

    if args.calib_copy:
        # a plain device copy of known size, so HBM counters can be scaled
        n = int(args.calib_copy * (1 << 30))
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy: {n} bytes read, {n} bytes written")
        del src, dst

    results = {}
    prof = None
    direct_median = None
    for s in args.skips:
        mask = masks[s]
        v.truncate(0, 0)
        v.set_mask(0, mask)
        t1 = time.time()
        v.prefill(0, ctx)
        # greedy continuation of this masked target (dry runs)
        cur = [root]
        for _ in range(K_DRAFT):
            v.verify(0, cur)
            cur.append(int(v.greedy(len(cur))[-1]))
        greedy = np.asarray(cur[1:])
        log(f"skip {s}: layers {np.nonzero(mask)[0].tolist()} prefill+greedy {time.time() - t1:.1f}s")
        drafts = [np.concatenate([[root], synth.chain_draft(greedy, shape.vocab, p_accept=P_ACCEPT, stream=i)])
                  for i in range(DRAFT_POOL)]
        # accept length of each pool draft: its leading run of greedy tokens
        pool_accept = np.array([int(np.cumprod(d[1:] == greedy).sum()) for d in drafts])

        def timed(n_steps, tag, after_warmup=None):
            for i in range(args.warmup):
                v.verify(0, drafts[i % DRAFT_POOL], commit=True)
                v.truncate(0, CTX)
            if after_warmup:
                after_warmup()
            log(f"skip {s}: timing {n_steps} steps ({tag})")
            torch.cuda.synchronize()
            lat = np.empty(n_steps)
            acc = np.empty(n_steps, dtype=np.int64)
            t_start = time.perf_counter()
            for i in range(n_steps):
                a = time.perf_counter()
                al, _ = v.verify(0, drafts[i % DRAFT_POOL], commit=True)
                lat[i] = time.perf_counter() - a
                acc[i] = al
                v.truncate(0, CTX)
            torch.cuda.synchronize()
            return lat, acc, time.perf_counter() - t_start

        v.set_launch_mode(abi.TSS_LAUNCH_GRAPH)
        lat, acc, total = timed(args.steps, "graph launches")
        if s == 0:
            # the gate/up kernel timed with HIP events (these steps use direct launches)
            v.set_launch_mode(abi.TSS_LAUNCH_DIRECT)
            abi.tss_profile_kernel(v.ctx, abi.TSS_K_GATEUP, 0)
            dlat, _, _ = timed(args.steps, "direct launches, gate/up kernel timed with events",
                               after_warmup=lambda: abi.tss_profile_read(v.ctx, reset=True))
            prof = abi.tss_profile_read(v.ctx, reset=True)
            abi.tss_profile_kernel(v.ctx, -1)
            v.set_launch_mode(abi.TSS_LAUNCH_GRAPH)
            direct_median = float(np.median(dlat))
        active = shape.n_layers - s
        by = algorithmic_bytes(shape, active, CTX, M)
        med = float(np.median(lat))
        assert all(int(a) == int(pool_accept[i % DRAFT_POOL]) for i, a in enumerate(acc)), \
            "accept lengths differ from the drafts' greedy prefixes"
        results[s] = {
            "skipped_layers": np.nonzero(mask)[0].tolist(),
            "latency_us_median": med * 1e6,
            "latency_us_p10": float(np.percentile(lat, 10)) * 1e6,
            "latency_us_p90": float(np.percentile(lat, 90)) * 1e6,
            "accepted_tok_s": float((acc + 1).sum() / lat.sum()),
            "accepted_tok_s_at_expected": EXPECTED_TOKENS / med,
            "accepted_tok_s_pool_mean": float((pool_accept + 1).mean()) / med,
            "mean_accept_len": float(acc.mean()),
            "pool_mean_accept_len": float(pool_accept.mean()),
            "algorithmic_GB": by / 1e9,
            "roofline_latency_us": by / PEAK_HBM * 1e6,
            "roofline_frac": by / PEAK_HBM / med,
            "wall_s": total,
        }
        if s == 0:
            results[s]["latency_us_median_direct_launches"] = direct_median * 1e6
        log(f"skip {s}: median {med * 1e6:.0f} us, accepted {results[s]['accepted_tok_s']:.0f} tok/s, "
            f"roofline frac {results[s]['roofline_frac']:.3f}")
    d0 = results[args.skips[0]]
    for s in args.skips[1:]:
        results[s]["latency_ratio_vs_dense"] = results[s]["latency_us_median"] / d0["latency_us_median"]
        results[s]["byte_ratio_vs_dense"] = results[s]["algorithmic_GB"] / d0["algorithmic_GB"]
    return shape, results, prof, v


def _load_verifier(shape, **kw):
    from paper_2609_26100_amd.verifier import Verifier
    t0 = time.time()
    v = Verifier(shape, device="cuda:0", **kw)
    gen = synth.abi_tensor_loader(shape)
    n = 3 + 9 * shape.n_layers

    def get(idx):
        if idx and idx % 90 == 0:
            log(f"{shape.name}: tensor {idx}/{n} ({time.time() - t0:.0f}s)")
        return gen(idx)
    v.load(get)
    log(f"{shape.name}: weights generated and loaded in {time.time() - t0:.1f}s")
    return v


def _free(v):
    import torch
    v.close()
    del v.weights, v.workspace, v.kv_pool
    v.prefix = None
    torch.cuda.empty_cache()


def _timed(step, n_warmup, n_steps):
    """Blocking steps; returns per-step latency (s) and per-step accepted tokens."""
    for _ in range(n_warmup):
        step(0)
    lat, acc = np.empty(n_steps), np.empty(n_steps)
    for i in range(n_steps):
        a = time.perf_counter()
        acc[i] = step(i)
        lat[i] = time.perf_counter() - a
    return lat, acc


def _summary(lat, acc, by):
    med = float(np.median(lat))
    return {"latency_us_median": med * 1e6, "latency_us_p10": float(np.percentile(lat, 10)) * 1e6,
            "latency_us_p90": float(np.percentile(lat, 90)) * 1e6, "accepted_tok_s": float(acc.sum() / lat.sum()),
            "mean_accepted_per_step": float(acc.mean()), "algorithmic_GB": by / 1e9,
            "roofline_latency_us": by / PEAK_HBM * 1e6, "roofline_frac": by / PEAK_HBM / med, "steps": len(lat)}


def workload_tree_7b(args, v=None):
    """7B, 2048-token context, 60-node top-k-style tree (depth 6, branching
    4,3,2,2,1,1, level quotas 4,12,20,12,8,4), 6 layers skipped from 16-31;
    the greedy token sits in a random child slot with probability 0.6."""
    shape = synth.LLAMA_7B
    ctx_n = 2048
    if v is None:
        v = _load_verifier(shape, n_seqs=1, max_tokens=ctx_n + 64, max_nodes=64)
    v.truncate(0, 0)
    mask = synth.random_skip_mask(shape.n_layers, 16, 31, 6, stream=3)
    toks = synth.context_tokens(shape.vocab, ctx_n + 1, stream=3)
    v.set_mask(0, mask)
    v.prefill(0, toks[:ctx_n])
    parent = synth.topk_tree_parents((4, 3, 2, 2, 1, 1), (4, 12, 20, 12, 8, 4))

    def greedy_of(tok, node):
        path = [node]
        while parent[path[-1]] >= 0:
            path.append(int(parent[path[-1]]))
        chain = tok[path[::-1]]
        v.verify(0, chain)
        return int(v.greedy(len(chain))[-1])
    tokens = synth.tree_draft_tokens(parent, int(toks[ctx_n]), greedy_of, shape.vocab, 0.6, stream=3)

    def step(i):
        al, _ = v.verify(0, tokens, parent, commit=True)
        v.truncate(0, ctx_n)
        return al + 1
    lat, acc = _timed(step, args.warmup, args.aux_steps)
    out = _summary(lat, acc, batch_bytes(shape, [(mask, ctx_n, len(parent))]))
    out.update({"workload": "7B-shape, 60-node draft tree + root, 2048-token context, 6 layers skipped",
                "skipped_layers": np.nonzero(mask)[0].tolist(), "nodes": len(parent)})
    _free(v)
    return out


def workload_batch_13b(args):
    """13B, 8 sequences with contexts U{512..4096}, chain k=8 (p=0.6 on each
    sequence's masked greedy continuation), per-sequence masks of U{0..10}
    layers from 2-39."""
    shape = synth.LLAMA_13B
    B, k = 8, 8
    rng = np.random.default_rng(synth.BASE_SEED + 13)
    ctx_lens = [int(x) for x in rng.integers(512, 4097, size=B)]
    masks = [synth.random_skip_mask(shape.n_layers, 2, 39, int(rng.integers(0, 11)), stream=40 + i) for i in range(B)]
    v = _load_verifier(shape, n_seqs=B, max_tokens=4096 + k + 8, max_nodes=k + 1, max_batch=B)
    drafts = []
    t0 = time.time()
    for i in range(B):
        toks = synth.context_tokens(shape.vocab, ctx_lens[i] + 1, stream=50 + i)
        v.set_mask(i, masks[i])
        v.prefill(i, toks[:-1])
        cur = [int(toks[-1])]
        for _ in range(k):
            v.verify(i, cur)
            cur.append(int(v.greedy(len(cur))[-1]))
        drafts.append(cur)
    log(f"13B batch: prefilled {sum(ctx_lens)} tokens and drafted in {time.time() - t0:.1f}s")
    seqs = list(range(B))
    inst = [[np.concatenate([[d[0]], synth.chain_draft(np.asarray(d[1:]), shape.vocab, p_accept=0.6,
                                                        stream=1000 * j + i)]) for i, d in enumerate(drafts)]
            for j in range(args.warmup + args.aux_steps)]

    def step(j):
        al, _ = v.verify_batch(seqs, inst[j], commit=True)
        for i in seqs:
            v.truncate(i, ctx_lens[i])
        return int((al + 1).sum())
    lat, acc = _timed(step, args.warmup, args.aux_steps)
    out = _summary(lat, acc, batch_bytes(shape, [(masks[i], ctx_lens[i], k + 1) for i in seqs]))
    union = np.zeros(shape.n_layers, bool)
    for mk in masks:
        union |= mk == 0
    out.update({"workload": "13B-shape, batch of 8 sequences, chain k=8, contexts 512-4096, per-sequence masks",
                "contexts": ctx_lens, "skipped_per_sequence": [int(mk.sum()) for mk in masks],
                "blocks_launched": int(union.sum())})
    _free(v)
    return out


def workload_sweep_33b(args):
    """33B, one 4096-token context prefilled dense, 32-node tree + root (depth
    5, branching 4,3,2,1,1, quotas 4,10,10,5,3), 64 masks of U{4..16} layers
    from 2-59 verified back to back as dry runs (timing only); then the same
    64 masks through the packed sweep (3 masks per step), without and with
    reuse of the shared dense prefix."""
    shape = synth.LLAMA_33B
    ctx_n = 4096
    v = _load_verifier(shape, n_seqs=1, max_tokens=ctx_n + 112, max_nodes=33, max_batch=4)
    toks = synth.context_tokens(shape.vocab, ctx_n + 1, stream=5)
    v.prefill(0, toks[:ctx_n])
    parent = synth.topk_tree_parents((4, 3, 2, 1, 1), (4, 10, 10, 5, 3))

    def greedy_of(tok, node):
        path = [node]
        while parent[path[-1]] >= 0:
            path.append(int(parent[path[-1]]))
        chain = tok[path[::-1]]
        v.verify(0, chain)
        return int(v.greedy(len(chain))[-1])
    tokens = synth.tree_draft_tokens(parent, int(toks[ctx_n]), greedy_of, shape.vocab, 0.6, stream=5)
    rng = np.random.default_rng(synth.BASE_SEED + 33)
    masks = [synth.random_skip_mask(shape.n_layers, 2, 59, int(rng.integers(4, 17)), stream=100 + i)
             for i in range(64)]
    per_mask, lat_all, acc_all, by_all = [], [], [], []
    n_steps = max(3, args.aux_steps // 10)
    for mi, mk in enumerate(masks):
        if mi % 16 == 0:
            log(f"33B sweep: mask {mi}/64")

        def step(i, mk=mk):
            al, _ = v.verify(0, tokens, parent, mask=mk)
            return al + 1
        lat, acc = _timed(step, 1, n_steps)
        by = batch_bytes(shape, [(mk, ctx_n, len(parent))])
        per_mask.append((int(mk.sum()), float(np.median(lat)) * 1e6, by / PEAK_HBM / float(np.median(lat))))
        lat_all.append(lat)
        acc_all.append(acc)
        by_all.append(by)
    all_masks = np.stack(masks)

    def sweep_ms(reuse):
        v.verify_sweep(0, tokens, all_masks, parent, reuse_prefix=reuse)
        t0 = time.perf_counter()
        for _ in range(n_steps):
            v.verify_sweep(0, tokens, all_masks, parent, reuse_prefix=reuse)
        return (time.perf_counter() - t0) / n_steps
    packed_plain = sweep_ms(False)
    packed = sweep_ms(True)
    # the first evaluations of the breadth search: dense and every single-layer skip
    singles = np.zeros((shape.n_layers + 1, shape.n_layers), np.uint8)
    for l in range(shape.n_layers):
        singles[l + 1, l] = 1

    def singles_ms(reuse):
        v.verify_sweep(0, tokens, singles, parent, reuse_prefix=reuse)
        t0 = time.perf_counter()
        for _ in range(n_steps):
            v.verify_sweep(0, tokens, singles, parent, reuse_prefix=reuse)
        return (time.perf_counter() - t0) / n_steps
    singles_plain = singles_ms(False)
    singles_reuse = singles_ms(True)
    log(f"33B sweep: dense + 60 single-layer skips packed {singles_plain * 1e3:.1f} ms, "
        f"with prefix reuse {singles_reuse * 1e3:.1f} ms")
    log(f"33B sweep: 64 masks packed {packed_plain * 1e3:.1f} ms, with prefix reuse {packed * 1e3:.1f} ms, "
        f"{sum(p[1] for p in per_mask) / 1e3:.1f} ms one by one")
    sk = np.array([p[0] for p in per_mask], float)
    us = np.array([p[1] for p in per_mask])
    slope, icpt = np.polyfit(sk, us, 1)
    lat = np.concatenate(lat_all)
    med = float(np.median([p[1] for p in per_mask])) * 1e-6
    out = {"workload": "33B-shape, 32-node tree + root, 4096-token context, 64 skip masks of 4-16 layers (dry runs)",
           "masks": 64, "steps_per_mask": n_steps, "latency_us_median": med * 1e6,
           "latency_us_p10": float(np.percentile(us, 10)), "latency_us_p90": float(np.percentile(us, 90)),
           "accepted_tok_s": float(np.concatenate(acc_all).sum() / lat.sum()),
           "algorithmic_GB_mean": float(np.mean(by_all)) / 1e9,
           "roofline_frac_median": float(np.median([p[2] for p in per_mask])),
           "us_per_skipped_layer": float(-slope), "us_at_zero_skips_fit": float(icpt),
           "roofline_us_per_skipped_layer": batch_bytes(shape, [(np.zeros(shape.n_layers), ctx_n, 33)]) / PEAK_HBM * 1e6
           - batch_bytes(shape, [(synth.mask_from_layers(shape.n_layers, [2]), ctx_n, 33)]) / PEAK_HBM * 1e6,
           "per_mask": [{"skipped": p[0], "latency_us": p[1], "roofline_frac": p[2]} for p in per_mask],
           "packed_sweep_ms": packed * 1e3, "packed_sweep_no_prefix_reuse_ms": packed_plain * 1e3,
           "one_by_one_ms": sum(p[1] for p in per_mask) / 1e3,
           "singles_61_masks_packed_ms": singles_plain * 1e3, "singles_61_masks_prefix_reuse_ms": singles_reuse * 1e3,
           "packed_speedup": sum(p[1] for p in per_mask) / 1e6 / packed}
    _free(v)
    return out


def workload_decode_7b(args, v):
    """7B, 1024-token prompt, T = 96 new tokens (the paper's decoding length):
    plain autoregressive greedy decoding (one verify per token) against
    speculative decoding with a synthetic drafter that follows the reference
    continuation with p = 0.8 (chain k = 5, and the 60-node top-k tree), dense
    and with 4 layers skipped.  Wall time of the whole loop, host included."""
    from paper_2609_26100_amd.decode import autoregressive_decode, speculative_decode
    shape = synth.LLAMA_7B
    T, ctx_n = 96, CTX
    prompt = synth.context_tokens(shape.vocab, ctx_n + 1, stream=9)
    tree = synth.topk_tree_parents((4, 3, 2, 2, 1, 1), (4, 12, 20, 12, 8, 4))
    out = {"workload": "7B-shape, 1024-token prompt, 96 new tokens, synthetic drafter p=0.8", "T": T, "runs": {}}
    for skip in (0, 4):
        mask = synth.nested_skip_masks(shape.n_layers, 16, 31, [skip], stream=1)[skip]
        v.truncate(0, 0)
        v.set_mask(0, mask)
        v.prefill(0, prompt[:ctx_n])
        base = ctx_n
        autoregressive_decode(v, 0, int(prompt[ctx_n]), 8)      # capture the one-node step
        v.truncate(0, base)
        ref = autoregressive_decode(v, 0, int(prompt[ctx_n]), T)
        runs = {"autoregressive": ref}
        for name, drafter in [("chain_k5", synth.ReferenceDrafter(ref.tokens, shape.vocab, 0.8, k=5, stream=11)),
                              ("tree60", synth.ReferenceDrafter(ref.tokens, shape.vocab, 0.8, parent=tree, stream=12))]:
            v.truncate(0, base)
            speculative_decode(v, 0, int(prompt[ctx_n]), 16, drafter)  # capture the step shapes
            v.truncate(0, base)
            drafter.rng = np.random.default_rng(1000 + skip)
            runs[name] = speculative_decode(v, 0, int(prompt[ctx_n]), T, drafter)
        for name, r in runs.items():
            same = int(np.sum(np.cumprod(r.tokens == ref.tokens)))
            out["runs"][f"skip{skip}_{name}"] = {
                "tok_s": r.tokens_per_second, "steps": r.steps, "tokens_per_step": r.tokens_per_step,
                "ms": r.seconds * 1e3, "draft_ms": r.draft_seconds * 1e3, "equal_prefix": same,
                "speedup_vs_autoregressive": ref.seconds / r.seconds}
            log(f"decode skip {skip} {name}: {r.tokens_per_second:.0f} tok/s, {r.steps} steps, "
                f"{r.tokens_per_step:.2f} tokens/step, equal to autoregressive for {same}/{T}")
    v.truncate(0, 0)
    v.set_mask(0, None)
    best = out["runs"]["skip0_chain_k5"]
    out["latency_us_median"] = best["ms"] * 1e3 / best["steps"]
    out["accepted_tok_s"] = best["tok_s"]
    return out


def workload_search_7b(args):
    """Algorithm 1 on the 7B shape: 8 calibration items (512-token contexts,
    chain k = 5 drafts that follow, with p = 0.9, the greedy tokens of the
    verifier with a hidden set of 4 layers from 16-31 skipped, a stand-in for a
    drafter aligned with a shallower verifier).  Acceptance and the metric
    stand-in come from packed mask sweeps, the cost from timed single verifies
    of the feasible sets.  The task metric is not available here; its
    stand-in (the fraction of draft nodes whose greedy token equals the dense
    verifier's) must stay within 50 % of the dense value, and acceptance within
    5 %: both constraints of Algorithm 1 bind (the record counts the sets only
    the metric rejected).  Also times the sweep against one verify per mask."""
    from paper_2609_26100_amd.search import MeasuredCost, SweepQuality, breadth_search
    shape = synth.LLAMA_7B
    n_items, ctx_n, k = 8, 512, 5
    v = _load_verifier(shape, n_seqs=n_items, max_tokens=ctx_n + 130, max_nodes=64, max_batch=8)
    hidden = synth.random_skip_mask(shape.n_layers, 16, 31, 4, stream=77)
    items = []
    for i in range(n_items):
        toks = synth.context_tokens(shape.vocab, ctx_n + 1, stream=700 + i)
        v.prefill(i, toks[:ctx_n])
        cur = [int(toks[ctx_n])]
        for _ in range(k):
            v.verify(i, cur, mask=hidden)
            cur.append(int(v.greedy(len(cur))[-1]))
        d = np.concatenate([[cur[0]], synth.chain_draft(np.asarray(cur[1:]), shape.vocab, p_accept=0.9,
                                                        stream=800 + i)])
        items.append((i, d.astype(np.int32), None))
    quality = SweepQuality(v, items)
    cost = MeasuredCost(v, items[0], reps=5)
    eps_A, eps_M = 0.05, 0.5
    res = breadth_search(shape.n_layers, 4, quality, cost, eps_A=eps_A, eps_M=eps_M, tau_A=0.0, tau_M=0.0,
                         relative=True, log=lambda ln: log("search: " + ln))
    A0, M0 = res.baseline.A, res.baseline.M
    metric_only = sum(1 for S, (a, m) in res.entries.items()
                      if len(S) > 1 and a >= A0 * (1 - eps_A) and m < M0 * (1 - eps_M))
    # sweep throughput: 64 masks of 1-4 layers from 16-31, packed vs one verify per mask
    rng = np.random.default_rng(5)
    masks = np.stack([synth.random_skip_mask(shape.n_layers, 16, 31, int(rng.integers(1, 5)), stream=900 + j)
                      for j in range(64)])
    seq, tok, _ = items[0]
    v.verify_sweep(seq, tok, masks)
    t0 = time.perf_counter()
    reps = 5
    for _ in range(reps):
        v.verify_sweep(seq, tok, masks)
    packed = (time.perf_counter() - t0) / reps
    for mk in masks:
        v.verify(seq, tok, mask=mk)
    t0 = time.perf_counter()
    for _ in range(reps):
        for mk in masks:
            v.verify(seq, tok, mask=mk)
    single = (time.perf_counter() - t0) / reps
    cfg = res.config(shape.n_layers)
    out = {"workload": "7B-shape breadth search (Algorithm 1), 8 calibration items, chain k=5, 512-token contexts",
           "hidden_skip": np.nonzero(hidden)[0].tolist(), "pool": res.pool, "per_depth": res.per_depth,
           "evaluations": res.evaluations, "cost_evaluations": res.cost_evaluations, "search_s": res.seconds,
           "sweep_calls": quality.sweeps, "best": cfg, "eps_A": eps_A, "eps_M": eps_M,
           "rejected_by_metric_only": metric_only,
           "baseline": {"accept": res.baseline.A, "metric": res.baseline.M, "cost_ms": res.baseline.C},
           "pareto": [{"skip": list(e.skip), "accept": e.A, "metric": e.M, "cost_ms": e.C} for e in res.pareto],
           "sweep_64_masks_ms": packed * 1e3, "single_verifies_64_masks_ms": single * 1e3,
           "sweep_speedup": single / packed, "masks_per_s_sweep": 64 / packed, "masks_per_s_single": 64 / single}
    log(f"search: best {cfg}, {res.evaluations} evaluations in {res.seconds:.1f}s; 64-mask sweep "
        f"{packed * 1e3:.1f} ms vs {single * 1e3:.1f} ms one verify per mask ({single / packed:.2f}x)")
    out["latency_us_median"] = packed / 64 * 1e6
    out["accepted_tok_s"] = None
    _free(v)
    return out


def workload_domains_13b(args):
    """13B, 16 requests in two domains whose configurations skip 8 different
    layers each (from 20-39), admitted through the domain controller (mask
    set before prefill, 1024-token contexts), one chain k=5 verify per request
    per round, at most 8 sequences per step.  One round in arrival order
    (domains interleaved, so each step launches the union of both domains'
    layers) against one round planned by the controller (a step per domain)."""
    from paper_2609_26100_amd.controller import ConfigMap, SkipController, plan_cost
    shape = synth.LLAMA_13B
    B, n_req, ctx_n, k = 8, 16, 1024, 5
    layers = np.random.default_rng(13).permutation(np.arange(20, 40))
    phi = ConfigMap(shape.n_layers, {"translation": {"skip": layers[:8].tolist()},
                                     "qa": {"skip": layers[8:16].tolist()}})
    v = _load_verifier(shape, n_seqs=n_req, max_tokens=ctx_n + 16, max_nodes=k + 1, max_batch=B)
    ctl = SkipController(v, phi)
    drafts = []
    for s in range(n_req):
        ctl.admit(s, "translation" if s % 2 == 0 else "qa")
        toks = synth.context_tokens(shape.vocab, ctx_n + k + 1, stream=1300 + s)
        v.prefill(s, toks[:ctx_n])
        drafts.append(toks[ctx_n:])
    skip_of = {s: phi.skip_set(ctl.domain_of[s]) for s in range(n_req)}
    plans = {"arrival_order": [list(range(0, 8)), list(range(8, 16))], "controller": ctl.plan(range(n_req), B)}
    out = {"workload": "13B-shape, 16 requests in 2 domains (8 skipped layers each), chain k=5, 1024-token contexts",
           "skip": {d: c.skip for d, c in phi.domains.items()}}
    for name, plan in plans.items():
        def rnd(_i, plan=plan):
            for b in plan:
                v.verify_batch(b, [drafts[s] for s in b])
            return 0
        lat, _ = _timed(rnd, 3, max(5, args.aux_steps // 2))
        by = sum(batch_bytes(shape, [(phi.mask(ctl.domain_of[s]), ctx_n, k + 1) for s in b]) for b in plan)
        out[name] = {"round_us_median": float(np.median(lat)) * 1e6, "steps": len(plan),
                     "blocks_launched": plan_cost(plan, skip_of, shape.n_layers), "algorithmic_GB": by / 1e9,
                     "roofline_frac": by / PEAK_HBM / float(np.median(lat)), "batches": plan}
        log(f"domains 13B {name}: {out[name]['round_us_median']:.0f} us per round, "
            f"{out[name]['blocks_launched']} blocks launched")
    out["speedup"] = out["arrival_order"]["round_us_median"] / out["controller"]["round_us_median"]
    out["latency_us_median"] = out["controller"]["round_us_median"]
    out["accepted_tok_s"] = None
    _free(v)
    return out


def _blas_info():
    from threadpoolctl import threadpool_info
    info = [d for d in threadpool_info() if d.get("user_api") == "blas"] or threadpool_info()
    threads = max([d.get("num_threads", 1) for d in info] + [1])
    name = ", ".join(f"{d.get('internal_api', '?')} {d.get('version', '')} ({d.get('threading_layer', '?')})"
                     for d in info) or "unknown"
    return int(threads), name


def cpu_baseline(args, shape, tokens_per_step):
    """The oracle, untouched, on bounded samples of the workload's own inputs.

    7B chain k=5 step at a 1024-token context: measured with four of the 32
    blocks active (their K/V from the oracle's own prefill of the context
    through those blocks, not timed) and with every block skipped; the dense
    step is extrapolated as the block-free time plus 32 x the measured
    per-block time (the oracle's blocks are identical in shape and cost).
    Tiny fp32 model (4 layers, d 256, mask {2}, 128-token context, chain k=5):
    the full verify step, timed with one BLAS thread."""
    from threadpoolctl import threadpool_limits

    from oracle import OracleModel, OracleSequence, prefill, verify

    def model(sh):
        cache = {}

        def get(name, layer):
            if (name, layer) not in cache:
                cache[(name, layer)] = synth.weight_tensor(sh, name, layer)
            return cache[(name, layer)]
        return OracleModel(sh, get)

    def median_time(fn, reps):
        fn()
        t = []
        for _ in range(reps):
            a = time.perf_counter()
            fn()
            t.append(time.perf_counter() - a)
        return float(np.median(t))

    threads, blas = _blas_info()
    m = model(shape)
    toks = synth.context_tokens(shape.vocab, CTX + 1)
    ctx, root = toks[:CTX], int(toks[CTX])
    n_act = 4
    some = np.ones(shape.n_layers, np.uint8)
    some[:n_act] = 0
    seq = OracleSequence(m, some)
    t = time.time()
    prefill(m, seq, ctx)
    log(f"oracle prefill through {n_act} blocks: {time.time() - t:.1f}s")
    tokens = np.concatenate([[root], synth.context_tokens(shape.vocab, K_DRAFT, stream=7)])
    none = np.ones(shape.n_layers, np.uint8)
    t_some = median_time(lambda: verify(m, seq, tokens, mask=some), args.cpu_reps)
    t_none = median_time(lambda: verify(m, seq, tokens, mask=none), args.cpu_reps)
    per_block = (t_some - t_none) / n_act
    dense = t_none + shape.n_layers * per_block
    del m, seq

    tiny = synth.TINY
    mt = model(tiny)
    tt = synth.context_tokens(tiny.vocab, 129)
    tmask = synth.mask_from_layers(tiny.n_layers, [2])
    tseq = OracleSequence(mt, tmask)
    prefill(mt, tseq, tt[:128])
    cur = [int(tt[128])]
    for _ in range(K_DRAFT):
        cur.append(int(verify(mt, tseq, np.asarray(cur)).greedy[-1]))
    tdraft = np.concatenate([cur[:1], synth.chain_draft(np.asarray(cur[1:]), tiny.vocab, n_greedy=3)])
    with threadpool_limits(limits=1):
        t_tiny = median_time(lambda: verify(mt, tseq, tdraft), 20)
    tiny_accept = verify(mt, tseq, tdraft).accept_len
    return {
        "value": tokens_per_step / dense,
        "unit": "accepted tok/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"numpy fp32 oracle, 7B chain k=5 verify at context 1024, {threads} BLAS threads: measured with "
                   f"blocks 0-{n_act - 1} active ({t_some * 1e3:.0f} ms) and with every block skipped "
                   f"({t_none * 1e3:.0f} ms), median of {args.cpu_reps}; dense step extrapolated as "
                   f"skipped + {shape.n_layers} x per-block = {dense * 1e3:.0f} ms; tokens per step as in the GPU run"),
        "host_cpus": os.cpu_count(),
        "blas": blas,
        "latency_ms_extrapolated": dense * 1e3,
        "tiny_single_thread": {"latency_ms": t_tiny * 1e3, "accept_len": int(tiny_accept),
                               "accepted_tok_s": (tiny_accept + 1) / t_tiny},
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--cpu-reps", type=int, default=5)
    ap.add_argument("--aux-steps", type=int, default=50, help="timed steps of the tree / batch workloads")
    ap.add_argument("--workloads", default="decode7b,tree7b,batch13b,domains13b,sweep33b,search7b",
                    help="other workloads to time after the headline one (comma list, or none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--skips", default="0,4,8", help="skip counts to time; the first is the headline")
    ap.add_argument("--calib-copy", type=float, default=0.0,
                    help="GiB of a plain device copy run first (HBM counter calibration)")
    ap.add_argument("--detail-out", default="", help="file for the full per-skip, per-mask and workload records")
    args = ap.parse_args()
    args.skips = [int(x) for x in args.skips.split(",")]
    if args.skips[0] != 0 or any(x not in SKIPS for x in args.skips):
        raise SystemExit(f"--skips must start with 0 and use counts from {SKIPS}")
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported by this build "
              "(the verify step runs on a single MI355X)", file=sys.stderr)
        sys.exit(2)
    shape, res, prof, v7 = run_gpu(args)
    d0 = res[0]
    M = K_DRAFT + 1
    roof = None
    if prof and prof[1] > 0:
        avg_s = prof[0] / prof[1] / 1e3
        gb = gateup_bytes(shape, M)
        achieved = gb / avg_s / 1e9
        roof = {"kernel": "gate/up projection + SwiGLU (layer 0, dense)", "bound": "hbm",
                "achieved": achieved, "peak": PEAK_HBM / 1e9, "unit": "GB/s", "frac": achieved / (PEAK_HBM / 1e9),
                "traffic": gateup_traffic(), "avg_launch_us": avg_s * 1e6, "launches": prof[1],
                "algorithmic_bytes_per_launch": gb}
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args, shape, d0["mean_accept_len"] + 1)
    workloads = {}
    runners = {"tree7b": workload_tree_7b, "batch13b": workload_batch_13b, "sweep33b": workload_sweep_33b,
               "decode7b": workload_decode_7b, "search7b": workload_search_7b, "domains13b": workload_domains_13b}
    names = [w for w in args.workloads.split(",") if w and w != "none"]
    for name in names:
        if name not in runners:
            raise SystemExit(f"unknown workload {name}; choose from {sorted(runners)}")
    # the 7B verifier of the headline serves decode7b and tree7b (which frees it)
    names = sorted(names, key=lambda w: {"decode7b": 0, "tree7b": 1}.get(w, 2))
    if "tree7b" not in names:
        if "decode7b" in names:
            log("workload decode7b")
            workloads["decode7b"] = workload_decode_7b(args, v7)
            names.remove("decode7b")
        _free(v7)
    for name in names:
        log(f"workload {name}")
        if name in ("tree7b", "decode7b"):
            workloads[name] = runners[name](args, v7)
        else:
            workloads[name] = runners[name](args)
        w = workloads[name]
        tok_s = w.get("accepted_tok_s")
        log(f"workload {name}: median {w['latency_us_median']:.0f} us"
            + (f", {tok_s:.0f} accepted tok/s" if tok_s is not None else ""))
    detail = {"by_skip": {str(k): v for k, v in res.items()}, "workloads": workloads, "roofline": roof,
              "cpu_baseline": cpu}
    if args.detail_out:
        with open(args.detail_out, "w") as fh:
            json.dump(detail, fh, indent=1)
        log(f"full results written to {args.detail_out}")

    def r(x, n=4):
        return None if x is None else float(f"{x:.{n}g}")

    by_skip = {str(k): {"skipped": v["skipped_layers"], "us": r(v["latency_us_median"]),
                        "us_p10_p90": [r(v["latency_us_p10"]), r(v["latency_us_p90"])],
                        "tok_s": r(v["accepted_tok_s"]), "tok_s_at_E": r(v["accepted_tok_s_at_expected"]),
                        "frac": r(v["roofline_frac"], 3),
                        **({"lat_ratio": r(v["latency_ratio_vs_dense"], 3), "byte_ratio": r(v["byte_ratio_vs_dense"], 3)}
                           if "latency_ratio_vs_dense" in v else {})}
               for k, v in res.items()}
    wl = {}
    for name, w in workloads.items():
        e = {"us": r(w.get("latency_us_median"))}
        for key, short in (("roofline_frac", "frac"), ("roofline_frac_median", "frac"), ("accepted_tok_s", "tok_s"),
                           ("us_per_skipped_layer", "us_per_skip"), ("packed_sweep_ms", "packed_ms"),
                           ("one_by_one_ms", "one_by_one_ms"), ("speedup", "speedup"),
                           ("sweep_speedup", "sweep_speedup")):
            if w.get(key) is not None:
                e[short] = r(w[key], 3)
        wl[name] = e
    out = {
        "metric": METRIC,
        "value": d0["accepted_tok_s"],
        "unit": "accepted tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": d0["wall_s"] / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "7B-shape decoder, chain k=5 (p=0.6), 1024-token paged context, dense mask",
                   "draft_pool": DRAFT_POOL, "parallelism": "single GPU"},
        "latency_us_median": r(d0["latency_us_median"]),
        "step_roofline_frac": r(d0["roofline_frac"], 3),
        "tok_s_at_expected_accept": r(d0["accepted_tok_s_at_expected"]),
        "roofline": None if roof is None else {k: (r(v) if isinstance(v, float) else v) for k, v in roof.items()
                                               if k not in ("launches",)},
        "cpu_baseline": None if cpu is None else {
            "value": r(cpu["value"]), "unit": cpu["unit"], "cores": cpu["cores"], "kind": cpu["kind"],
            "sample": "oracle 7B step extrapolated from a measured 4-block sample (numpy fp32); tiny step 1 thread",
            "host_cpus": cpu["host_cpus"], "blas": cpu["blas"], "ms": r(cpu["latency_ms_extrapolated"]),
            "tiny_1thread_ms": r(cpu["tiny_single_thread"]["latency_ms"])},
        "by_skip": by_skip,
        "workloads": wl,
    }
    print(json.dumps(out, separators=(",", ":")), flush=True)


if __name__ == "__main__":
    main()
