"""Benchmark of the sparse-depth verification step on one MI355X.

Workload: 7B-shape decoder (32 layers, d 4096, 32 heads x 128, FFN 11008,
vocab 32000), bf16 random-init N(0, 0.02) weights, one sequence with a
1024-token uniform-random context in paged KV (16-token pages), chain drafts
of k=5 where each drafted token equals the target's greedy token with
probability 0.6, skip masks of 0, 4 and 8 layers drawn from layers 16-31
(nested).  One step is one blocking tss_verify (embedding, every active block,
lm_head, argmax and accept scan) with commit, followed by a rewind of the
sequence to its 1024-token context.

Prints one JSON line.  value = accepted tokens/s of the dense verifier
(sum(accept_len + 1) / sum(step latency)); the skip-4 and skip-8 figures are
in "by_skip".
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


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(shape, active, n_ctx, M):
    """Bytes one verify must move: active blocks' bf16 weights, their KV read
    and write, norm gains; lm_head, embedding rows, final norm and logits."""
    d, f, v = shape.d_model, shape.ffn_dim, shape.vocab
    per_layer = 2 * (4 * d * d + 3 * d * f) + 4 * d * n_ctx + 4 * d * M + 4 * d
    return active * per_layer + 2 * v * d + 2 * M * d + 2 * d + 4 * M * v


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
    v = Verifier(shape, n_seqs=1, max_tokens=CTX + 64, max_nodes=64, device="cuda:0")
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
                  for i in range(args.warmup + args.steps)]
        def timed(n_steps, tag, after_warmup=None):
            for i in range(args.warmup):
                v.verify(0, drafts[i], commit=True)
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
                al, _ = v.verify(0, drafts[args.warmup + i], commit=True)
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
        results[s] = {
            "skipped_layers": np.nonzero(mask)[0].tolist(),
            "latency_us_median": med * 1e6,
            "latency_us_p10": float(np.percentile(lat, 10)) * 1e6,
            "latency_us_p90": float(np.percentile(lat, 90)) * 1e6,
            "accepted_tok_s": float((acc + 1).sum() / lat.sum()),
            "mean_accept_len": float(acc.mean()),
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
    v.close()
    return shape, results, prof


def cpu_baseline(args, shape, gpu_accept_mean):
    """The oracle, untouched, on a bounded sample: the 7B verify step with two
    of the 32 blocks active (KV for the 1024-token context from the oracle's
    own prefill of those blocks, not timed) and with every block skipped;
    per-block time x 32 + the block-free time gives the dense step."""
    from threadpoolctl import threadpool_info

    from oracle import OracleModel, OracleSequence, prefill, verify

    cache = {}

    def get(name, layer):
        if (name, layer) not in cache:
            cache[(name, layer)] = synth.weight_tensor(shape, name, layer)
        return cache[(name, layer)]
    m = OracleModel(shape, get)
    toks = synth.context_tokens(shape.vocab, CTX + 1)
    ctx, root = toks[:CTX], int(toks[CTX])
    two = np.ones(shape.n_layers, np.uint8)
    two[[0, 1]] = 0
    seq = OracleSequence(m, two)
    t = time.time()
    prefill(m, seq, ctx)
    log(f"oracle prefill of 2 blocks: {time.time() - t:.1f}s")
    tokens = np.concatenate([[root], synth.context_tokens(shape.vocab, K_DRAFT, stream=7)])
    none = np.ones(shape.n_layers, np.uint8)

    def timed(mask, reps):
        verify(m, seq, tokens, mask=mask)
        best = []
        for _ in range(reps):
            a = time.perf_counter()
            verify(m, seq, tokens, mask=mask)
            best.append(time.perf_counter() - a)
        return float(np.median(best))
    t2 = timed(two, args.cpu_reps)
    t0 = timed(none, args.cpu_reps)
    per_block = (t2 - t0) / 2
    dense = t0 + shape.n_layers * per_block
    threads = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    return {
        "value": (gpu_accept_mean + 1) / dense,
        "unit": "accepted tok/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": (f"oracle verify of the 7B chain k=5 step at context 1024 with blocks 0-1 active "
                   f"({t2 * 1e3:.0f} ms) and with all blocks skipped ({t0 * 1e3:.0f} ms), median of "
                   f"{args.cpu_reps}; dense latency extrapolated as skipped-time + 32 x per-block = "
                   f"{dense * 1e3:.0f} ms; accepted tokens per step taken from the GPU run's mean"),
        "latency_ms_extrapolated": dense * 1e3,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--cpu-reps", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--skips", default="0,4,8", help="skip counts to time; the first is the headline")
    ap.add_argument("--calib-copy", type=float, default=0.0,
                    help="GiB of a plain device copy run first (HBM counter calibration)")
    args = ap.parse_args()
    args.skips = [int(x) for x in args.skips.split(",")]
    if args.skips[0] != 0 or any(x not in SKIPS for x in args.skips):
        raise SystemExit(f"--skips must start with 0 and use counts from {SKIPS}")
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported by this build "
              "(the verify step runs on a single MI355X)", file=sys.stderr)
        sys.exit(2)
    shape, res, prof = run_gpu(args)
    d0 = res[0]
    M = K_DRAFT + 1
    roof = None
    if prof and prof[1] > 0:
        avg_s = prof[0] / prof[1] / 1e3
        gb = gateup_bytes(shape, M)
        achieved = gb / avg_s / 1e9
        roof = {"kernel": "gate/up projection + SwiGLU (layer 0, dense)", "bound": "hbm",
                "achieved": achieved, "peak": PEAK_HBM / 1e9, "unit": "GB/s", "frac": achieved / (PEAK_HBM / 1e9),
                "traffic": None, "avg_launch_us": avg_s * 1e6, "launches": prof[1],
                "algorithmic_bytes_per_launch": gb}
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args, shape, d0["mean_accept_len"])
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
                   "context": CTX, "k": K_DRAFT, "p_accept": P_ACCEPT, "page_tokens": 16,
                   "skip_counts": args.skips, "parallelism": "single GPU"},
        "latency_us_median": d0["latency_us_median"],
        "step_roofline_frac": d0["roofline_frac"],
        "roofline": roof,
        "cpu_baseline": cpu,
        "by_skip": {str(k): v for k, v in res.items()},
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
