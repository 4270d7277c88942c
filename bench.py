#!/usr/bin/env python3
"""Benchmark of one mixed serving iteration over a paged KV cache on one MI355X.

A step is the whole hot path on one synthetic batch: copy-on-write block
copies, KV append, then mixed attention (decode split-KV + prefill chunks +
merge), all through the C ABI on one stream.  Inputs are resident in HBM
before the timed region.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 2]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "mixed-iteration attention tokens/s; decode HBM GB/s and prefill MFMA % of peak"
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0    # MI355X dense bf16 MFMA

DESCRIPTIONS = {
    1: "tiny mixed batch: 2 decode + 2 prefill rows, MHA 4x64, 64-block pool",
    2: "decode-only offline batch: 256 rows, MHA 32x128, contexts U[512,2048], "
       "groups of 16 share a 1024-token prefix, 40,000-block pool",
    3: "mixed online/offline: 8 online decode + 1 prefill chunk (2048 on 1024) + "
       "128 offline decode sharing 512-token prefixes in groups of 32, GQA 32/8, D 128",
    4: "long-context: 32 rows at 32,768-token contexts, GQA 64/8, groups of 8 share "
       "16,384-token prefixes, 28 decode + 4 prefill chunks of 4,096",
    5: "config 3 at 4x batch with fp8-e4m3 KV and per-(block, head) fp32 scales",
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=2, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=0)
    return ap.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_baseline(w, threads):
    """The fp64 oracle on the host cores: the whole iteration when it is
    short, else a bounded sample of queries (stated in the record)."""
    import oracle
    from tests.gpu_util import compact
    c, _ = compact(w)
    t0 = time.perf_counter()
    pool = oracle.prepare(c)
    t_prep = time.perf_counter() - t0
    t0 = time.perf_counter()
    if c.cow_pairs.shape[0]:
        oracle.block_copy(pool, c.cow_pairs)
    oracle.kv_append(pool, c.batch, c.k_new, c.v_new)
    t_app = time.perf_counter() - t0
    T, Hq = c.batch.num_tokens, c.num_q_heads
    # estimate the cost of all queries from their key counts, sample if long
    q = np.diff(c.batch.q_start)
    klim = np.concatenate([c.batch.seq_lens[r] - q[r] + 1 + np.arange(q[r])
                           for r in range(c.batch.num_rows)])
    budget_keys = 1.5e8 * threads    # roughly 10-20 s of fp64 work
    total_keys = float(klim.sum()) * Hq
    if total_keys <= budget_keys:
        sel, frac, what = None, 1.0, "whole iteration (all queries)"
    else:
        g = np.random.Generator(np.random.PCG64(0))
        n = int(T * Hq * budget_keys / total_keys)
        sel = np.sort(g.choice(T * Hq, size=max(n, 1), replace=False)).astype(np.int32)
        frac = float(klim[sel // Hq].sum()) / float(klim.sum() * Hq)
        what = f"{len(sel)} of {T * Hq} query vectors ({frac:.3%} of the key work)"
    t0 = time.perf_counter()
    oracle.attention(pool, c.batch, c.q, Hq, c.sm_scale, sel=sel, threads=threads)
    t_attn = time.perf_counter() - t0
    t_iter = t_app + t_attn / frac
    return {"value": T / t_iter, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"append of the full batch + attention over {what}; time scaled to the "
                      f"whole iteration ({t_app:.2f} s append, {t_attn:.2f} s attention measured; "
                      f"pool build {t_prep:.1f} s not counted)"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the hot path "
              "shards by KV head or prefix group with no exchange, but this build runs on a "
              "single MI355X.", file=sys.stderr)
        return 2
    import torch
    from paper_2504_03651_amd import echo
    from paper_2504_03651_amd import workload as W
    from paper_2504_03651_amd.session import Iteration

    echo.lib()
    t0 = time.perf_counter()
    w = W.config(args.config)
    log(f"[bench] generated {w.name} in {time.perf_counter() - t0:.1f} s")
    it = Iteration(w)
    torch.cuda.synchronize()
    log("[bench] pool built on device")
    cp, cb, _ = echo.host_structs(w)
    st = echo.plan_stats(cp, cb, w.num_q_heads)

    for _ in range(args.warmup):
        it.step()
    torch.cuda.synchronize()
    log(f"[bench] {args.warmup} warmup steps done")

    stream = torch.cuda.current_stream()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    t_host = time.perf_counter()
    for k in range(args.steps):
        e = ev[k]
        e[0].record(stream)
        it.copy()
        e[1].record(stream)
        it.append()
        e[2].record(stream)
        it.attend()
        e[3].record(stream)
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_host
    ms = start.elapsed_time(stop) / args.steps
    t_copy = np.mean([e[0].elapsed_time(e[1]) for e in ev])
    t_app = np.mean([e[1].elapsed_time(e[2]) for e in ev])
    t_attn = np.mean([e[2].elapsed_time(e[3]) for e in ev])
    log(f"[bench] {args.steps} steps: {ms:.3f} ms/step (copy {t_copy:.3f}, append {t_app:.3f}, "
        f"attention {t_attn:.3f}); host wall {wall / args.steps * 1e3:.3f} ms/step")

    T, Hq, Hkv, D = w.batch.num_tokens, w.num_q_heads, w.num_kv_heads, w.head_dim
    eb = w.kv_bytes_per_elem()
    tok_bytes = 2 * Hkv * D * eb + (2 * Hkv * 4 if eb == 1 else 0) / 16
    q_out = T * Hq * D * (2 + 4)
    kv_unique = st["unique_kv_tokens"] * tok_bytes
    kv_logical = st["logical_kv_tokens"] * tok_bytes
    attn_bytes = kv_unique + q_out
    flops = 4.0 * Hq * D * st["causal_pairs"]
    achieved_gbs = attn_bytes / (t_attn * 1e-3) / 1e9
    achieved_tflops = flops / (t_attn * 1e-3) / 1e12
    hbm_time = attn_bytes / (HBM_PEAK_GBS * 1e9)
    mfma_time = flops / (BF16_PEAK_TFLOPS * 1e12)
    if hbm_time >= mfma_time:
        roof = {"bound": "hbm", "achieved": round(achieved_gbs, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved_gbs / HBM_PEAK_GBS, 4)}
    else:
        roof = {"bound": "mfma", "achieved": round(achieved_tflops, 1), "peak": BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved_tflops / BF16_PEAK_TFLOPS, 4)}
    roof["traffic"] = None
    roof["kernel"] = "echo_attn_mixed (plan upload + attn_items_kernel + merge_kernel)"
    roof["algorithmic_bytes"] = int(attn_bytes)
    roof["algorithmic_flops"] = int(flops)
    roof["avg_ms"] = round(float(t_attn), 4)

    rec = {"metric": METRIC, "value": round(T / (ms * 1e-3), 1), "unit": "tokens/s",
           "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16" if eb == 2 else "bf16 (fp8-e4m3 KV)",
           "data": "synthetic",
           "config": {"workload": f"{w.name}: {DESCRIPTIONS[args.config]}",
                      "rows": w.batch.num_rows, "query_tokens": T, "q_heads": Hq,
                      "kv_heads": Hkv, "head_dim": D, "pool_blocks": w.num_blocks,
                      "cow_pairs": int(w.cow_pairs.shape[0])},
           "roofline": roof,
           "kernels_ms": {"block_copy": round(float(t_copy), 4), "kv_append": round(float(t_app), 4),
                          "attention": round(float(t_attn), 4)},
           "decode_gbs": {"unique": round(achieved_gbs, 1),
                          "logical": round((kv_logical + q_out) / (t_attn * 1e-3) / 1e9, 1)},
           "attention_tflops": round(achieved_tflops, 2),
           "plan": st}
    if not args.no_cpu_baseline:
        threads = args.cpu_threads or min(16, os.cpu_count() or 1)
        log(f"[bench] timing the oracle on {threads} host threads")
        rec["cpu_baseline"] = cpu_baseline(w, threads)
    print(json.dumps(rec), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
