"""Shared helpers of the GPU parity tests (no GPU work at import time)."""
from __future__ import annotations

import copy
import os
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle
from paper_2504_03651_amd import workload as W

# Attention tolerance: bf16 operands, fp32 accumulation, probabilities
# rounded to bf16 for the PV product (relative 2^-9 per weight), so outputs
# that are convex combinations of O(1) values carry errors of a few 1e-3.
ATOL = 1e-2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def compact(w):
    """Copy of ``w`` whose pool holds only the blocks it touches, renumbered
    0..n-1 in ascending id order (placement does not change any result), plus
    the original ids so that device blocks can be gathered in that order."""
    ids = set(int(b) for b in w.used_blocks)
    ids.update(int(b) for b in w.ctx.block_tables.ravel())
    ids.update(int(b) for b in np.asarray(w.cow_pairs).ravel())
    ids = np.array(sorted(ids), dtype=np.int64)
    lut = np.full(w.num_blocks, -1, np.int64)
    lut[ids] = np.arange(len(ids))

    def remap(bt):
        out = np.where(bt >= 0, lut[np.maximum(bt, 0)], -1)
        return out.astype(np.int32)

    c = copy.copy(w)
    c.batch = W.Batch(remap(w.batch.block_tables), w.batch.seq_lens, w.batch.q_start,
                      w.batch.row_kind)
    c.ctx = W.Batch(remap(w.ctx.block_tables), w.ctx.seq_lens, w.ctx.q_start, w.ctx.row_kind)
    c.cow_pairs = remap(np.asarray(w.cow_pairs)).reshape(-1, 2)
    c.num_blocks = int(len(ids))
    return c, ids


def same_pool(gpu, orc):
    """Bitwise comparison of (K, V, k_scale, v_scale) host arrays."""
    gk, gv, gks, gvs = gpu
    assert np.array_equal(gk, orc.k), "K codes differ"
    assert np.array_equal(gv, orc.v), "V codes differ"
    if orc.fp8:
        assert np.array_equal(gks.view(np.uint32), orc.k_scale.view(np.uint32)), "K scales differ"
        assert np.array_equal(gvs.view(np.uint32), orc.v_scale.view(np.uint32)), "V scales differ"


def attn_error(got, ref):
    err = np.abs(got.astype(np.float64) - ref)
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 1.0
    return float(err.max()) if err.size else 0.0, float(err.max() / rms) if err.size else 0.0


def sample_queries(w, n, seed=0):
    """Query indices t*Hq + h: every prefill chunk's first and last token,
    plus n random ones."""
    g = np.random.Generator(np.random.PCG64(seed))
    T, Hq = w.batch.num_tokens, w.num_q_heads
    picks = set(int(x) for x in g.integers(0, T * Hq, size=n))
    qs = w.batch.q_start
    for r in range(w.batch.num_rows):
        for t in (int(qs[r]), int(qs[r + 1]) - 1):
            for h in (0, Hq - 1):
                picks.add(t * Hq + h)
    return np.array(sorted(picks), dtype=np.int32)


def cpu_share() -> int:
    """Host threads this process may use: its CPU affinity, capped by the
    cgroup's CPU quota when one is set."""
    n = len(os.sched_getaffinity(0))
    try:
        with open("/sys/fs/cgroup/cpu.max") as f:
            quota, period = f.read().split()[:2]
        if quota != "max":
            n = min(n, max(1, int(quota) // int(period)))
    except (OSError, ValueError):
        pass
    return max(1, n)


def oracle_pool(c, threads=None):
    """``oracle.prepare(c)`` with the context append spread over host threads.
    The context batch has one pseudo-row per physical block, so its rows write
    disjoint blocks and any split of them gives the same pool."""
    ctx = c.ctx
    B = ctx.num_rows
    ids = ctx.block_tables[:, 0]
    assert len(np.unique(ids)) == B, "context rows must write disjoint blocks"
    pool = oracle.Pool(c.num_blocks, c.num_kv_heads, c.head_dim, c.kv_dtype != W.KV_BF16)
    threads = threads or cpu_share()
    cuts = np.linspace(0, B, min(threads, max(B, 1)) + 1).astype(np.int64)
    qs = ctx.q_start

    def part(i):
        r0, r1 = int(cuts[i]), int(cuts[i + 1])
        if r1 <= r0:
            return
        sub = W.Batch(ctx.block_tables[r0:r1], ctx.seq_lens[r0:r1],
                      (qs[r0:r1 + 1] - qs[r0]).astype(np.int32), ctx.row_kind[r0:r1])
        t0, t1 = int(qs[r0]), int(qs[r1])
        oracle.kv_append(pool, sub, c.ctx_k[t0:t1], c.ctx_v[t0:t1])

    with ThreadPoolExecutor(len(cuts) - 1) as ex:
        list(ex.map(part, range(len(cuts) - 1)))
    return pool


def tile_queries(w, tiles_per_chunk=3):
    """Query indices t*Hq + h of every decode token and of whole prefill
    tiles (all query heads of 256 / G consecutive tokens, the tiles of the
    prefill kernel): the first, middle and last tile of every chunk."""
    Hq, Hkv = w.num_q_heads, w.num_kv_heads
    bt = max(1, 256 // (Hq // Hkv))
    qs, kind = w.batch.q_start, w.batch.row_kind
    toks = []
    for r in range(w.batch.num_rows):
        t0, t1 = int(qs[r]), int(qs[r + 1])
        if kind[r] == W.DECODE:
            toks.append(np.arange(t0, t1))
            continue
        n = (t1 - t0 + bt - 1) // bt
        for k in sorted({0, n // 2, n - 1} if tiles_per_chunk >= 3 else {0, n - 1}):
            toks.append(np.arange(t0 + k * bt, min(t1, t0 + (k + 1) * bt)))
    toks = np.unique(np.concatenate(toks))
    return (toks[:, None] * Hq + np.arange(Hq)[None, :]).ravel().astype(np.int32)
