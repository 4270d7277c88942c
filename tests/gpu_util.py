"""Shared helpers of the GPU parity tests (no GPU work at import time)."""
from __future__ import annotations

import copy
import sys

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
