"""A seeded serving loop that feeds the iteration entry points from the KV
block manager (shared by the CPU and GPU tests; no GPU work here).

Each iteration finishes some running sequences, starts new ones (prompts drawn
from a few families that share long prefixes, so later prompts hit cached
blocks), forks a few running ones, and gives every other running sequence one
decode token.  The manager's block tables, sequence lengths and copy-on-write
pairs become one batch of the hot path: prefill rows carry the prompt tokens
the cache did not cover, decode rows one token.  K, V and Q of the new tokens
are seeded N(0, 1) bf16 draws (the serving loop has no model).
"""
from __future__ import annotations

from types import SimpleNamespace

import numpy as np

from paper_2504_03651_amd import kvm
from paper_2504_03651_amd import workload as W


def _bf16(rng, shape):
    x = rng.standard_normal(shape, dtype=np.float32)
    u = x.view(np.uint32)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def iterations(seed, num_blocks=48, offline_limit=36, num_q_heads=8, num_kv_heads=2,
               head_dim=64, n_iter=12):
    rng = np.random.default_rng(seed)
    m = kvm.KVManager(num_blocks, offline_limit)
    fams = [list(rng.integers(0, 1000, size=int(rng.integers(40, 120)))) for _ in range(4)]
    running = {}          # seq -> task
    nxt = 0
    for it in range(n_iter):
        for s in list(running):
            if rng.random() < 0.2:
                m.finish(s)
                del running[s]
        rows = []         # (seq, kind, new tokens)
        fresh = set()
        for _ in range(int(rng.integers(1, 4))):
            f = fams[int(rng.integers(len(fams)))]
            prompt = f[:int(rng.integers(17, len(f) + 1))] + \
                list(rng.integers(0, 1000, size=int(rng.integers(0, 40))))
            task = int(rng.integers(2))
            code, cached = m.start(nxt, task, prompt, check=False)
            if code == 0:
                running[nxt] = task
                fresh.add(nxt)
                rows.append((nxt, W.PREFILL, len(prompt) - cached))
            nxt += 1
        for s in [s for s in list(running) if s not in fresh]:
            if rng.random() < 0.15 and m.fork(s, nxt, check=False)[0] == 0:
                # the child's first token; one of parent and child copies the
                # shared partial block on its append
                running[nxt] = running[s]
                fresh.add(nxt)
                if m.append(nxt, [int(rng.integers(1000))], check=False)[0] == 0:
                    rows.append((nxt, W.DECODE, 1))
                else:
                    m.finish(nxt)
                    del running[nxt]
            nxt += 1
            if m.append(s, [int(rng.integers(1000))], check=False)[0] == 0:
                rows.append((s, W.DECODE, 1))
        pairs = m.take_copies().reshape(-1, 2)
        evicted = m.take_evictions()
        if not rows:
            m.tick()
            continue
        seqs = [r[0] for r in rows]
        mbr = 1
        while True:
            code, out = m.block_tables(seqs, mbr, check=False)
            if code == 0:
                break
            mbr *= 2
        bt, sl = out
        q = np.array([r[2] for r in rows], np.int32)
        batch = W.Batch(bt, sl, np.concatenate([[0], np.cumsum(q)]).astype(np.int32),
                        np.array([r[1] for r in rows], np.uint8))
        T = int(q.sum())
        yield SimpleNamespace(
            it=it, batch=batch, cow_pairs=pairs, evicted=evicted,
            q=_bf16(rng, (T, num_q_heads, head_dim)),
            k_new=_bf16(rng, (T, num_kv_heads, head_dim)),
            v_new=_bf16(rng, (T, num_kv_heads, head_dim)),
            num_blocks=num_blocks, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
            head_dim=head_dim, kv_dtype=W.KV_BF16, sm_scale=1.0 / float(np.sqrt(head_dim)),
            stats=m.stats())
        m.tick()
