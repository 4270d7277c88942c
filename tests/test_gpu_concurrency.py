"""Concurrent callers: several host threads, each on its own stream.

Each thread owns a pool, a workspace and a stream (default priority) and
repeats its iteration; the library is entered from all threads at once (the
binding releases the interpreter lock during calls), so the per-thread plan
buffers, each thread's pinned host-workspace ring and the per-thread timing
state are exercised under contention.  Every thread's final pool and outputs must match the
oracle, as in the single-stream parity tests.
"""
import threading

import numpy as np
import pytest

import oracle
from paper_2504_03651_amd import workload as W
from tests.gpu_util import ATOL, attn_error, same_pool, say

pytestmark = pytest.mark.gpu


def test_threads_on_separate_streams():
    import torch
    from paper_2504_03651_amd import echo
    from paper_2504_03651_amd.session import Iteration
    assert torch.cuda.is_available()
    echo.lib()
    cases = [W.random_case(300 + i, num_rows=7, num_q_heads=8, num_kv_heads=2, head_dim=128,
                           kv_dtype=W.KV_FP8 if i % 2 else W.KV_BF16, max_ctx=900, max_q=70)
             for i in range(4)]
    say(f"[case] {len(cases)} threads x 6 steps on separate streams")
    results, errors = [None] * len(cases), []

    def run(i):
        try:
            torch.cuda.set_device(0)
            stream = torch.cuda.Stream()
            with torch.cuda.stream(stream):
                it = Iteration(cases[i])
                for _ in range(6):
                    it.step()
                stream.synchronize()
                results[i] = (it.pool_host(), it.out.cpu().numpy())
        except Exception as e:  # reported below, after every thread has ended
            errors.append((i, repr(e)))

    threads = [threading.Thread(target=run, args=(i,)) for i in range(len(cases))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a thread did not finish"
    assert not errors, errors
    for w, (pool_dev, out) in zip(cases, results):
        pool, ref = oracle.run_iteration(w)
        same_pool(pool_dev, pool)
        err, _ = attn_error(out.reshape(ref.shape), ref)
        say(f"       {w.name}: max abs err {err:.3e}")
        assert err <= ATOL
