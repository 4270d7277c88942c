"""The test harness's own helpers (CPU): the threaded oracle pool build equals
the oracle's sequential one, and the tile selection names whole tiles."""
import numpy as np

import oracle
from paper_2504_03651_amd import workload as W
from tests.gpu_util import compact, oracle_pool, tile_queries


def test_threaded_pool_build_matches_sequential():
    for w in (W.config1(), W.random_case(41, num_rows=9, kv_dtype=W.KV_FP8, max_ctx=700),
              W.random_case(42, num_rows=12, num_q_heads=8, num_kv_heads=4, head_dim=64,
                            max_ctx=900, n_groups=3)):
        c, _ids = compact(w)
        a = oracle.prepare(c)
        for th in (1, 3, 8):
            b = oracle_pool(c, th)
            assert np.array_equal(a.k, b.k) and np.array_equal(a.v, b.v), (w.name, th)
            if a.fp8:
                assert np.array_equal(a.k_scale.view(np.uint32), b.k_scale.view(np.uint32))
                assert np.array_equal(a.v_scale.view(np.uint32), b.v_scale.view(np.uint32))


def test_tile_queries_cover_decode_rows_and_whole_tiles():
    w = W.random_case(43, num_rows=10, num_q_heads=12, num_kv_heads=2, head_dim=64,
                      max_ctx=500, max_q=200, values=False)
    sel = tile_queries(w)
    Hq = w.num_q_heads
    toks = set((sel // Hq).tolist())
    assert len(sel) == len(toks) * Hq
    qs, kind = w.batch.q_start, w.batch.row_kind
    bt = 256 // 6
    for r in range(w.batch.num_rows):
        t0, t1 = int(qs[r]), int(qs[r + 1])
        if kind[r] == W.DECODE:
            assert t0 in toks
            continue
        n = (t1 - t0 + bt - 1) // bt
        for k in {0, n // 2, n - 1}:
            assert set(range(t0 + k * bt, min(t1, t0 + (k + 1) * bt))) <= toks
