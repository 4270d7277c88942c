"""The KV block manager driving the HIP iteration over several iterations.

One device pool and one oracle pool live through a seeded serving loop
(tests/kvm_serving.py): each iteration's copy-on-write pairs, appends and
attention come from the manager's block tables.  After every iteration the
device pool must equal the oracle's bit for bit and the attention outputs must
match within the attention tolerance, so prefix hits (rows reading blocks an
earlier sequence wrote), forks (copied partial blocks) and evicted-then-reused
blocks all reach the kernels.
"""
import numpy as np
import pytest

import oracle
from tests import kvm_serving
from tests.gpu_util import ATOL, attn_error, same_pool, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed", [0, 2])
def test_serving_loop_matches_the_oracle(seed):
    import torch
    from paper_2504_03651_amd import echo
    assert torch.cuda.is_available()
    echo.lib()
    pool = opool = None
    n = 0
    for w in kvm_serving.iterations(seed):
        say(f"[case] serving seed {seed} iteration {w.it}: rows {w.batch.num_rows}, "
            f"tokens {w.batch.num_tokens}, copies {len(w.cow_pairs)}, evicted {len(w.evicted)}")
        if pool is None:
            pool = echo.KVPool(w.num_blocks, w.num_kv_heads, w.head_dim, False).poison()
            opool = oracle.Pool(w.num_blocks, w.num_kv_heads, w.head_dim, False)
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()
        batch = echo.DeviceBatch(w.batch)
        if len(w.cow_pairs):
            pairs = np.ascontiguousarray(w.cow_pairs, np.int32)
            echo.block_copy(pool, torch.from_numpy(pairs).cuda(), pairs)
            oracle.block_copy(opool, pairs)
        echo.kv_append(pool, batch, dev(w.k_new), dev(w.v_new))
        oracle.kv_append(opool, w.batch, w.k_new, w.v_new)
        out = torch.zeros((w.batch.num_tokens, w.num_q_heads, w.head_dim), dtype=torch.float32,
                          device="cuda")
        ws = torch.empty(echo.workspace_bytes(pool, batch, w.num_q_heads), dtype=torch.uint8,
                         device="cuda")
        echo.attn_mixed(pool, batch, dev(w.q), w.num_q_heads, w.sm_scale, out, ws)
        torch.cuda.synchronize()
        ref = oracle.attention(opool, w.batch, w.q, w.num_q_heads, w.sm_scale)
        same_pool((pool.k.cpu().numpy().view(np.uint16), pool.v.cpu().numpy().view(np.uint16),
                   None, None), opool)
        err, _ = attn_error(out.cpu().numpy().reshape(ref.shape), ref)
        assert err <= ATOL, (w.it, err)
        n += 1
    say(f"       {n} iterations, manager {w.stats}")
    assert n >= 8 and w.stats["hits_tokens"] > 0
