"""The scheduler simulation with its batches executed on the GPU.

Hundreds of iterations of the KV-cache-aware scheduler (Echo policy) drive
echo_kv_append + echo_attn_mixed with the block manager's own tables:
prefix hits, evictions and recompute preemptions reach the kernels.  Every
call must succeed and produce finite outputs, and the calibrated estimator's
prediction of each iteration's append + attention time is compared with the
measured one."""
import numpy as np
import pytest

from paper_2504_03651_amd import scheduler as S
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


def test_scheduler_batches_run_on_the_gpu():
    import torch
    from paper_2504_03651_amd.engine import AttentionEngine
    nb = 2500
    eng = AttentionEngine(nb)
    reqs = S.synthetic_trace(5, n_online=30, n_offline=150, rate_per_s=15, groups=8)
    sim = S.Simulator(nb, policy="echo", max_batch=64, candidates=16, engine=eng)
    say(f"[case] scheduler + engine: {nb} blocks, {len(reqs)} requests")
    st = sim.run(reqs, horizon_ms=3000)
    log = np.array([(e, m, k) for e, m, rows, tok, k in sim.engine_log])
    rel = np.abs(log[:, 0] - log[:, 1]) / log[:, 1]
    relk = np.abs(log[:, 2] - log[:, 1]) / log[:, 1]
    say(f"       {st.iterations} iterations on the GPU, {st.preemptions} preemptions, "
        f"prefix hits {sum(r.cached_tokens for r in reqs)} tokens; GPU time vs estimate: "
        f"paper form median rel err {np.median(rel):.3f} (estimate/measured "
        f"{np.median(log[:, 0] / log[:, 1]):.3f}), kernel form {np.median(relk):.3f} "
        f"({np.median(log[:, 2] / log[:, 1]):.3f})")
    assert eng.calls == st.iterations >= 100
    assert sum(r.cached_tokens for r in reqs) > 0
    assert torch.isfinite(eng.last_out).all()
    assert np.median(relk) < 0.35
