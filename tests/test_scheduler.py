"""The KV-cache-aware scheduler simulation (CPU): the selection rule of
Section 4.1 (an offline request whose prefix is cached beats the next one in
pool order), the mu + 2 sigma threshold of Section 5.3 applied to the
manager, online requests preempting offline work, pausing offline decodes to
meet an online deadline, and Echo's policy against first-come first-served on
a seeded synthetic trace."""
import math

import numpy as np
import pytest

from paper_2504_03651_amd import scheduler as S
from paper_2504_03651_amd.kvm import OFFLINE, ONLINE


def _doc(tag, n):
    return [tag * 1000 + i for i in range(n)]


def test_cached_prefix_is_chosen_over_pool_order():
    for policy, expect in (("echo", 5), ("fcfs", 1)):
        sim = S.Simulator(400, policy=policy, prefill_budget=600, max_batch=64)
        # R2 runs first and leaves its document's blocks cached
        r2 = S.Request(2, OFFLINE, _doc(2, 512) + [1, 2, 3], 2)
        sim.run([r2])
        assert r2.done
        pool = [S.Request(1, OFFLINE, _doc(1, 512) + [4], 2),
                S.Request(5, OFFLINE, _doc(2, 512) + [7, 8], 2),
                S.Request(3, OFFLINE, _doc(3, 512) + [5], 2)]
        for r in pool:
            sim.m.register_offline(r.rid, r.prompt)
        running = []
        batch = sim.step([], pool, running)
        # with room for one start this iteration, Echo takes R5 (its 512-token
        # document is cached: 3 tokens to compute); first come first served
        # takes R1
        assert batch[0][0].rid == expect, (policy, [(e[0].rid, e[2]) for e in batch])
        if policy == "echo":
            assert batch[0][2] < 16


def test_threshold_is_mean_plus_two_sigma():
    sim = S.Simulator(200, policy="echo")
    sim.online_use = [10, 20, 30]
    sim._set_threshold()
    limit = 200 - math.ceil(20 + 2 * np.std([10, 20, 30]))   # 200 - 37
    # an offline start of limit + 1 blocks is refused, one of limit blocks fits
    assert sim.m.start(1, OFFLINE, list(range(16 * (limit + 1))), check=False)[0] == -7
    assert sim.m.start(2, OFFLINE, list(range(16 * limit)), check=False)[0] == 0


def test_online_arrival_preempts_offline_work():
    sim = S.Simulator(64, policy="fcfs", max_batch=64)
    offline = [S.Request(i, OFFLINE, _doc(10 + i, 16 * 20), 50) for i in range(3)]
    online = S.Request(99, ONLINE, _doc(50, 16 * 20), 4, arrival=5.0, ttft_slo=1e9, tpot_slo=1e9)
    st = sim.run(offline + [online], horizon_ms=1e6)
    assert online.done and all(r.done for r in offline)
    assert st.preemptions >= 1 and st.recomputed_tokens > 0


def test_offline_decodes_pause_for_a_tight_deadline():
    sim = S.Simulator(12000, policy="fcfs", max_batch=128)
    offline = [S.Request(i, OFFLINE, _doc(10 + i, 1000), 400) for i in range(120)]
    # online requests whose per-token deadline is below the full batch's time
    online = [S.Request(1000 + i, ONLINE, _doc(700 + i, 64), 40, arrival=2000.0 + 50 * i,
                        ttft_slo=20.0, tpot_slo=3.0) for i in range(5)]
    probe = [S.Request(i, OFFLINE, [0], 1, computed=1000) for i in range(120)]
    assert sim._time([(r, "decode", 1) for r in probe]) > 3.0   # a full decode batch
    st = sim.run(offline + online, horizon_ms=4000)
    assert st.paused > 0
    assert all(r.done for r in online)


def test_echo_beats_first_come_first_served_on_a_trace():
    out = {}
    for policy in ("fcfs", "echo"):
        reqs = S.synthetic_trace(3, n_online=40, n_offline=300, rate_per_s=10, groups=10)
        sim = S.Simulator(1500, policy=policy, max_batch=64, candidates=16)
        out[policy] = S.summary(reqs, sim.run(reqs, horizon_ms=5000))
    e, f = out["echo"], out["fcfs"]
    assert e["offline_goodput_tokens_per_s"] > 1.2 * f["offline_goodput_tokens_per_s"], out
    assert e["online_slo_attainment"] >= f["online_slo_attainment"] - 0.02, out
    assert e["recomputed_tokens"] < f["recomputed_tokens"], out
