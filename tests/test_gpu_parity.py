"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Append and block copy must match bit for bit (whole pools for small cases,
every block the batch touches for full-size ones).  Attention outputs must
stay within ATOL (max abs error) of the oracle: all outputs for small and
fuzzed cases and for the full-size decode-only and mixed configurations; for
the long-context and e4m3 configurations every decode output and whole
prefill tiles (first, middle and last of every chunk).  Both planning modes
run: with host mirrors (host plan, prefix groups) and without (device plan).
"""
import numpy as np
import pytest

import oracle
from paper_2504_03651_amd import workload as W
from tests.gpu_util import (ATOL, attn_error, compact, cpu_share, oracle_pool, same_pool,
                            sample_queries, say, tile_queries)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "no GPU"
    from paper_2504_03651_amd import echo
    echo.lib()
    return torch


def _run(w, torch, mirrors=True):
    from paper_2504_03651_amd.session import Iteration
    it = Iteration(w, mirrors=mirrors)
    it.step()
    torch.cuda.synchronize()
    return it


def _check_small(w, torch, label):
    say(f"[case] {label}: rows={w.batch.num_rows} T={w.batch.num_tokens} "
        f"Hq={w.num_q_heads} Hkv={w.num_kv_heads} D={w.head_dim} kv={w.kv_dtype}")
    it = _run(w, torch)
    pool, ref = oracle.run_iteration(w)
    same_pool(it.pool_host(), pool)
    got = it.out.cpu().numpy().reshape(ref.shape)
    assert not np.isnan(got).any()
    err, nerr = attn_error(got, ref)
    say(f"       max abs err {err:.3e}  normalised {nerr:.3e}")
    assert err <= ATOL
    return it, got


def test_config1(torch_cuda):
    _check_small(W.config1(), torch_cuda, "config1")


def test_config1_prefix_shared_with_prefill_row(torch_cuda):
    _check_small(W.config1(share_with_prefill=True), torch_cuda, "config1-share-prefill")


FUZZ = [
    # seed, rows, Hq, Hkv, D, kv, max_ctx, max_q
    (101, 6, 8, 2, 128, W.KV_BF16, 600, 80),
    (102, 8, 4, 4, 64, W.KV_BF16, 900, 40),
    (103, 5, 8, 1, 128, W.KV_BF16, 500, 120),
    (104, 7, 32, 8, 128, W.KV_BF16, 1200, 60),
    (105, 6, 64, 8, 64, W.KV_BF16, 700, 50),
    (106, 6, 8, 2, 128, W.KV_FP8, 600, 80),
    (107, 6, 4, 4, 64, W.KV_FP8, 800, 33),
    (108, 9, 16, 16, 128, W.KV_BF16, 5000, 300),
    (109, 6, 32, 1, 128, W.KV_BF16, 400, 40),
]


@pytest.mark.parametrize("case", FUZZ, ids=[f"seed{c[0]}" for c in FUZZ])
def test_fuzz(torch_cuda, case):
    seed, rows, hq, hkv, d, kv, mc, mq = case
    w = W.random_case(seed, num_rows=rows, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                      kv_dtype=kv, max_ctx=mc, max_q=mq, n_groups=2)
    _check_small(w, torch_cuda, f"fuzz{seed}")


def test_edge_rows(torch_cuda):
    rows = [W.RowSpec(W.DECODE, 0, 1), W.RowSpec(W.DECODE, 16, 1, 0), W.RowSpec(W.DECODE, 17, 1, 0),
            W.RowSpec(W.DECODE, 31, 1, 0), W.RowSpec(W.PREFILL, 0, 1), W.RowSpec(W.PREFILL, 15, 17),
            W.RowSpec(W.PREFILL, 33, 300), W.RowSpec(W.DECODE, 1023, 1, 1),
            W.RowSpec(W.DECODE, 1024, 1, 1), W.RowSpec(W.DECODE, 1025, 1, 1)]
    w = W.build("edges", rows, {0: 16, 1: 1024}, 8, 2, 128, num_blocks=512, seed=9)
    _check_small(w, torch_cuda, "edge-rows")


@pytest.mark.parametrize("kv", [W.KV_BF16, W.KV_FP8])
def test_many_rows(torch_cuda, kv):
    # more rows than the append kernel scans per LDS window (4096)
    w = W.random_case(114, num_rows=4500, num_q_heads=4, num_kv_heads=2, head_dim=64,
                      kv_dtype=kv, max_ctx=60, max_q=20, n_groups=3)
    _check_small(w, torch_cuda, f"many-rows-{kv}")


def _bf16_doubled(bits):
    """bf16 bit patterns of twice the values (exact)."""
    x = (bits.astype(np.uint32) << 16).view(np.float32) * np.float32(2.0)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def test_fp8_queries_seeing_few_keys(torch_cuda):
    # The first queries of prefill chunks that start at position 0 see one or
    # two keys, so their outputs are single V values.  An e4m3 value times its
    # block scale is not bf16-exact; with V doubled (|v| up to about 10) a
    # bf16 P.V operand would be off by up to 2^-9 |v|, beyond the tolerance.
    rows = [W.RowSpec(W.PREFILL, 0, 40), W.RowSpec(W.PREFILL, 0, 3), W.RowSpec(W.DECODE, 0, 1),
            W.RowSpec(W.PREFILL, 0, 17)]
    w = W.build("fp8-few-keys", rows, {}, 16, 4, 128, kv_dtype=W.KV_FP8, seed=23)
    w.v_new = _bf16_doubled(w.v_new)
    _check_small(w, torch_cuda, "fp8-few-keys")


def _bf16_scaled(bits, factor):
    """bf16 bit patterns of the values times a power of two (exact)."""
    x = (bits.astype(np.uint32) << 16).view(np.float32) * np.float32(factor)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def test_fp8_prefill_values_near_the_fp16_range(torch_cuda):
    # chunked prefill over an e4m3 pool carries V times its block scale in
    # fp16: values up to the header's +-65504 stay finite.  V is N(0, 1) times
    # 2^13 (largest |v| about 4e4), so outputs and their rounding scale by
    # 2^13 as well: the bar is ATOL times that factor
    rows = [W.RowSpec(W.PREFILL, 0, 200), W.RowSpec(W.PREFILL, 300, 64), W.RowSpec(W.DECODE, 500, 1),
            W.RowSpec(W.PREFILL, 1000, 17)]
    w = W.build("fp8-large-v", rows, {}, 16, 4, 128, kv_dtype=W.KV_FP8, seed=29)
    f = 2.0 ** 13
    w.v_new = _bf16_scaled(w.v_new, f)
    w.ctx_v = _bf16_scaled(w.ctx_v, f)
    vmax = float(np.abs((w.v_new.astype(np.uint32) << 16).view(np.float32)).max())
    say(f"[case] fp8 prefill with |V| up to {vmax:.0f}")
    assert 2.0e4 < vmax < 65504.0
    it = _run(w, torch_cuda)
    pool, ref = oracle.run_iteration(w)
    same_pool(it.pool_host(), pool)
    got = it.out.cpu().numpy().reshape(ref.shape)
    assert np.isfinite(got).all()
    err, nerr = attn_error(got, ref)
    say(f"       max abs err {err:.3e} (bar {ATOL * f:.1f})  normalised {nerr:.3e}")
    assert err <= ATOL * f


@pytest.mark.parametrize("log2f", [-12, 6])
def test_fp8_prefill_v_scales(torch_cuda, log2f):
    # The e4m3 prefill widens V codes with the power-of-two part of the block
    # scale and multiplies by its mantissa in fp16.  V times 2^-12 and 2^6 (on
    # N(0, 1) data the scales sit near 2^-7) moves the scales' exponents to
    # about 2^-19 and 2^-1; outputs scale with V, and so does the bar
    rows = [W.RowSpec(W.PREFILL, 0, 120), W.RowSpec(W.PREFILL, 200, 64), W.RowSpec(W.DECODE, 300, 1),
            W.RowSpec(W.PREFILL, 700, 33)]
    w = W.build(f"fp8-v-2^{log2f}", rows, {}, 16, 4, 128, kv_dtype=W.KV_FP8, seed=41)
    f = 2.0 ** log2f
    w.v_new = _bf16_scaled(w.v_new, f)
    w.ctx_v = _bf16_scaled(w.ctx_v, f)
    say(f"[case] fp8 prefill with V x 2^{log2f}")
    it = _run(w, torch_cuda)
    pool, ref = oracle.run_iteration(w)
    same_pool(it.pool_host(), pool)
    got = it.out.cpu().numpy().reshape(ref.shape)
    assert np.isfinite(got).all()
    err, nerr = attn_error(got, ref)
    say(f"       max abs err {err:.3e} (bar {ATOL * f:.3e})  normalised {nerr:.3e}")
    assert err <= ATOL * f


LARGE_LOGITS = [
    # seed, Hq, Hkv, D, kv, query factor
    (131, 8, 2, 128, W.KV_BF16, 4.0),
    (132, 8, 2, 128, W.KV_BF16, 16.0),
    (133, 16, 4, 64, W.KV_BF16, 16.0),
    (134, 8, 2, 128, W.KV_FP8, 16.0),
]


@pytest.mark.parametrize("case", LARGE_LOGITS, ids=[f"seed{c[0]}-x{int(c[5])}" for c in LARGE_LOGITS])
def test_large_logits(torch_cuda, case):
    # Queries times 4 and 16 (exact in bf16): logits 4 and 16 times those of
    # N(0, 1) data, softmax rows from flat to nearly one-hot.  Scores are
    # scaled in fp32 after the product, so the error bound does not grow with
    # the logits' magnitude (rounding q * scale to bf16 first would put up to
    # 2^-9 |logit| into every exponent: beyond the bar at these sizes).
    seed, hq, hkv, d, kv, f = case
    w = W.random_case(seed, num_rows=8, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                      kv_dtype=kv, max_ctx=900, max_q=150, n_groups=2, prefill_frac=0.5)
    w.q = _bf16_scaled(w.q, f)
    _check_small(w, torch_cuda, f"large-logits-{seed}-x{f:g}")


@pytest.mark.parametrize("log2f", [-120, -90, 100, 110])
def test_fp8_append_scales_at_the_range_edges(torch_cuda, log2f):
    # The e4m3 append takes x / s from a reciprocal and one correction for
    # tile scales s in [2^-100, 2^100] and divides outside.  K and V (new and
    # cached) times 2^log2f put the scales (about amax / 448, amax ~ 3-4 times
    # the factor) below 2^-100 (a subnormal scale at 2^-120), just inside the
    # low edge, inside the high edge and above it; codes and scales must equal
    # the oracle's bit for bit
    rows = [W.RowSpec(W.PREFILL, 0, 40), W.RowSpec(W.DECODE, 20, 1), W.RowSpec(W.PREFILL, 16, 33),
            W.RowSpec(W.DECODE, 47, 1)]
    w = W.build(f"fp8-scale-2^{log2f}", rows, {}, 8, 2, 128, kv_dtype=W.KV_FP8, seed=37)
    for name in ("k_new", "v_new", "ctx_k", "ctx_v"):
        setattr(w, name, _bf16_scaled(getattr(w, name), 2.0 ** log2f))
    it = _run(w, torch_cuda)
    pool, _ = oracle.run_iteration(w)
    same_pool(it.pool_host(), pool)
    ks = pool.k_scale[pool.k_scale > 0]
    lo, hi = float(ks.min()), float(ks.max())
    say(f"[case] fp8 append, K/V x 2^{log2f}: tile scales {lo:.3e} .. {hi:.3e}")
    fast = (ks >= 2.0 ** -100) & (ks <= 2.0 ** 100)
    assert fast.all() if log2f in (-90, 100) else not fast.any()


def _rows_case(name, n_decode, prefill_q, kv, seed):
    g = np.random.Generator(np.random.PCG64(seed))
    rows = [W.RowSpec(W.DECODE, int(g.integers(0, 80)), 1, int(g.integers(-1, 2)))
            for _ in range(n_decode)]
    if prefill_q:
        rows.insert(n_decode // 2, W.RowSpec(W.PREFILL, 40, prefill_q))
    return W.build(name, rows, {0: 32, 1: 48}, 4, 2, 64, kv_dtype=kv, seed=seed)


@pytest.mark.parametrize("kv", [W.KV_BF16, W.KV_FP8])
def test_append_direct_form(torch_cuda, kv):
    # decode rows only: every row writes one block, the padded per-row grid is used
    _check_small(_rows_case(f"direct-{kv}", 300, 0, kv, 115), torch_cuda, f"append-direct-{kv}")


@pytest.mark.parametrize("kv", [W.KV_BF16, W.KV_FP8])
def test_append_scan_form(torch_cuda, kv):
    # one long prefill row among 2,600 rows: the padded grid would be large, so
    # units are enumerated by the LDS scan, over two row windows
    _check_small(_rows_case(f"scan-{kv}", 2600, 600, kv, 116), torch_cuda, f"append-scan-{kv}")


@pytest.mark.parametrize("hq,hkv,d,kv", [(32, 1, 64, W.KV_BF16), (8, 2, 128, W.KV_FP8),
                                         (4, 4, 128, W.KV_BF16)])
def test_prefill_split_key_ranges(torch_cuda, hq, hkv, d, kv):
    # few prefill tiles with long cached contexts: their key ranges are cut
    # into pieces whose partial results the merge kernel combines
    rows = [W.RowSpec(W.PREFILL, 3000, 40), W.RowSpec(W.DECODE, 700, 1),
            W.RowSpec(W.PREFILL, 1500, 300), W.RowSpec(W.PREFILL, 64, 17)]
    w = W.build(f"split-{hq}-{hkv}-{d}-{kv}", rows, {}, hq, hkv, d, kv_dtype=kv, seed=118)
    _check_small(w, torch_cuda, f"prefill-split-{hq}/{hkv}/{d}/{kv}")


@pytest.mark.parametrize("kv", [W.KV_BF16, W.KV_FP8])
def test_prefill_one_round_chained(torch_cuda, kv):
    # one round of prefill workgroups (24 tiles x 8 KV heads, tiles of 1 to 40
    # 64-key tiles; the same shape as the plan-invariant case): short tiles'
    # workgroups also run the leading keys of long tiles, chained
    rows = [W.RowSpec(W.PREFILL, 0, 1024), W.RowSpec(W.DECODE, 900, 1),
            W.RowSpec(W.PREFILL, 2000, 512), W.RowSpec(W.DECODE, 40, 1)]
    w = W.build(f"one-round-{kv}", rows, {}, 32, 8, 128, kv_dtype=kv, seed=131)
    _check_small(w, torch_cuda, f"prefill-one-round-{kv}")


def test_deterministic(torch_cuda):
    w = W.random_case(110, num_rows=8, num_q_heads=8, num_kv_heads=2, head_dim=128,
                      max_ctx=2000, max_q=64)
    say("[case] determinism")
    a = _run(w, torch_cuda).out.cpu().numpy()
    b = _run(w, torch_cuda).out.cpu().numpy()
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_alias_vs_duplicate(torch_cuda):
    a = W.random_case(111, num_rows=8, num_q_heads=8, num_kv_heads=2, head_dim=128,
                      max_ctx=1500, max_q=40, n_groups=2)
    b = W.random_case(111, num_rows=8, num_q_heads=8, num_kv_heads=2, head_dim=128,
                      max_ctx=1500, max_q=40, n_groups=2, duplicate_prefix=True)
    say("[case] alias vs duplicate")
    ga = _run(a, torch_cuda).out.cpu().numpy()
    gb = _run(b, torch_cuda).out.cpu().numpy()
    assert np.abs(ga - gb).max() <= ATOL


def test_empty_batch(torch_cuda):
    from paper_2504_03651_amd import echo
    say("[case] empty batch")
    pool = echo.KVPool(16, 2, 64).poison()
    empty = W.Batch(np.zeros((0, 1), np.int32), np.zeros(0, np.int32), np.zeros(1, np.int32),
                    np.zeros(0, np.uint8))
    b = echo.DeviceBatch(empty)
    z = torch_cuda.zeros(1, dtype=torch_cuda.int16, device="cuda")
    echo.kv_append(pool, b, z, z)
    out = torch_cuda.zeros(1, dtype=torch_cuda.float32, device="cuda")
    ws = torch_cuda.empty(256, dtype=torch_cuda.uint8, device="cuda")
    echo.attn_mixed(pool, b, z, 4, 0.125, out, ws)
    b.mirrors = False
    echo.attn_mixed(pool, b, z, 4, 0.125, out, ws)
    torch_cuda.cuda.synchronize()


def test_append_without_mirrors(torch_cuda):
    w = W.random_case(112, num_rows=6, head_dim=64, max_ctx=300, max_q=40)
    from paper_2504_03651_amd.session import Iteration
    say("[case] append without host mirrors")
    it = Iteration(w, mirrors=False)
    it.copy()
    it.append()
    torch_cuda.cuda.synchronize()
    pool = oracle.prepare(w)
    oracle.block_copy(pool, w.cow_pairs)
    oracle.kv_append(pool, w.batch, w.k_new, w.v_new)
    same_pool(it.pool_host(), pool)


def test_block_copy_many_pairs(torch_cuda):
    from paper_2504_03651_amd.session import Iteration
    for kv in (W.KV_BF16, W.KV_FP8):
        w = W.random_case(113, num_rows=5, head_dim=128, num_kv_heads=4, num_q_heads=8,
                          kv_dtype=kv, max_ctx=500)
        say(f"[case] block copy {kv}")
        it = Iteration(w)
        g = np.random.Generator(np.random.PCG64(5))
        src = g.choice(w.used_blocks, size=min(40, len(w.used_blocks)), replace=False)
        dst = g.choice(w.free_blocks, size=len(src), replace=False)
        pairs = np.stack([src, dst], 1).astype(np.int32)
        from paper_2504_03651_amd import echo
        echo.block_copy(it.pool, torch_cuda.from_numpy(pairs).cuda(), pairs)
        torch_cuda.cuda.synchronize()
        pool = oracle.prepare(w)
        oracle.block_copy(pool, pairs)
        same_pool(it.pool_host(), pool)


# block ids a prefill workgroup can stage in LDS at head_dim 128:
# (160 KiB - 3 stages x 32 KiB - 3 x 16 B of scales) / 4 B; pinned on the host
# by test_abi_host.test_prefill_row_beyond_the_staging_limit
PF_MAX_BLOCKS_D128 = 16372


def test_prefill_at_the_staging_limit(torch_cuda):
    # one prefill row whose key range fills the block-id staging exactly:
    # 8,448 new tokens after 253,504 cached ones, GQA 8/4 (66 tiles x 4 KV
    # heads = 264 workgroups, more than one round, so the key range is
    # neither cut into pieces nor shared out to chained workgroups)
    q = 8448
    w = W.build("pf-limit", [W.RowSpec(W.PREFILL, PF_MAX_BLOCKS_D128 * 16 - q, q)], {}, 8, 4, 128,
                seed=31)
    say(f"[case] prefill at the staging limit: T={w.batch.num_tokens} "
        f"L={int(w.batch.seq_lens[0])} NB={w.num_blocks}")
    it = _run(w, torch_cuda)
    c, ids = compact(w)
    pool = oracle.prepare(c)
    oracle.kv_append(pool, c.batch, c.k_new, c.v_new)
    same_pool(it.pool_host(ids), pool)
    sel = sample_queries(w, 48, seed=31)
    ref = oracle.attention(pool, c.batch, c.q, c.num_q_heads, c.sm_scale, sel=sel)
    got = it.out.cpu().numpy().reshape(-1, w.head_dim)[sel]
    err, nerr = attn_error(got, ref)
    say(f"       {len(sel)} sampled outputs: max abs err {err:.3e}  normalised {nerr:.3e}")
    assert err <= ATOL


@pytest.mark.parametrize("cfg", [2, 3, 4, 5])
def test_full_size_config(torch_cuda, cfg):
    # the launch configuration bench.py times: host mirrors, host plan
    w = W.config(cfg)
    th = cpu_share()
    say(f"[case] config{cfg} full size: rows={w.batch.num_rows} T={w.batch.num_tokens} "
        f"NB={w.num_blocks} kv={w.kv_dtype} (oracle on {th} threads)")
    it = _run(w, torch_cuda)
    out = it.out.cpu().numpy().reshape(-1, w.head_dim)
    assert not np.isnan(out).any()
    c, ids = compact(w)
    pool = oracle_pool(c, th)
    oracle.block_copy(pool, c.cow_pairs)
    oracle.kv_append(pool, c.batch, c.k_new, c.v_new)
    say("       comparing touched blocks bit for bit")
    same_pool(it.pool_host(ids), pool)
    # every output where the oracle takes seconds; else every decode output
    # and whole prefill tiles
    sel = None if cfg in (2, 3) else tile_queries(w)
    what = "all" if sel is None else f"{len(sel)} of {out.shape[0]}"
    say(f"       oracle attention over {what} query vectors")
    ref = oracle.attention(pool, c.batch, c.q, c.num_q_heads, c.sm_scale, sel=sel, threads=th)
    got = out if sel is None else out[sel]
    err, nerr = attn_error(got, ref)
    say(f"       {what} outputs: max abs err {err:.3e}  normalised {nerr:.3e}")
    assert err <= ATOL


# --------------------------------------------------------- non-power-of-two groups

GQA = [(g, hkv, d, kv) for g, hkv, d in ((3, 2, 128), (6, 2, 64), (12, 1, 128), (24, 2, 128))
       for kv in (W.KV_BF16, W.KV_FP8)]


@pytest.mark.parametrize("case", GQA, ids=[f"g{c[0]}-d{c[2]}-{c[3]}" for c in GQA])
def test_gqa_groups_not_powers_of_two(torch_cuda, case):
    # query heads per KV head of 3, 6, 12 and 24: partial lanes of a decode
    # wave's 16 query vectors, two head chunks (24), prefill tiles of 85, 42,
    # 21 and 10 tokens
    g, hkv, d, kv = case
    w = W.random_case(210 + g, num_rows=9, num_q_heads=g * hkv, num_kv_heads=hkv, head_dim=d,
                      kv_dtype=kv, max_ctx=2000, max_q=150, n_groups=2)
    _check_small(w, torch_cuda, f"gqa{g}-{kv}")


# ------------------------------------------------------ plan built on the device

NOMIRROR = [
    ("cfg1", lambda: W.config1()),
    ("random-301", lambda: W.random_case(301, num_rows=8, num_q_heads=8, num_kv_heads=2,
                                         head_dim=128, max_ctx=3000, max_q=200, n_groups=2)),
    ("random-302-e4m3", lambda: W.random_case(302, num_rows=7, num_q_heads=32, num_kv_heads=8,
                                              head_dim=128, kv_dtype=W.KV_FP8, max_ctx=2500,
                                              max_q=120, n_groups=2)),
    ("random-303-gqa6", lambda: W.random_case(303, num_rows=9, num_q_heads=12, num_kv_heads=2,
                                              head_dim=64, max_ctx=1500, max_q=90, n_groups=3)),
    ("random-304-gqa24", lambda: W.random_case(304, num_rows=6, num_q_heads=48, num_kv_heads=2,
                                               head_dim=128, max_ctx=1200, max_q=60)),
    ("many-rows", lambda: W.random_case(305, num_rows=1500, num_q_heads=4, num_kv_heads=2,
                                        head_dim=64, max_ctx=90, max_q=20, n_groups=3)),
]


@pytest.mark.parametrize("make", [m for _, m in NOMIRROR], ids=[n for n, _ in NOMIRROR])
def test_attention_without_mirrors(torch_cuda, make):
    # the same iteration, planned on the device (no prefix grouping): outputs
    # within ATOL of the oracle and of the host-planned path
    w = make()
    say(f"[case] no mirrors {w.name}: rows={w.batch.num_rows} T={w.batch.num_tokens} "
        f"Hq={w.num_q_heads} Hkv={w.num_kv_heads} D={w.head_dim} kv={w.kv_dtype}")
    it = _run(w, torch_cuda, mirrors=False)
    pool, ref = oracle.run_iteration(w)
    same_pool(it.pool_host(), pool)
    got = it.out.cpu().numpy().reshape(ref.shape)
    err, nerr = attn_error(got, ref)
    say(f"       max abs err {err:.3e}  normalised {nerr:.3e}")
    assert err <= ATOL
    hdr = it.workspace[:64 * 4].view(torch_cuda.int32).cpu().numpy()
    assert hdr[4] == 0, "no row may be skipped"
    host = _run(w, torch_cuda).out.cpu().numpy().reshape(ref.shape)
    assert np.abs(host - got).max() <= ATOL


def test_attention_without_mirrors_full_size_config3(torch_cuda):
    w = W.config(3)
    th = cpu_share()
    say(f"[case] no mirrors config3 full size (oracle on {th} threads)")
    it = _run(w, torch_cuda, mirrors=False)
    out = it.out.cpu().numpy().reshape(-1, w.head_dim)
    c, ids = compact(w)
    pool = oracle_pool(c, th)
    oracle.block_copy(pool, c.cow_pairs)
    oracle.kv_append(pool, c.batch, c.k_new, c.v_new)
    same_pool(it.pool_host(ids), pool)
    ref = oracle.attention(pool, c.batch, c.q, c.num_q_heads, c.sm_scale, threads=th)
    err, nerr = attn_error(out, ref)
    say(f"       all outputs: max abs err {err:.3e}  normalised {nerr:.3e}")
    assert err <= ATOL


def test_attention_without_mirrors_skips_inconsistent_rows(torch_cuda):
    # a decode row whose block table names a block outside the pool, and a
    # prefill row with more keys than its block table holds: both are skipped
    # by the device planner (their outputs stay as they were), the others match
    w = W.random_case(306, num_rows=8, num_q_heads=8, num_kv_heads=2, head_dim=128,
                      max_ctx=800, max_q=50, n_groups=2)
    say("[case] no mirrors, inconsistent rows")
    from paper_2504_03651_amd.session import Iteration
    it = Iteration(w, mirrors=False)
    it.copy()
    it.append()
    kind = w.batch.row_kind
    rd = int(np.flatnonzero(kind == W.DECODE)[0])
    rp = int(np.flatnonzero(kind == W.PREFILL)[0])
    it.batch.bt[rd, 0] = w.num_blocks + 7
    it.batch.sl[rp] = it.batch.max_seq_len + 1
    it.out.fill_(7.0)
    it.attend()
    torch_cuda.cuda.synchronize()
    hdr = it.workspace[:64 * 4].view(torch_cuda.int32).cpu().numpy()
    assert hdr[4] == 2
    pool, ref = oracle.run_iteration(w)
    got = it.out.cpu().numpy().reshape(w.batch.num_tokens, w.num_q_heads, w.head_dim)
    ref = ref.reshape(got.shape)
    qs = w.batch.q_start
    skipped = np.zeros(w.batch.num_tokens, bool)
    for r in (rd, rp):
        skipped[qs[r]:qs[r + 1]] = True
    assert (got[skipped] == 7.0).all()
    assert np.abs(got[~skipped] - ref[~skipped]).max() <= ATOL


def test_host_workspace_must_be_pinned(torch_cuda):
    import ctypes
    from paper_2504_03651_amd import echo
    from paper_2504_03651_amd.session import Iteration
    w = W.config1()
    say("[case] host workspace: pageable memory refused, pinned accepted")
    it = Iteration(w)
    it.copy()
    it.append()
    cp, cb = it.pool.c(), it.batch.c()
    n = echo.host_workspace_bytes(it.pool, it.batch, w.num_q_heads)
    pageable = np.zeros(n + 16, np.uint8)
    L = echo.lib()
    s = ctypes.c_void_p(torch_cuda.cuda.current_stream().cuda_stream)
    ws = it.workspace
    rc = L.echo_attn_mixed(ctypes.byref(cp), ctypes.byref(cb), it.q.data_ptr(), w.num_q_heads,
                           w.sm_scale, it.out.data_ptr(), ws.data_ptr(), ws.numel(),
                           ctypes.c_void_p(pageable.ctypes.data), n, s)
    assert rc == echo.ECHO_E_WORKSPACE and "pinned" in echo.last_error()
    hw = echo.HostWorkspace(slots=1)
    try:
        ptr, size, slot = hw.acquire(n)
        rc = L.echo_attn_mixed(ctypes.byref(cp), ctypes.byref(cb), it.q.data_ptr(),
                               w.num_q_heads, w.sm_scale, it.out.data_ptr(), ws.data_ptr(),
                               ws.numel(), ctypes.c_void_p(ptr), size, s)
        assert rc == echo.ECHO_OK, echo.last_error()
        hw.release(slot, torch_cuda.cuda.current_stream())
        torch_cuda.cuda.synchronize()
    finally:
        hw.close()
    pool, ref = oracle.run_iteration(w)
    err, _ = attn_error(it.out.cpu().numpy().reshape(ref.shape), ref)
    assert err <= ATOL


def _random_batch(k):
    """Random batch k: GQA group, KV heads, head_dim, cache dtype, row count,
    context and chunk lengths and prefix groups all drawn (seeded)."""
    g = np.random.Generator(np.random.PCG64([4242, k]))
    G = int(g.choice([1, 2, 3, 4, 5, 6, 8, 12, 16, 24, 32]))
    hkv = int(g.choice([1, 2, 4])) if G <= 16 else int(g.choice([1, 2]))
    D = int(g.choice([64, 128]))
    kv = W.KV_FP8 if g.random() < 0.5 else W.KV_BF16
    return W.random_case(4242 + k, num_rows=int(g.integers(1, 40)), num_q_heads=G * hkv,
                         num_kv_heads=hkv, head_dim=D, kv_dtype=kv,
                         max_ctx=int(g.choice([50, 300, 1500, 4000])),
                         max_q=int(g.choice([1, 20, 100, 400])), n_groups=int(g.integers(0, 4)))


@pytest.mark.parametrize("k", range(40))
def test_random_batches(torch_cuda, k):
    # forty random batches, host-planned (even k) and device-planned (odd k):
    # pools bit-exact and every output within the tolerance
    w = _random_batch(k)
    mirrors = k % 2 == 0
    say(f"[case] random batch {k}: rows={w.batch.num_rows} T={w.batch.num_tokens} "
        f"Hq={w.num_q_heads} Hkv={w.num_kv_heads} D={w.head_dim} kv={w.kv_dtype} mirrors={mirrors}")
    it = _run(w, torch_cuda, mirrors=mirrors)
    pool, ref = oracle.run_iteration(w)
    same_pool(it.pool_host(), pool)
    err, _ = attn_error(it.out.cpu().numpy().reshape(ref.shape), ref)
    assert err <= ATOL
