"""Pins of the fp64 oracle against facts that do not come from the oracle.

* dense brute force (tests/bruteforce.py): rows rebuilt densely from the
  inputs, one masked matrix softmax per row;
* closed forms: a one-token sequence returns its value, a zero query returns
  the mean value, constant keys return the mean, one dominant logit returns
  that value, all-ones values give exactly one (softmax rows sum to one);
* invariants: aliased prefix blocks equal physically duplicated ones, any
  placement of blocks in the pool gives identical bits, a prefill chunk equals
  the same tokens decoded one by one, row kind does not matter, GQA equals
  MHA with repeated KV heads;
* codecs: bf16 decode, and the e4m3 encoder over every bf16 input at three
  scales against a nearest-value search over all finite codes;
* golden fixtures with their sources under tests/golden/.
"""
import copy
import json
import os

import numpy as np
import pytest

import oracle
from paper_2504_03651_amd import workload as W
from tests import bruteforce as BF

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _oracle_out(w, **kw):
    _, out = oracle.run_iteration(w, **kw)
    return out.reshape(w.batch.num_tokens, w.num_q_heads, w.head_dim)


# ---------------------------------------------------------------- brute force


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_bruteforce_random_bf16(seed):
    w = W.random_case(seed, num_rows=6, num_q_heads=8, num_kv_heads=2, head_dim=64,
                      max_ctx=300, max_q=40)
    ref = BF.dense_attention(w)
    got = _oracle_out(w)
    assert np.abs(got - ref).max() < 1e-12


def test_bruteforce_config1_both_aliasings():
    for share in (False, True):
        w = W.config1(share_with_prefill=share)
        np.testing.assert_allclose(_oracle_out(w), BF.dense_attention(w), atol=1e-12, rtol=0)


@pytest.mark.parametrize("seed", [5, 6])
def test_bruteforce_random_fp8(seed):
    w = W.random_case(seed, num_rows=5, num_q_heads=4, num_kv_heads=2, head_dim=64,
                      kv_dtype=W.KV_FP8, max_ctx=200, max_q=40)
    ref = BF.dense_attention(w)
    got = _oracle_out(w)
    assert np.abs(got - ref).max() < 1e-12


def test_bruteforce_mha_d128():
    w = W.random_case(11, num_rows=4, num_q_heads=4, num_kv_heads=4, head_dim=128,
                      max_ctx=150, max_q=30)
    assert np.abs(_oracle_out(w) - BF.dense_attention(w)).max() < 1e-12


# --------------------------------------------------------------- closed forms


def _with(w, **arrays):
    w2 = copy.copy(w)
    for k, v in arrays.items():
        setattr(w2, k, v)
    return w2


def test_single_token_returns_its_value():
    rows = [W.RowSpec(W.DECODE, 0, 1), W.RowSpec(W.PREFILL, 0, 1)]
    w = W.build("l1", rows, {}, 4, 2, 64, num_blocks=32, seed=3)
    out = _oracle_out(w)
    v = BF.bf16_to_f64(w.v_new)                      # [T][Hkv][D]
    for t in range(2):
        for h in range(4):
            assert np.array_equal(out[t, h], v[t, h // 2])


def test_zero_query_gives_mean_value():
    w = W.random_case(21, num_rows=4, num_q_heads=4, num_kv_heads=4, head_dim=64, max_ctx=120)
    w = _with(w, q=np.zeros_like(w.q))
    out = _oracle_out(w)
    dense = BF.dense_rows(w)
    qs, sl = w.batch.q_start, w.batch.seq_lens
    for r in range(w.batch.num_rows):
        c = int(sl[r] - (qs[r + 1] - qs[r]))
        V = dense[r][1]
        for i in range(int(qs[r + 1] - qs[r])):
            np.testing.assert_allclose(out[qs[r] + i], V[:c + i + 1].mean(axis=0),
                                       atol=1e-12, rtol=0)


def test_constant_keys_give_mean_value():
    w = W.random_case(22, num_rows=3, num_q_heads=2, num_kv_heads=2, head_dim=64, max_ctx=90)
    one = np.full_like(w.k_new, 0x3F80)   # bf16 1.0 everywhere
    w = _with(w, k_new=one, ctx_k=np.full_like(w.ctx_k, 0x3F80))
    out = _oracle_out(w)
    dense = BF.dense_rows(w)
    qs, sl = w.batch.q_start, w.batch.seq_lens
    for r in range(w.batch.num_rows):
        c = int(sl[r] - (qs[r + 1] - qs[r]))
        for i in range(int(qs[r + 1] - qs[r])):
            np.testing.assert_allclose(out[qs[r] + i], dense[r][1][:c + i + 1].mean(axis=0),
                                       atol=1e-12, rtol=0)


def test_softmax_rows_sum_to_one():
    w = W.random_case(23, num_rows=5, num_q_heads=4, num_kv_heads=2, head_dim=64, max_ctx=200)
    w = _with(w, v_new=np.full_like(w.v_new, 0x3F80), ctx_v=np.full_like(w.ctx_v, 0x3F80))
    out = _oracle_out(w)
    assert np.abs(out - 1.0).max() < 1e-12


def test_dominant_logit_selects_its_value():
    # one decode row of 20 tokens; key 7 is 8*e_0 and the query is 8*e_0, so
    # its logit exceeds every other by 64/8 = 8 units... make it 64 via scale
    rows = [W.RowSpec(W.DECODE, 19, 1)]
    w = W.build("dom", rows, {}, 1, 1, 64, num_blocks=16, seed=4)
    ck = np.zeros_like(w.ctx_k)
    ck[7, 0, 0] = 0x4100                   # bf16 8.0
    q = np.zeros_like(w.q)
    q[0, 0, 0] = 0x4100
    w = _with(w, ctx_k=ck, k_new=np.zeros_like(w.k_new), q=q, sm_scale=1.0)
    out = _oracle_out(w)
    v7 = BF.bf16_to_f64(w.ctx_v[7, 0])
    # weight of key 7 is 1 / (1 + 19 e^-64)
    np.testing.assert_allclose(out[0, 0], v7, atol=1e-25 * 20 * 8, rtol=1e-26)


def test_golden_two_key_softmax():
    g = json.load(open(os.path.join(GOLDEN, "two_key_softmax.json")))
    rows = [W.RowSpec(W.DECODE, 1, 1)]
    w = W.build("two", rows, {}, 1, 1, g["head_dim"], num_blocks=4, seed=0)
    bf = lambda x: np.uint16(np.float32(x).view(np.uint32) >> 16)
    ck = np.zeros_like(w.ctx_k); cv = np.zeros_like(w.ctx_v)
    kn = np.zeros_like(w.k_new); vn = np.zeros_like(w.v_new)
    q = np.zeros_like(w.q)
    q[0, 0, 0] = bf(g["q0"]); ck[0, 0, 0] = bf(g["k0_0"]); kn[0, 0, 0] = bf(g["k1_0"])
    cv[0, 0, 0] = bf(g["v0_0"]); vn[0, 0, 1] = bf(g["v1_1"])
    w = _with(w, ctx_k=ck, ctx_v=cv, k_new=kn, v_new=vn, q=q, sm_scale=g["sm_scale"])
    out = _oracle_out(w)
    assert abs(out[0, 0, 0] - g["expected_out_0"]) < 1e-15
    assert abs(out[0, 0, 1] - g["expected_out_1"]) < 1e-15


# ----------------------------------------------------------------- invariants


@pytest.mark.parametrize("cfg", ["config1", "random"])
def test_alias_equals_duplicate(cfg):
    if cfg == "config1":
        a, b = W.config1(), W.config1(duplicate_prefix=True)
    else:
        a = W.random_case(31, num_rows=6, head_dim=64, max_ctx=400)
        b = W.random_case(31, num_rows=6, head_dim=64, max_ctx=400, duplicate_prefix=True)
    assert not np.array_equal(a.batch.block_tables, b.batch.block_tables)
    assert np.array_equal(_oracle_out(a), _oracle_out(b))


def test_alias_equals_duplicate_fp8():
    a = W.random_case(32, num_rows=5, head_dim=64, kv_dtype=W.KV_FP8, max_ctx=300)
    b = W.random_case(32, num_rows=5, head_dim=64, kv_dtype=W.KV_FP8, max_ctx=300,
                      duplicate_prefix=True)
    assert np.array_equal(_oracle_out(a), _oracle_out(b))


@pytest.mark.parametrize("kv", [W.KV_BF16, W.KV_FP8])
def test_pool_permutation_invariance(kv):
    a = W.random_case(33, num_rows=6, head_dim=64, kv_dtype=kv, max_ctx=300)
    b = W.random_case(33, num_rows=6, head_dim=64, kv_dtype=kv, max_ctx=300, perm_seed=9)
    assert not np.array_equal(a.batch.block_tables, b.batch.block_tables)
    assert np.array_equal(_oracle_out(a), _oracle_out(b))


def test_chunked_prefill_equals_stepwise_decode():
    ctx, n = 37, 21
    w = W.build("chunk", [W.RowSpec(W.PREFILL, ctx, n)], {}, 4, 2, 64, num_blocks=64, seed=5)
    out_chunk = _oracle_out(w)
    pool = oracle.prepare(w)
    bt = w.batch.block_tables
    for i in range(n):
        step = W.Batch(bt, np.array([ctx + i + 1], np.int32), np.array([0, 1], np.int32),
                       np.array([W.DECODE], np.uint8))
        oracle.kv_append(pool, step, w.k_new[i:i + 1], w.v_new[i:i + 1])
        o = oracle.attention(pool, step, w.q[i:i + 1], 4, w.sm_scale)
        assert np.array_equal(o.reshape(4, 64), out_chunk[i])


def test_row_kind_does_not_matter():
    w = W.random_case(34, num_rows=6, head_dim=64, max_ctx=200)
    flip = copy.copy(w.batch)
    flip = W.Batch(w.batch.block_tables, w.batch.seq_lens, w.batch.q_start,
                   np.where(w.batch.q_lens == 1, 1 - w.batch.row_kind, w.batch.row_kind)
                   .astype(np.uint8))
    assert np.array_equal(_oracle_out(w), _oracle_out(_with(w, batch=flip)))


def test_gqa_equals_mha_with_repeated_heads():
    w = W.random_case(35, num_rows=5, num_q_heads=8, num_kv_heads=2, head_dim=64, max_ctx=200)
    G = 4
    rep = lambda a: np.repeat(a, G, axis=1)
    m = _with(w, num_kv_heads=8, k_new=rep(w.k_new), v_new=rep(w.v_new),
              ctx_k=rep(w.ctx_k), ctx_v=rep(w.ctx_v))
    assert np.array_equal(_oracle_out(w), _oracle_out(m))


# ---------------------------------------------------------------------- codecs


def test_bf16_decode_matches_numpy():
    bits = np.arange(0, 65536, 97, dtype=np.uint32).astype(np.uint16)
    ref = BF.bf16_to_f64(bits)
    got = np.array([oracle.bf16_value(b) for b in bits])
    same = (got == ref) | (np.isnan(got) & np.isnan(ref))
    assert same.all()


def test_e4m3_golden_anchors():
    g = json.load(open(os.path.join(GOLDEN, "e4m3_anchors.json")))
    for code, val in g["values"].items():
        v = oracle.e4m3_value(int(code, 16))
        assert v == val and np.signbit(v) == np.signbit(val), code
    for code in g["nan_codes"]:
        assert np.isnan(oracle.e4m3_value(int(code, 16)))
    for x, code, why in g["encode"]:
        assert oracle.e4m3_encode(x) == int(code, 16), why


def test_e4m3_decode_table_matches_bruteforce_table():
    tab = BF.e4m3_table()
    for c in range(256):
        v = oracle.e4m3_value(c)
        assert (np.isnan(v) and np.isnan(tab[c])) or v == tab[c]


def test_e4m3_encoder_exhaustive_over_bf16():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    x = BF.bf16_to_f64(bits)
    finite = np.isfinite(x)
    bits, x = bits[finite], x[finite]
    amax_scale = BF.fresh_scale(np.float32(3.71875))
    for s in (np.float32(1.0), amax_scale, np.float32(2.0 ** -6)):
        with np.errstate(over="ignore"):
            y = (x / np.float64(s)).astype(np.float32)
        ref = BF.e4m3_encode_bruteforce(y)
        enc = np.frompyfunc(lambda v: oracle.e4m3_encode(float(v)), 1, 1)
        got = enc(y).astype(np.uint8)
        bad = np.nonzero(got != ref)[0]
        assert bad.size == 0, (s, y[bad[:5]], got[bad[:5]], ref[bad[:5]])
        # round trip within half a step (times the scale) inside the range
        tab = BF.e4m3_table()
        inr = np.abs(y) <= 448
        dec = tab[got[inr]] * np.float64(s)
        step = np.maximum(2.0 ** (np.floor(np.log2(np.maximum(np.abs(y[inr]), 2.0 ** -6))) - 3),
                          2.0 ** -9)
        assert np.all(np.abs(dec - x[inr]) <= 0.5 * step * np.float64(s) * (1 + 1e-12) +
                      np.abs(x[inr]) * 2.0 ** -24)


def test_fresh_scale_rule():
    assert oracle.e4m3_fresh_scale(0.0) == 1.0
    assert oracle.e4m3_fresh_scale(448.0) == 1.0
    assert oracle.e4m3_fresh_scale(3.5) == np.float32(3.5 / 448.0)


# ------------------------------------------------------------ append and copy


@pytest.mark.parametrize("kv", [W.KV_BF16, W.KV_FP8])
def test_append_writes_exactly_the_new_slots(kv):
    w = W.random_case(41, num_rows=6, head_dim=64, kv_dtype=kv, max_ctx=300, max_q=50)
    pool = oracle.prepare(w)
    before = pool.copy()
    oracle.kv_append(pool, w.batch, w.k_new, w.v_new)
    bt, sl, qs = w.batch.block_tables, w.batch.seq_lens, w.batch.q_start
    written_k = np.zeros(pool.k.shape, bool)
    written_v = np.zeros(pool.v.shape, bool)
    for r in range(w.batch.num_rows):
        L = int(sl[r]); q = int(qs[r + 1] - qs[r])
        for i in range(q):
            p = L - q + i
            blk, slot = int(bt[r, p // 16]), p % 16
            written_k[blk, :, slot, :] = True
            written_v[blk, :, :, slot] = True
            if kv == W.KV_BF16:
                assert np.array_equal(pool.k[blk, :, slot, :], w.k_new[qs[r] + i])
                assert np.array_equal(pool.v[blk, :, :, slot], w.v_new[qs[r] + i])
    assert np.array_equal(pool.k[~written_k], before.k[~written_k])
    assert np.array_equal(pool.v[~written_v], before.v[~written_v])
    if kv == W.KV_FP8:
        dense = BF.dense_rows(w)
        for r in range(w.batch.num_rows):
            L = int(sl[r]); q = int(qs[r + 1] - qs[r])
            for i in range(q):
                p = L - q + i
                blk, slot = int(bt[r, p // 16]), p % 16
                deq = BF.e4m3_table()[pool.k[blk, :, slot, :]] * pool.k_scale[blk][:, None]
                np.testing.assert_array_equal(deq, dense[r][0][p])


def test_block_copy_is_a_byte_copy():
    w = W.random_case(42, num_rows=4, head_dim=64, kv_dtype=W.KV_FP8, max_ctx=200)
    pool = oracle.prepare(w)
    before = pool.copy()
    src = w.used_blocks[:3]
    dst = w.free_blocks[:3]
    oracle.block_copy(pool, np.stack([src, dst], 1))
    for s, d in zip(src, dst):
        assert np.array_equal(pool.k[d], before.k[s]) and np.array_equal(pool.v[d], before.v[s])
        assert np.array_equal(pool.k_scale[d], before.k_scale[s])
    keep = np.ones(pool.num_blocks, bool)
    keep[dst] = False
    assert np.array_equal(pool.k[keep], before.k[keep])
    assert np.array_equal(pool.v[keep], before.v[keep])
