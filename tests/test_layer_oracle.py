"""Pins of the decoder-layer oracle (CPU): properties of RoPE, RMSNorm and SiLU
that the definitions fix, the GEMM orientation (out_features x in_features
weights), and the residual structure of the layer."""
import numpy as np
import pytest

import oracle
from oracle import layer_oracle as LO
from paper_2504_03651_amd import workload as W


def test_rope_is_a_position_dependent_rotation():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 3, 64))
    pos = np.array([0, 1, 17, 1000, 32767])
    r = LO.rope(x, pos, 500000.0)
    assert np.allclose(np.linalg.norm(r, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-12)
    assert np.array_equal(r[0], x[0])                       # position 0: identity
    # relative positions: <R(q,p), R(k,p')> depends on p - p' only
    q, k = rng.standard_normal((1, 1, 64)), rng.standard_normal((1, 1, 64))
    d = lambda p, pp: float(np.sum(LO.rope(q, [p], 1e4) * LO.rope(k, [pp], 1e4)))
    assert d(10, 3) == pytest.approx(d(110, 103), rel=1e-10)
    assert d(0, 0) == pytest.approx(float(np.sum(q * k)), rel=1e-12)
    # the first pair turns by exactly one radian per position (theta^0 = 1)
    e = np.zeros((1, 1, 8))
    e[0, 0, 0] = 1.0
    out = LO.rope(e, [1], 10000.0)[0, 0]
    assert out[0] == pytest.approx(np.cos(1.0)) and out[4] == pytest.approx(np.sin(1.0))


def test_rmsnorm_and_silu():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((4, 256)) * 3.0
    y = LO.rmsnorm(x, np.ones(256), 0.0)
    assert np.allclose(np.mean(y * y, axis=-1), 1.0, rtol=1e-12)
    assert LO.silu(np.array([0.0]))[0] == 0.0
    assert LO.silu(np.array([1.0]))[0] == pytest.approx(1.0 / (1.0 + np.exp(-1.0)))
    assert LO.silu(np.array([40.0]))[0] == pytest.approx(40.0)
    assert abs(LO.silu(np.array([-40.0]))[0]) < 1e-15


def test_bf16_rounding_is_nearest_even():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to the even pattern (1.0)
    assert LO.bf16_bits([1.0 + 2.0 ** -8])[0] == 0x3F80
    assert LO.bf16_bits([1.0 + 3 * 2.0 ** -8])[0] == 0x3F82
    assert LO.bf16_bits([-2.0])[0] == 0xC000


def _small():
    lw = W.layer_weights(3, 256, 4, 2, 64, 512)
    w = W.random_case(11, num_rows=5, num_q_heads=4, num_kv_heads=2, head_dim=64, max_ctx=300,
                      max_q=40)
    return lw, w


def test_zero_projections_leave_the_residual():
    lw, w = _small()
    lw.w_o = np.zeros_like(lw.w_o)
    lw.w_down = np.zeros_like(lw.w_down)
    x = W.layer_hidden(5, w.batch.num_tokens, lw.hidden)
    out, _ = LO.forward(lw, oracle.prepare(w), w.batch, x)
    assert np.array_equal(out, x)


def test_gemm_orientation_and_kv_written():
    lw, w = _small()
    T = w.batch.num_tokens
    x = W.layer_hidden(5, T, lw.hidden)
    pool = oracle.prepare(w)
    out, t = LO.forward(lw, pool, w.batch, x)
    # qkv row t = W_qkv @ y[t]: check one entry by hand
    f = LO.bf16_value
    j = 7
    assert t["qkv"][2, j] == LO.bf(np.dot(f(lw.w_qkv)[j], t["y"][2]))
    # the rotated keys landed in the pool at each token's slot
    pos = LO.positions(w.batch)
    r = int(np.searchsorted(w.batch.q_start, 0, side="right") - 1)
    blk = int(w.batch.block_tables[r][pos[0] // 16])
    assert np.array_equal(pool.k[blk, :, pos[0] % 16, :], LO.bf16_bits(t["k"][0]))
    assert out.shape == (T, lw.hidden) and np.isfinite(LO.bf16_value(out)).all()
