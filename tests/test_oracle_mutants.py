"""Planted mistakes in the oracle must break at least one pin.

Each case copies the oracle's C source, plants one plausible mistake (a wrong
causal alignment, head mapping, layout, scale, rounding or fresh-block rule),
builds it on the CPU and checks that the pin named for it fails.  This shows
that the pins in test_oracle_pins.py constrain the oracle, not just agree
with it.
"""
import os
import shutil

import numpy as np
import pytest

import oracle
from paper_2504_03651_amd import workload as W
from tests import bruteforce as BF

SRC = os.path.join(os.path.dirname(oracle.__file__), "echo_oracle.c")


def _bruteforce_err(kv=W.KV_BF16, G=4):
    w = W.random_case(3, num_rows=6, num_q_heads=8, num_kv_heads=8 // G, head_dim=64, kv_dtype=kv, max_ctx=200, max_q=30)
    _, out = oracle.run_iteration(w)
    ref = BF.dense_attention(w).reshape(out.shape)
    err = np.abs(out - ref)
    return np.inf if np.isnan(err).any() else err.max()


def _append_slots_ok():
    w = W.random_case(41, num_rows=4, head_dim=64, max_ctx=100, max_q=20)
    pool = oracle.prepare(w)
    oracle.kv_append(pool, w.batch, w.k_new, w.v_new)
    bt, sl, qs = w.batch.block_tables, w.batch.seq_lens, w.batch.q_start
    for r in range(w.batch.num_rows):
        L = int(sl[r]); q = int(qs[r + 1] - qs[r])
        for i in range(q):
            p = L - q + i
            blk, slot = int(bt[r, p // 16]), p % 16
            if not np.array_equal(pool.v[blk, :, :, slot], w.v_new[qs[r] + i]):
                return False
    return True


def _codec_ok():
    ys = np.array([1.0625, 1.1875, 0.0009765625, 0.0029296875, 3.3, -7.77, 500.0],
                  np.float32)
    ref = BF.e4m3_encode_bruteforce(ys)
    return all(oracle.e4m3_encode(float(y)) == int(c) for y, c in zip(ys, ref))


def _bf16_ok():
    bits = np.arange(0, 65536, 101, dtype=np.uint32).astype(np.uint16)
    ref = BF.bf16_to_f64(bits)
    got = np.array([oracle.bf16_value(b) for b in bits])
    return bool(((got == ref) | (np.isnan(got) & np.isnan(ref))).all())


MUTANTS = [
    ("top-left causal alignment",
     "const int32_t pos = b->seq_lens[r] - qlen + (t - b->q_start[r]);",
     "const int32_t pos = (t - b->q_start[r]);",
     lambda: _bruteforce_err() < 1e-12),
    ("query head mapped modulo the KV heads",
     "const int32_t g = h / (J->hq / p->num_kv_heads);",
     "const int32_t g = h % p->num_kv_heads;",
     lambda: _bruteforce_err() < 1e-12),
    ("V stored in the K layout",
     "return (((size_t)blk * p->num_kv_heads + h) * p->head_dim + d) * BS + slot;",
     "return (((size_t)blk * p->num_kv_heads + h) * BS + slot) * p->head_dim + d;",
     _append_slots_ok),
    ("softmax scale applied twice",
     "s[j] = J->scale * dot;",
     "s[j] = J->scale * J->scale * dot;",
     lambda: _bruteforce_err() < 1e-12),
    ("last key dropped",
     "double dot = 0.0;\n        for (int32_t d = 0; d < D; ++d)",
     "double dot = (j == pos) ? -1e300 : 0.0;\n        for (int32_t d = 0; d < D; ++d)",
     lambda: _bruteforce_err() < 1e-12),
    ("fp8 V scale dropped",
     "return orc_e4m3_value(((const uint8_t *)p->v)[v_index(p, blk, h, slot, d)]) *\n"
     "           (double)p->v_scale[(size_t)blk * p->num_kv_heads + h];",
     "return orc_e4m3_value(((const uint8_t *)p->v)[v_index(p, blk, h, slot, d)]);",
     lambda: _bruteforce_err(W.KV_FP8) < 1e-12),
    ("every written block treated as fresh",
     "const int fresh = (BS * j >= p0);",
     "const int fresh = 1;",
     lambda: _bruteforce_err(W.KV_FP8) < 1e-12),
    ("ties rounded away from zero",
     "return fmod(fl, 2.0) == 0.0 ? fl : fl + 1.0;",
     "return fl + 1.0;",
     _codec_ok),
    ("bf16 decoded with a wrong shift",
     "uint32_t w = (uint32_t)bits << 16;",
     "uint32_t w = (uint32_t)bits << 15;",
     _bf16_ok),
]


@pytest.fixture
def restore_oracle():
    saved = oracle._lib
    yield
    oracle._lib = saved


@pytest.mark.parametrize("name,old,new,pin", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, restore_oracle, name, old, new, pin):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for '{name}' not unique"
    # the unmutated oracle passes the pin
    assert pin(), f"pin for '{name}' fails on the real oracle"
    mut = tmp_path / "mutant.c"
    mut.write_text(src.replace(old, new))
    shutil.copy(os.path.join(os.path.dirname(SRC), "echo_oracle.h"), tmp_path / "echo_oracle.h")
    so = oracle.build(str(mut), str(tmp_path / "libmutant.so"))
    oracle._lib = oracle.load(so)
    assert not pin(), f"planted mistake '{name}' passed its pin"
