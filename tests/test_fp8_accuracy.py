"""Accuracy of the e4m3 cache reading itself (CPU, oracle only): attention
over an e4m3 pool against the same attention over the unquantised bf16
values.  Not a parity test (both sides are the oracle): it bounds what the
quantisation costs, for blocks written whole and for blocks filled one token
per call, whose scale is fixed by their first token's largest value (later
tokens saturate at 448 times it)."""
import numpy as np

import oracle
from paper_2504_03651_amd import workload as W

R, HKV, HQ, D = 48, 2, 8, 128


def _bf16(x):
    u = x.astype(np.float32).view(np.uint32)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def _attend(K, V, Q, fp8, token_by_token):
    """R rows of 16 tokens in one block each; attention of one query per row
    over the 16 keys."""
    bt = (np.arange(R, dtype=np.int32) * 3 + 1).reshape(R, 1)
    pool = oracle.Pool(3 * R + 1, HKV, D, fp8)
    if token_by_token:
        for i in range(16):
            b = W.Batch(bt, np.full(R, i + 1, np.int32), np.arange(R + 1, dtype=np.int32),
                        np.zeros(R, np.uint8))
            oracle.kv_append(pool, b, np.ascontiguousarray(K[:, i]), np.ascontiguousarray(V[:, i]))
    else:
        b = W.Batch(bt, np.full(R, 16, np.int32), (np.arange(R + 1) * 16).astype(np.int32),
                    np.ones(R, np.uint8))
        oracle.kv_append(pool, b, K.reshape(R * 16, HKV, D), V.reshape(R * 16, HKV, D))
    b = W.Batch(bt, np.full(R, 16, np.int32), np.arange(R + 1, dtype=np.int32), np.zeros(R, np.uint8))
    return oracle.attention(pool, b, Q, HQ, float(np.float32(1 / np.sqrt(D))), threads=4)


def test_e4m3_error_against_the_unquantised_cache():
    rng = np.random.default_rng(0)
    K = _bf16(rng.standard_normal((R, 16, HKV, D)))
    V = _bf16(rng.standard_normal((R, 16, HKV, D)))
    Q = _bf16(rng.standard_normal((R, HQ, D)))
    ref = _attend(K, V, Q, False, True)
    rms_ref = float(np.sqrt(np.mean(ref ** 2)))
    whole = np.abs(_attend(K, V, Q, True, False) - ref)
    tbt = np.abs(_attend(K, V, Q, True, True) - ref)
    rms = lambda d: float(np.sqrt(np.mean(d ** 2))) / rms_ref
    # blocks written whole: 3 mantissa bits, about 3.5% RMS relative error
    assert rms(whole) < 0.05 and whole.max() < 0.2
    # blocks filled token by token: saturation of later tokens costs more
    assert rms(tbt) > 1.3 * rms(whole) and rms(tbt) < 0.1 and tbt.max() < 1.0
