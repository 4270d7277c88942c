"""The decoder layer (echo_layer_forward) against the fp64 layer oracle.

The attention inside the layer meets its own bar (max abs error 1e-2: bf16
probabilities in the P.V product), so its bf16-rounded output differs from
the oracle's by a step in a good part of its entries, and the layer's other
bf16 activations (rounded from fp32 on the GPU, from fp64 in the oracle) add
occasional steps; they propagate through the later GEMMs.  The bar: output
max abs error <= 2^-5 times the largest output magnitude (a few bf16 steps),
mean abs error <= 2^-7 times the mean magnitude, and the appended K/V within a
few steps of their scale (they pass only through the first GEMM and RoPE).
"""
import numpy as np
import pytest

import oracle
from oracle import layer_oracle as LO
from paper_2504_03651_amd import workload as W
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


def _batch(shape):
    H, Hq, Hkv, D, I = shape
    if H < 4096:
        return W.random_case(21, num_rows=7, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D,
                             max_ctx=700, max_q=60)
    # LLaMA-3.1-8B layer shapes (hidden 4,096, GQA 32/8, head_dim 128,
    # intermediate 14,336): two prefill chunks, one on a 300-token context,
    # and three decode rows, two of them sharing a 256-token prefix
    rows = [W.RowSpec(W.PREFILL, 300, 40), W.RowSpec(W.DECODE, 500, 1, 0),
            W.RowSpec(W.PREFILL, 0, 33), W.RowSpec(W.DECODE, 257, 1, 0),
            W.RowSpec(W.DECODE, 129, 1)]
    return W.build("layer-llama8b", rows, {0: 256}, Hq, Hkv, D, seed=24)


@pytest.mark.parametrize("shape", [(256, 4, 2, 64, 512), (512, 8, 2, 128, 1024),
                                   (4096, 32, 8, 128, 14336)])
def test_layer_matches_the_oracle(shape):
    import torch
    from paper_2504_03651_amd import echo, layer
    from paper_2504_03651_amd.session import Iteration
    H, Hq, Hkv, D, I = shape
    lw = W.layer_weights(7, H, Hq, Hkv, D, I)
    w = _batch(shape)
    T = w.batch.num_tokens
    x = W.layer_hidden(8, T, H)
    say(f"[case] layer {shape}: {w.batch.num_rows} rows, {T} tokens")
    it = Iteration(w)                     # device pool with the context appended
    L = layer.Layer(lw)
    hid = torch.from_numpy(x.view(np.int16)).cuda()
    ws = torch.empty(L.workspace_bytes(it.pool, it.batch), dtype=torch.uint8, device="cuda")
    L.forward(it.pool, it.batch, hid, ws)
    torch.cuda.synchronize()
    got = hid.cpu().numpy().view(np.uint16)
    pool = oracle.prepare(w)
    ref, t = LO.forward(lw, pool, w.batch, x)
    gv, rv = LO.bf16_value(got), LO.bf16_value(ref)
    err = float(np.abs(gv - rv).max())
    same = float(np.mean(got == ref))
    say(f"       output max abs err {err:.3e} (scale {np.abs(rv).max():.2f}), identical {same:.3f}")
    assert err <= 2.0 ** -5 * float(np.abs(rv).max())
    assert float(np.abs(gv - rv).mean()) <= 2.0 ** -7 * float(np.abs(rv).mean())
    # the new keys and values in the pool
    k = it.pool.k.cpu().numpy().view(np.uint16)
    v = it.pool.v.cpu().numpy().view(np.uint16)
    def diff(a, b):
        av, bv = LO.bf16_value(a), LO.bf16_value(b)
        assert np.array_equal(np.isnan(av), np.isnan(bv)), "written slots differ"
        m = ~np.isnan(av)
        return float(np.abs(av[m] - bv[m]).max())
    kerr, verr = diff(k, pool.k), diff(v, pool.v)
    say(f"       pool K max abs err {kerr:.3e}, V {verr:.3e}")
    assert kerr <= 2.0 ** -5 * 8 and verr <= 2.0 ** -5 * 8
