"""Plain fp64 reference of one LLaMA-style decoder layer around the iteration.

TEST INFRASTRUCTURE ONLY: the test suite is its only caller.  NumPy in fp64
for every step except the KV append and the attention, which call the fp64 C
oracle of this package; it shares no code with the library.  Activations are
rounded to bf16 (round to nearest even) at the points where the library's
tensors are bf16 (the paper fixes no precision for these layers; the layer's
own tensors decide it): the normed input, qkv, the rotated q and k, the
attention output, h, the second normed input, gate/up, the activation and the
output.

RoPE: each head's pair (i, i + D/2) is rotated by the angle
position * theta^(-2i/D) (rotary position embedding, Su et al. 2021, in the
half-split pairing of LLaMA implementations).
"""
from __future__ import annotations

import numpy as np

import oracle


def bf16_bits(x) -> np.ndarray:
    """fp64 values -> bf16 bit patterns, round to nearest even (via fp32)."""
    f = np.atleast_1d(np.asarray(x, np.float64)).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    out = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    out[np.isnan(f)] = 0x7FC0
    return out.reshape(np.shape(x))


def bf16_value(bits) -> np.ndarray:
    b = np.asarray(bits, np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def bf(x) -> np.ndarray:
    return bf16_value(bf16_bits(x))


def rmsnorm(x, w, eps):
    """x / sqrt(mean(x^2) + eps) * w along the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def rope(x, pos, theta):
    """x [T][heads][D], pos [T]: rotate pair (i, i + D/2) by pos * theta^(-2i/D)."""
    D = x.shape[-1]
    half = D // 2
    freq = theta ** (-2.0 * np.arange(half) / D)
    ang = np.asarray(pos, np.float64)[:, None] * freq[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x):
    return x / (1.0 + np.exp(-x))


def positions(batch) -> np.ndarray:
    q = np.diff(batch.q_start)
    return np.concatenate([batch.seq_lens[r] - q[r] + np.arange(q[r]) for r in range(len(q))]) \
        if len(q) else np.zeros(0, np.int64)


def forward(lw, pool, batch, hidden_bits):
    """One layer step.  pool: oracle.Pool (receives the new K/V); returns the
    output bf16 bits [T][H] and the intermediate tensors (fp64 values)."""
    H, Hq, Hkv, D, I = lw.hidden, lw.num_q_heads, lw.num_kv_heads, lw.head_dim, lw.intermediate
    f = lambda a: bf16_value(a)
    x = f(hidden_bits)
    T = x.shape[0]
    y = bf(rmsnorm(x, f(lw.attn_norm), lw.rms_eps))
    qkv = bf(y @ f(lw.w_qkv).T)
    q = qkv[:, :Hq * D].reshape(T, Hq, D)
    k = qkv[:, Hq * D:(Hq + Hkv) * D].reshape(T, Hkv, D)
    v = qkv[:, (Hq + Hkv) * D:].reshape(T, Hkv, D)
    pos = positions(batch)
    q = bf(rope(q, pos, lw.rope_theta))
    k = bf(rope(k, pos, lw.rope_theta))
    oracle.kv_append(pool, batch, bf16_bits(k), bf16_bits(v))
    att = oracle.attention(pool, batch, bf16_bits(q), Hq, 1.0 / np.sqrt(D)).reshape(T, Hq * D)
    a16 = bf(att)
    h = bf(x + a16 @ f(lw.w_o).T)
    y2 = bf(rmsnorm(h, f(lw.mlp_norm), lw.rms_eps))
    gu = bf(y2 @ f(lw.w_gate_up).T)
    act = bf(silu(gu[:, :I]) * gu[:, I:])
    out = bf(h + act @ f(lw.w_down).T)
    return bf16_bits(out), dict(y=y, qkv=qkv, q=q, k=k, v=v, attn=a16, h=h, y2=y2, gu=gu,
                                act=act, out=out)
