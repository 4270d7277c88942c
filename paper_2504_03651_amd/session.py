"""Device-resident state of one synthetic iteration, driven through the C ABI.

Used by the tests, the smoke check and the benchmark: it uploads a workload's
inputs, builds the starting pool by appending the workload's context through
``echo_kv_append`` onto a NaN-poisoned pool, and runs the iteration's three
calls (block copy, append, attention) on the current stream.
"""
from __future__ import annotations

import numpy as np

from . import echo
from .workload import KV_BF16


def _dev_u16(a, device):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device)


class Iteration:
    def __init__(self, w, device: str = "cuda", mirrors: bool = True, pool_blocks=None):
        import torch
        self.w = w
        self.device = device
        nb = w.num_blocks if pool_blocks is None else pool_blocks
        self.pool = echo.KVPool(nb, w.num_kv_heads, w.head_dim, w.kv_dtype != KV_BF16,
                                device).poison()
        ctx = echo.DeviceBatch(w.ctx, device)
        if w.ctx.num_rows:
            echo.kv_append(self.pool, ctx, _dev_u16(w.ctx_k, device), _dev_u16(w.ctx_v, device))
        self.batch = echo.DeviceBatch(w.batch, device, mirrors=mirrors)
        self.q = _dev_u16(w.q, device)
        self.k_new = _dev_u16(w.k_new, device)
        self.v_new = _dev_u16(w.v_new, device)
        T, Hq, D = w.batch.num_tokens, w.num_q_heads, w.head_dim
        self.out = torch.zeros((T, Hq, D), dtype=torch.float32, device=device)
        self.h_cow = np.ascontiguousarray(w.cow_pairs, np.int32).reshape(-1, 2)
        self.cow = torch.from_numpy(self.h_cow).to(device)
        self.workspace = None
        if w.batch.num_rows:
            n = echo.workspace_bytes(self.pool, self.batch, Hq)
            self.workspace = torch.empty(n, dtype=torch.uint8, device=device)

    def copy(self):
        if self.h_cow.shape[0]:
            echo.block_copy(self.pool, self.cow, self.h_cow)

    def append(self):
        echo.kv_append(self.pool, self.batch, self.k_new, self.v_new)

    def attend(self):
        ws = self.workspace
        if ws is None:
            import torch
            ws = torch.empty(256, dtype=torch.uint8, device=self.device)
        echo.attn_mixed(self.pool, self.batch, self.q, self.w.num_q_heads, self.w.sm_scale,
                        self.out, ws)

    def step(self):
        self.copy()
        self.append()
        self.attend()

    # host copies for comparisons
    def pool_host(self, blocks=None):
        """(K, V, k_scale, v_scale) as numpy, optionally only ``blocks``."""
        import torch
        idx = None if blocks is None else torch.from_numpy(
            np.ascontiguousarray(blocks, np.int64)).to(self.device)
        def get(t):
            if t is None:
                return None
            t = t if idx is None else t.index_select(0, idx)
            a = t.cpu().numpy()
            return a.view(np.uint16) if a.dtype == np.int16 else a
        p = self.pool
        return get(p.k), get(p.v), get(p.k_scale), get(p.v_scale)
