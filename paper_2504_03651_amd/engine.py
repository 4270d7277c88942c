"""Runs the scheduler simulation's batches on the GPU through the hot path.

An ``AttentionEngine`` owns a device KV pool of the simulator's block count and
executes each iteration's batch exactly as the simulator's KV block manager
lays it out: its block tables and sequence lengths become the rows of an
``echo_kv_append`` + ``echo_attn_mixed`` call (prefill chunks and decode
tokens, with seeded N(0, 1) bf16 Q/K/V for the new tokens, drawn on the
device; there is no model), so the manager's tables, evictions and prefix hits all reach the
kernels.  The GPU time of each call (host planning excluded) is measured with
events on the stream, to set against the estimator's prediction for the same
batch.
"""
from __future__ import annotations

import numpy as np

from . import echo
from . import workload as W
from .calibrate import GATE_CYCLES

BS = 16


class AttentionEngine:
    def __init__(self, num_blocks: int, num_q_heads: int = 32, num_kv_heads: int = 8,
                 head_dim: int = 128, seed: int = 0, device: str = "cuda", observer=None):
        import torch
        self.torch = torch
        self.Hq, self.Hkv, self.D = num_q_heads, num_kv_heads, head_dim
        self.pool = echo.KVPool(num_blocks, num_kv_heads, head_dim, False, device).poison()
        self.gen = torch.Generator(device=device)
        self.gen.manual_seed(seed)
        self.device = device
        self.ws = None
        self.ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        self.calls = 0
        self.gate_cycles = GATE_CYCLES
        # optional: called after each batch as observer(engine, manager, batch,
        # rows, q, k_new, v_new, out) with the host inputs (rows: a
        # workload.Batch; q, k_new, v_new: bf16 bits) and the device output,
        # for checking the results outside the product path
        self.observer = observer

    def _bf16(self, shape):
        """Seeded N(0, 1) values rounded to bf16, drawn on the device (int16 bits)."""
        torch = self.torch
        x = torch.randn(shape, generator=self.gen, device=self.device, dtype=torch.float32)
        return x.to(torch.bfloat16).view(torch.int16)

    def __call__(self, manager, batch) -> float:
        """Runs one batch (list of (request, "prefill" | "decode", new tokens))
        whose KV blocks `manager` already holds; returns the GPU time in ms."""
        torch = self.torch
        seqs = [r.seq for r, kind, n in batch]
        mbr = max(1, max(-(-(r.computed + r.generated + 1) // BS) for r, k, n in batch))
        while True:
            code, out = manager.block_tables(seqs, mbr, check=False)
            if code == 0:
                break
            mbr *= 2
        bt, sl = out
        # what the kernel-level estimate needs: each prefill chunk's cached
        # context and the distinct KV tokens the decode rows read
        seen = {}
        for i, (r, k, n) in enumerate(batch):
            if k == "decode":
                L = int(sl[i])
                for j in range(-(-L // BS)):
                    b = int(bt[i, j])
                    seen[b] = max(seen.get(b, 0), min(BS, L - BS * j))
        self.last_shape = dict(
            prefill=[(n, int(sl[i]) - n) for i, (r, k, n) in enumerate(batch) if k == "prefill"],
            decode=[int(sl[i]) for i, (r, k, n) in enumerate(batch) if k == "decode"],
            decode_unique=sum(seen.values()))
        q = np.array([n for r, kind, n in batch], np.int32)
        kind = np.array([W.PREFILL if k == "prefill" else W.DECODE for r, k, n in batch], np.uint8)
        b = W.Batch(bt, sl, np.concatenate([[0], np.cumsum(q)]).astype(np.int32), kind)
        T = int(q.sum())
        qd = self._bf16((T, self.Hq, self.D))
        kd = self._bf16((T, self.Hkv, self.D))
        vd = self._bf16((T, self.Hkv, self.D))
        db = echo.DeviceBatch(b, self.device)
        n = echo.workspace_bytes(self.pool, db, self.Hq)
        if self.ws is None or self.ws.numel() < n:
            self.ws = torch.empty(max(n, 1 << 20), dtype=torch.uint8, device=self.device)
        out_t = torch.empty((T, self.Hq, self.D), dtype=torch.float32, device=self.device)
        # The events bracket GPU work only: a short spin keeps the stream busy
        # while the host validates and plans the two calls, so the first event
        # fires with their kernels already queued behind it.
        torch.cuda._sleep(self.gate_cycles)
        self.ev[0].record()
        echo.kv_append(self.pool, db, kd, vd)
        echo.attn_mixed(self.pool, db, qd, self.Hq, 1.0 / float(np.sqrt(self.D)), out_t, self.ws)
        self.ev[1].record()
        torch.cuda.synchronize()
        self.calls += 1
        self.last_out = out_t
        ms = float(self.ev[0].elapsed_time(self.ev[1]))
        if self.observer is not None:
            host = lambda t: t.cpu().numpy().view(np.uint16)
            self.observer(self, manager, batch, b, host(qd), host(kd), host(vd), out_t)
        return ms
