"""Python binding of the decoder layer (include/echo_layer.h): marshalling only.

Uploads a layer's weights to device memory with PyTorch and calls
echo_layer_forward on PyTorch's current stream; every step runs in the
library (HIP kernels and hipBLASLt).
"""
from __future__ import annotations

import ctypes

import numpy as np

from . import echo

SYMBOLS = ["echo_layer_workspace_bytes", "echo_layer_forward", "echo_layer_timing"]


class CLayer(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("intermediate", ctypes.c_int32), ("rope_theta", ctypes.c_float),
                ("rms_eps", ctypes.c_float),
                ("attn_norm", ctypes.c_void_p), ("w_qkv", ctypes.c_void_p),
                ("w_o", ctypes.c_void_p), ("mlp_norm", ctypes.c_void_p),
                ("w_gate_up", ctypes.c_void_p), ("w_down", ctypes.c_void_p)]


class CLayerTiming(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float) for n in ("norm_ms", "qkv_ms", "rope_ms", "append_ms",
                                              "attention_ms", "o_ms", "mlp_ms", "other_ms")]


_bound = False


def _lib():
    global _bound
    L = echo.lib()
    if not _bound:
        P, B, vp = ctypes.POINTER(CLayer), ctypes.POINTER(echo.CPool), ctypes.c_void_p
        L.echo_layer_workspace_bytes.argtypes = [P, B, ctypes.POINTER(echo.CBatch)]
        L.echo_layer_workspace_bytes.restype = ctypes.c_size_t
        L.echo_layer_forward.argtypes = [P, B, ctypes.POINTER(echo.CBatch), vp, vp,
                                         ctypes.c_size_t, vp, ctypes.c_size_t, vp]
        L.echo_layer_forward.restype = ctypes.c_int
        L.echo_layer_timing.argtypes = [ctypes.POINTER(CLayerTiming)]
        L.echo_layer_timing.restype = ctypes.c_int
        _bound = True
    return L


class Layer:
    """Device copy of a ``workload.LayerWeights``."""

    def __init__(self, lw, device: str = "cuda"):
        import torch
        self.lw = lw
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device)
        self.t = {n: dev(getattr(lw, n)) for n in ("attn_norm", "w_qkv", "w_o", "mlp_norm",
                                                    "w_gate_up", "w_down")}
        self.c = CLayer(lw.hidden, lw.num_q_heads, lw.num_kv_heads, lw.head_dim, lw.intermediate,
                        lw.rope_theta, lw.rms_eps,
                        *[self.t[n].data_ptr() for n in ("attn_norm", "w_qkv", "w_o", "mlp_norm",
                                                         "w_gate_up", "w_down")])

    def workspace_bytes(self, pool, batch) -> int:
        cp, cb = pool.c(), batch.c()
        n = _lib().echo_layer_workspace_bytes(ctypes.byref(self.c), ctypes.byref(cp),
                                              ctypes.byref(cb))
        if n == 0:
            raise echo.EchoError(echo.ECHO_E_INVALID, "echo_layer_workspace_bytes", echo.last_error())
        return int(n)

    def forward(self, pool, batch, hidden, workspace, stream=None, host_workspace=None) -> None:
        """hidden: device int16 tensor [T][H] (bf16 bits), overwritten.  The
        attention plan goes through ``host_workspace`` (the calling thread's
        pinned ring by default) when the batch has host mirrors."""
        import torch
        cp, cb = pool.c(), batch.c()
        s = torch.cuda.current_stream() if stream is None else stream
        hptr, hsize, slot, hw = None, 0, None, None
        if batch.mirrors and batch.num_rows:
            hw = host_workspace or echo.default_host_workspace()
            hptr, hsize, slot = hw.acquire(echo.host_workspace_bytes(pool, batch,
                                                                     self.lw.num_q_heads))
        echo._check(_lib().echo_layer_forward(
            ctypes.byref(self.c), ctypes.byref(cp), ctypes.byref(cb), hidden.data_ptr(),
            workspace.data_ptr(), workspace.numel() * workspace.element_size(),
            hptr, hsize, ctypes.c_void_p(s.cuda_stream)), "echo_layer_forward")
        if slot is not None:
            hw.release(slot, s)


def timing() -> dict:
    t = CLayerTiming()
    echo._check(_lib().echo_layer_timing(ctypes.byref(t)), "echo_layer_timing")
    return {n: float(getattr(t, n)) for n, _ in CLayerTiming._fields_}
