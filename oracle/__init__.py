"""ctypes front end of the fp64 CPU oracle (``echo_oracle.c``).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The oracle shares no code with the
HIP library; both read their inputs from the seeded workload generator.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "echo_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

BF16_NAN = 0x7FC0
FP8_NAN = 0x7F


def build(src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle with gcc (no fast-math: fp64 as written)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", "-Wall", "-Wextra",
           "-I", _HERE, "-o", out + ".tmp", src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


class _Pool(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("k_scale", ctypes.c_void_p), ("v_scale", ctypes.c_void_p),
                ("num_blocks", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("kv_fp8", ctypes.c_int32)]


class _Batch(ctypes.Structure):
    _fields_ = [("num_rows", ctypes.c_int32), ("max_blocks_per_row", ctypes.c_int32),
                ("block_tables", ctypes.c_void_p), ("seq_lens", ctypes.c_void_p),
                ("q_start", ctypes.c_void_p), ("row_kind", ctypes.c_void_p)]


def load(path: str):
    """Open an oracle build at ``path`` and declare its signatures."""
    L = ctypes.CDLL(path)
    L.orc_kv_append.restype = ctypes.c_int
    L.orc_kv_append.argtypes = [ctypes.POINTER(_Pool), ctypes.POINTER(_Batch),
                                ctypes.c_void_p, ctypes.c_void_p]
    L.orc_block_copy.restype = ctypes.c_int
    L.orc_block_copy.argtypes = [ctypes.POINTER(_Pool), ctypes.c_void_p, ctypes.c_int32]
    L.orc_attention.restype = ctypes.c_int
    L.orc_attention.argtypes = [ctypes.POINTER(_Pool), ctypes.POINTER(_Batch),
                                ctypes.c_void_p, ctypes.c_int32, ctypes.c_float,
                                ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                ctypes.c_int32]
    L.orc_bf16_value.restype = ctypes.c_double
    L.orc_bf16_value.argtypes = [ctypes.c_uint16]
    L.orc_e4m3_value.restype = ctypes.c_double
    L.orc_e4m3_value.argtypes = [ctypes.c_uint8]
    L.orc_e4m3_encode.restype = ctypes.c_uint8
    L.orc_e4m3_encode.argtypes = [ctypes.c_float]
    L.orc_e4m3_fresh_scale.restype = ctypes.c_float
    L.orc_e4m3_fresh_scale.argtypes = [ctypes.c_float]
    return L


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        _lib = load(_LIB)
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class Pool:
    """Host copy of the paged pool: K [NB][Hkv][16][D], V [NB][Hkv][D][16]."""

    def __init__(self, num_blocks: int, num_kv_heads: int, head_dim: int, fp8: bool):
        self.fp8 = bool(fp8)
        self.num_blocks, self.num_kv_heads, self.head_dim = num_blocks, num_kv_heads, head_dim
        if self.fp8:
            self.k = np.full((num_blocks, num_kv_heads, 16, head_dim), FP8_NAN, np.uint8)
            self.v = np.full((num_blocks, num_kv_heads, head_dim, 16), FP8_NAN, np.uint8)
            self.k_scale = np.full((num_blocks, num_kv_heads), np.nan, np.float32)
            self.v_scale = np.full((num_blocks, num_kv_heads), np.nan, np.float32)
        else:
            self.k = np.full((num_blocks, num_kv_heads, 16, head_dim), BF16_NAN, np.uint16)
            self.v = np.full((num_blocks, num_kv_heads, head_dim, 16), BF16_NAN, np.uint16)
            self.k_scale = self.v_scale = None

    def _c(self) -> _Pool:
        return _Pool(_ptr(self.k), _ptr(self.v), _ptr(self.k_scale), _ptr(self.v_scale),
                     self.num_blocks, self.num_kv_heads, self.head_dim, int(self.fp8))

    def copy(self) -> "Pool":
        out = Pool.__new__(Pool)
        out.__dict__.update(self.__dict__)
        out.k, out.v = self.k.copy(), self.v.copy()
        if self.fp8:
            out.k_scale, out.v_scale = self.k_scale.copy(), self.v_scale.copy()
        return out


def _cbatch(batch):
    keep = [np.ascontiguousarray(batch.block_tables, np.int32),
            np.ascontiguousarray(batch.seq_lens, np.int32),
            np.ascontiguousarray(batch.q_start, np.int32),
            np.ascontiguousarray(batch.row_kind, np.uint8)]
    cb = _Batch(int(keep[1].shape[0]), int(keep[0].shape[1]), _ptr(keep[0]), _ptr(keep[1]),
                _ptr(keep[2]), _ptr(keep[3]))
    return cb, keep


def kv_append(pool: Pool, batch, k_new, v_new) -> None:
    cb, keep = _cbatch(batch)
    k_new = np.ascontiguousarray(k_new, np.uint16)
    v_new = np.ascontiguousarray(v_new, np.uint16)
    cp = pool._c()
    rc = lib().orc_kv_append(ctypes.byref(cp), ctypes.byref(cb), _ptr(k_new), _ptr(v_new))
    if rc != 0:
        raise ValueError("oracle append rejected the batch")


def block_copy(pool: Pool, pairs) -> None:
    pairs = np.ascontiguousarray(pairs, np.int32).reshape(-1, 2)
    cp = pool._c()
    if lib().orc_block_copy(ctypes.byref(cp), _ptr(pairs), int(pairs.shape[0])) != 0:
        raise ValueError("oracle copy rejected the pairs")


def attention(pool: Pool, batch, q, num_q_heads: int, sm_scale: float, sel=None,
              threads: int | None = None) -> np.ndarray:
    """fp64 outputs [n][D] for the query indices ``sel`` (t*Hq + h), or all."""
    cb, keep = _cbatch(batch)
    q = np.ascontiguousarray(q, np.uint16)
    T = int(batch.q_start[-1])
    if sel is None:
        n, sp = T * num_q_heads, None
    else:
        sel = np.ascontiguousarray(sel, np.int32)
        n, sp = int(sel.shape[0]), sel
    out = np.zeros((n, pool.head_dim), np.float64)
    threads = threads or os.cpu_count() or 1
    cp = pool._c()
    rc = lib().orc_attention(ctypes.byref(cp), ctypes.byref(cb), _ptr(q), int(num_q_heads),
                             float(sm_scale), _ptr(sp), n, _ptr(out), int(threads))
    if rc != 0:
        raise ValueError("oracle attention rejected the input")
    return out


def bf16_value(bits: int) -> float:
    return lib().orc_bf16_value(int(bits))


def e4m3_value(code: int) -> float:
    return lib().orc_e4m3_value(int(code))


def e4m3_encode(x: float) -> int:
    return lib().orc_e4m3_encode(float(x))


def e4m3_fresh_scale(amax: float) -> float:
    return lib().orc_e4m3_fresh_scale(float(amax))


def prepare(w, pool_blocks=None):
    """Starting pool for workload ``w``: poisoned, then the context appended."""
    pool = Pool(w.num_blocks if pool_blocks is None else pool_blocks, w.num_kv_heads,
                w.head_dim, w.kv_dtype != "bf16")
    kv_append(pool, w.ctx, w.ctx_k, w.ctx_v)
    return pool


def run_iteration(w, pool: Pool | None = None, sel=None, threads=None):
    """copy -> append -> attention for workload ``w``; returns (pool, out)."""
    pool = prepare(w) if pool is None else pool
    if w.cow_pairs.shape[0]:
        block_copy(pool, w.cow_pairs)
    kv_append(pool, w.batch, w.k_new, w.v_new)
    out = attention(pool, w.batch, w.q, w.num_q_heads, w.sm_scale, sel=sel, threads=threads)
    return pool, out
