"""Python binding of the KV block manager (include/echo_kvm.h): marshalling only.

The manager is host code inside libecho.so; this wrapper converts token
lists to int32 arrays, raises EchoError on a failed call (except where a
caller asks for the status, as the scheduler does for ECHO_E_NOSPACE) and
returns the outputs as Python / NumPy values.
"""
from __future__ import annotations

import ctypes

import numpy as np

from . import echo

SYMBOLS = ["echo_kvm_create", "echo_kvm_destroy", "echo_kvm_register_offline",
           "echo_kvm_unregister_offline", "echo_kvm_start", "echo_kvm_append", "echo_kvm_fork",
           "echo_kvm_finish", "echo_kvm_tick", "echo_kvm_block_tables", "echo_kvm_take_copies",
           "echo_kvm_take_evictions", "echo_kvm_block_info", "echo_kvm_stats", "echo_kvm_probe",
           "echo_kvm_set_offline_limit"]

ONLINE, OFFLINE = 0, 1
EMPTY, HELD, CACHED = 0, 1, 2


class CBlockInfo(ctypes.Structure):
    _fields_ = [("state", ctypes.c_int32), ("holders", ctypes.c_int32), ("rc", ctypes.c_int32),
                ("task", ctypes.c_int32), ("lat", ctypes.c_int64), ("priority2", ctypes.c_int32),
                ("depth", ctypes.c_int32)]


class CStats(ctypes.Structure):
    _fields_ = [("empty", ctypes.c_int32), ("held", ctypes.c_int32), ("cached", ctypes.c_int32),
                ("running", ctypes.c_int32), ("now", ctypes.c_int64),
                ("hits_tokens", ctypes.c_int64), ("evictions", ctypes.c_int64),
                ("cached_reusable", ctypes.c_int32)]


_bound = False


def _lib():
    global _bound
    L = echo.lib()
    if not _bound:
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.echo_kvm_create.argtypes = [i32, i32, ctypes.POINTER(vp)]
        L.echo_kvm_destroy.argtypes = [vp]
        L.echo_kvm_destroy.restype = None
        L.echo_kvm_register_offline.argtypes = [vp, i64, vp, i32]
        L.echo_kvm_unregister_offline.argtypes = [vp, i64]
        L.echo_kvm_start.argtypes = [vp, i64, i32, vp, i32, ctypes.POINTER(i32)]
        L.echo_kvm_append.argtypes = [vp, i64, vp, i32]
        L.echo_kvm_fork.argtypes = [vp, i64, i64]
        L.echo_kvm_finish.argtypes = [vp, i64]
        L.echo_kvm_tick.argtypes = [vp]
        L.echo_kvm_block_tables.argtypes = [vp, vp, i32, i32, vp, vp]
        L.echo_kvm_take_copies.argtypes = [vp, vp, i32, ctypes.POINTER(i32)]
        L.echo_kvm_take_evictions.argtypes = [vp, vp, i32, ctypes.POINTER(i32)]
        L.echo_kvm_block_info.argtypes = [vp, i32, ctypes.POINTER(CBlockInfo)]
        L.echo_kvm_stats.argtypes = [vp, ctypes.POINTER(CStats)]
        L.echo_kvm_probe.argtypes = [vp, vp, i32, ctypes.POINTER(i32)]
        L.echo_kvm_set_offline_limit.argtypes = [vp, i32]
        for n in SYMBOLS:
            if n != "echo_kvm_destroy":
                getattr(L, n).restype = ctypes.c_int
        _bound = True
    return L


def _tok(tokens):
    a = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32).reshape(-1))
    return a, (a.ctypes.data if a.size else None), int(a.size)


class KVManager:
    """Owner of one echo_kvm_t.  Methods return what the C call outputs; with
    ``check=False`` they return (status, output) instead of raising."""

    def __init__(self, num_blocks: int, offline_limit: int | None = None):
        self.L = _lib()
        self.num_blocks = int(num_blocks)
        lim = self.num_blocks if offline_limit is None else int(offline_limit)
        h = ctypes.c_void_p()
        echo._check(self.L.echo_kvm_create(self.num_blocks, lim, ctypes.byref(h)), "echo_kvm_create")
        self.h = h

    def close(self):
        if self.h:
            self.L.echo_kvm_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _ret(self, code, where, out, check):
        if check:
            echo._check(code, where)
            return out
        return code, out

    def register_offline(self, req: int, tokens, check: bool = True):
        a, p, n = _tok(tokens)
        return self._ret(self.L.echo_kvm_register_offline(self.h, int(req), p, n),
                         "echo_kvm_register_offline", None, check)

    def unregister_offline(self, req: int, check: bool = True):
        return self._ret(self.L.echo_kvm_unregister_offline(self.h, int(req)),
                         "echo_kvm_unregister_offline", None, check)

    def start(self, seq: int, task: int, tokens, check: bool = True):
        """Returns the number of prompt tokens served from the cache."""
        a, p, n = _tok(tokens)
        c = ctypes.c_int32(-1)
        code = self.L.echo_kvm_start(self.h, int(seq), int(task), p, n, ctypes.byref(c))
        return self._ret(code, "echo_kvm_start", int(c.value), check)

    def probe(self, tokens) -> int:
        """Prompt tokens a start would find cached (no side effects)."""
        a, p, n = _tok(tokens)
        c = ctypes.c_int32(-1)
        echo._check(self.L.echo_kvm_probe(self.h, p, n, ctypes.byref(c)), "echo_kvm_probe")
        return int(c.value)

    def set_offline_limit(self, limit: int):
        echo._check(self.L.echo_kvm_set_offline_limit(self.h, int(limit)),
                    "echo_kvm_set_offline_limit")

    def append(self, seq: int, tokens, check: bool = True):
        a, p, n = _tok(tokens)
        return self._ret(self.L.echo_kvm_append(self.h, int(seq), p, n), "echo_kvm_append", None,
                         check)

    def fork(self, parent: int, child: int, check: bool = True):
        return self._ret(self.L.echo_kvm_fork(self.h, int(parent), int(child)), "echo_kvm_fork",
                         None, check)

    def finish(self, seq: int, check: bool = True):
        return self._ret(self.L.echo_kvm_finish(self.h, int(seq)), "echo_kvm_finish", None, check)

    def tick(self):
        echo._check(self.L.echo_kvm_tick(self.h), "echo_kvm_tick")

    def block_tables(self, seqs, max_blocks_per_row: int, check: bool = True):
        """(block_tables [rows][mbr] int32, seq_lens [rows] int32)."""
        s = np.ascontiguousarray(np.asarray(seqs, dtype=np.int64).reshape(-1))
        bt = np.full((len(s), int(max_blocks_per_row)), -1, np.int32)
        sl = np.zeros(len(s), np.int32)
        code = self.L.echo_kvm_block_tables(self.h, s.ctypes.data if len(s) else None, len(s),
                                            int(max_blocks_per_row),
                                            bt.ctypes.data if len(s) else None,
                                            sl.ctypes.data if len(s) else None)
        return self._ret(code, "echo_kvm_block_tables", (bt, sl), check)

    def take_copies(self, max_pairs: int = 1 << 16) -> np.ndarray:
        """Queued copy-on-write pairs as an int32 [k][2] array (src, dst)."""
        buf = np.zeros((max(int(max_pairs), 1), 2), np.int32)
        n = ctypes.c_int32(0)
        echo._check(self.L.echo_kvm_take_copies(self.h, buf.ctypes.data, int(max_pairs),
                                                ctypes.byref(n)), "echo_kvm_take_copies")
        return buf[:n.value].copy()

    def take_evictions(self, max_blocks: int = 1 << 16) -> list:
        buf = np.zeros(max(int(max_blocks), 1), np.int32)
        n = ctypes.c_int32(0)
        echo._check(self.L.echo_kvm_take_evictions(self.h, buf.ctypes.data, int(max_blocks),
                                                   ctypes.byref(n)), "echo_kvm_take_evictions")
        return buf[:n.value].tolist()

    def block_info(self, block: int) -> dict:
        i = CBlockInfo()
        echo._check(self.L.echo_kvm_block_info(self.h, int(block), ctypes.byref(i)),
                    "echo_kvm_block_info")
        return {n: int(getattr(i, n)) for n, _ in CBlockInfo._fields_}

    def stats(self) -> dict:
        st = CStats()
        echo._check(self.L.echo_kvm_stats(self.h, ctypes.byref(st)), "echo_kvm_stats")
        return {n: int(getattr(st, n)) for n, _ in CStats._fields_}
