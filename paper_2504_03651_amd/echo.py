"""Python binding of libecho.so (include/echo.h): argument marshalling only.

Every step of the iteration runs in the HIP library; this module allocates
device buffers with PyTorch, fills the C structs and calls the entry points
on PyTorch's current stream.  If the library has not been built, every call
raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# ECHO_LIBRARY selects another build of the library (the sanitized one of
# build.build_sanitized(), for the host-only tests)
LIB_PATH = os.environ.get("ECHO_LIBRARY") or os.path.join(_PKG, "libecho.so")

ECHO_OK = 0
ECHO_E_INVALID = -1
ECHO_E_RANGE = -2
ECHO_E_ALIAS_WRITE = -3
ECHO_E_WORKSPACE = -4
ECHO_E_UNSUPPORTED = -5
ECHO_E_HIP = -6
ECHO_E_NOSPACE = -7
KV_BF16 = 0
KV_FP8_E4M3 = 1

SYMBOLS = ["echo_kv_append", "echo_attn_mixed", "echo_attn_workspace_bytes",
           "echo_attn_host_workspace_bytes", "echo_attn_mixed_static", "echo_block_copy",
           "echo_attn_plan_stats", "echo_attn_plan_pack", "echo_validate", "echo_status_string",
           "echo_last_error",
           "echo_profile", "echo_attn_timing"]


class EchoError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str):
        super().__init__(f"{where}: {status_string(code)} ({code}): {detail}")
        self.code = code


class CPool(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("k_scale", ctypes.c_void_p), ("v_scale", ctypes.c_void_p),
                ("num_blocks", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("dtype", ctypes.c_int32)]


class CBatch(ctypes.Structure):
    _fields_ = [("num_rows", ctypes.c_int32), ("max_blocks_per_row", ctypes.c_int32),
                ("num_tokens", ctypes.c_int32), ("max_q_len", ctypes.c_int32),
                ("max_seq_len", ctypes.c_int32),
                ("block_tables", ctypes.c_void_p), ("seq_lens", ctypes.c_void_p),
                ("q_start", ctypes.c_void_p), ("row_kind", ctypes.c_void_p),
                ("h_block_tables", ctypes.c_void_p), ("h_seq_lens", ctypes.c_void_p),
                ("h_q_start", ctypes.c_void_p), ("h_row_kind", ctypes.c_void_p)]


class CPlanStats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in (
        "work_items", "decode_items", "prefill_items", "shared_segments", "partial_slots",
        "merged_queries", "unique_kv_tokens", "logical_kv_tokens", "causal_pairs",
        "decode_kv_tokens", "prefill_causal_pairs", "workspace_bytes")]


class CPlanLayout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in (
        "n_desc", "n_pdesc", "n_tok_list", "n_tokens", "n_merge_rows", "n_merge_entries", "n_slots",
        "off_desc", "off_pdesc", "off_tok_list", "off_klim", "off_merge_tok", "off_merge_ptr",
        "off_merge_ent", "upload_words", "off_part_lse", "off_part_o", "total_words")] + [
        ("head_chunks", ctypes.c_int32), ("heads_per_chunk", ctypes.c_int32)]


class CAttnTiming(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float) for n in ("upload_ms", "prefill_ms", "decode_ms", "merge_ms")]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -c 'import __graft_entry__ as g; g.build()'`")
        L = ctypes.CDLL(LIB_PATH)
        P, B, vp = ctypes.POINTER(CPool), ctypes.POINTER(CBatch), ctypes.c_void_p
        L.echo_kv_append.argtypes = [P, B, vp, vp, vp]
        L.echo_attn_mixed.argtypes = [P, B, vp, ctypes.c_int32, ctypes.c_float, vp, vp,
                                      ctypes.c_size_t, vp, ctypes.c_size_t, vp]
        L.echo_attn_workspace_bytes.argtypes = [P, B, ctypes.c_int32]
        L.echo_attn_workspace_bytes.restype = ctypes.c_size_t
        L.echo_attn_mixed_static.argtypes = [P, B, vp, ctypes.c_int32, ctypes.c_float, vp, vp]
        L.echo_attn_mixed_static.restype = ctypes.c_int
        L.echo_attn_host_workspace_bytes.argtypes = [P, B, ctypes.c_int32]
        L.echo_attn_host_workspace_bytes.restype = ctypes.c_size_t
        L.echo_block_copy.argtypes = [P, vp, ctypes.c_int32, vp, vp]
        L.echo_attn_plan_stats.argtypes = [P, B, ctypes.c_int32, ctypes.POINTER(CPlanStats)]
        L.echo_attn_plan_pack.argtypes = [P, B, ctypes.c_int32, ctypes.POINTER(CPlanLayout), vp,
                                          ctypes.c_size_t]
        L.echo_validate.argtypes = [P, B, ctypes.c_int32]
        L.echo_status_string.argtypes = [ctypes.c_int]
        L.echo_status_string.restype = ctypes.c_char_p
        L.echo_last_error.argtypes = []
        L.echo_last_error.restype = ctypes.c_char_p
        L.echo_profile.argtypes = [ctypes.c_int]
        L.echo_profile.restype = ctypes.c_int
        L.echo_attn_timing.argtypes = [ctypes.POINTER(CAttnTiming)]
        L.echo_attn_timing.restype = ctypes.c_int
        # the HIP runtime libecho.so links against, for caller-owned pinned memory
        L.hipHostMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t, ctypes.c_uint]
        L.hipHostMalloc.restype = ctypes.c_int
        L.hipHostFree.argtypes = [ctypes.c_void_p]
        L.hipHostFree.restype = ctypes.c_int
        for name in ("echo_kv_append", "echo_attn_mixed", "echo_block_copy",
                     "echo_attn_plan_stats", "echo_attn_plan_pack", "echo_validate"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(code: int) -> str:
    return lib().echo_status_string(int(code)).decode()


def last_error() -> str:
    return lib().echo_last_error().decode()


def _check(code: int, where: str) -> None:
    if code != ECHO_OK:
        raise EchoError(code, where, last_error())


def _np_ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


# ---------------------------------------------------------------- device data


class KVPool:
    """A paged KV pool in device memory: K [NB][Hkv][16][D], V [NB][Hkv][D][16]."""

    def __init__(self, num_blocks: int, num_kv_heads: int, head_dim: int, fp8: bool = False,
                 device: str = "cuda"):
        import torch
        self.num_blocks, self.num_kv_heads, self.head_dim = num_blocks, num_kv_heads, head_dim
        self.fp8 = bool(fp8)
        et = torch.uint8 if self.fp8 else torch.int16
        self.k = torch.empty((num_blocks, num_kv_heads, 16, head_dim), dtype=et, device=device)
        self.v = torch.empty((num_blocks, num_kv_heads, head_dim, 16), dtype=et, device=device)
        if self.fp8:
            self.k_scale = torch.empty((num_blocks, num_kv_heads), dtype=torch.float32,
                                       device=device)
            self.v_scale = torch.empty_like(self.k_scale)
        else:
            self.k_scale = self.v_scale = None

    def poison(self) -> "KVPool":
        """Fill every slot with NaN codes (unwritten slots must never matter)."""
        self.k.fill_(0x7F if self.fp8 else 0x7FC0)
        self.v.fill_(0x7F if self.fp8 else 0x7FC0)
        if self.fp8:
            self.k_scale.fill_(float("nan"))
            self.v_scale.fill_(float("nan"))
        return self

    def c(self) -> CPool:
        return CPool(self.k.data_ptr(), self.v.data_ptr(),
                     self.k_scale.data_ptr() if self.fp8 else None,
                     self.v_scale.data_ptr() if self.fp8 else None,
                     self.num_blocks, self.num_kv_heads, self.head_dim, 16,
                     KV_FP8_E4M3 if self.fp8 else KV_BF16)


class DeviceBatch:
    """Row metadata on the device plus its host mirrors (kept alive here)."""

    def __init__(self, batch, device: str = "cuda", mirrors: bool = True):
        import torch
        self.h_bt = np.ascontiguousarray(batch.block_tables, np.int32)
        self.h_sl = np.ascontiguousarray(batch.seq_lens, np.int32)
        self.h_qs = np.ascontiguousarray(batch.q_start, np.int32)
        self.h_kind = np.ascontiguousarray(batch.row_kind, np.uint8)
        self.num_rows = int(self.h_sl.shape[0])
        self.mbr = int(self.h_bt.shape[1])
        self.num_tokens = int(self.h_qs[-1])
        q = np.diff(self.h_qs)
        self.max_q_len = int(q.max()) if self.num_rows else 1
        self.max_seq_len = int(self.h_sl.max()) if self.num_rows else 1
        self.mirrors = mirrors
        self.bt = torch.from_numpy(self.h_bt).to(device)
        self.sl = torch.from_numpy(self.h_sl).to(device)
        self.qs = torch.from_numpy(self.h_qs).to(device)
        self.kind = torch.from_numpy(self.h_kind).to(device)

    def c(self) -> CBatch:
        m = self.mirrors
        return CBatch(self.num_rows, self.mbr, self.num_tokens, self.max_q_len, self.max_seq_len,
                      self.bt.data_ptr(), self.sl.data_ptr(), self.qs.data_ptr(),
                      self.kind.data_ptr(),
                      _np_ptr(self.h_bt) if m else None, _np_ptr(self.h_sl) if m else None,
                      _np_ptr(self.h_qs) if m else None, _np_ptr(self.h_kind) if m else None)


# ---------------------------------------------------------------- entry points


def kv_append(pool: KVPool, batch: DeviceBatch, k_new, v_new, stream=None) -> None:
    cp, cb = pool.c(), batch.c()
    _check(lib().echo_kv_append(ctypes.byref(cp), ctypes.byref(cb), k_new.data_ptr(),
                                v_new.data_ptr(), _stream(stream)), "echo_kv_append")


def workspace_bytes(pool: KVPool, batch: DeviceBatch, num_q_heads: int) -> int:
    cp, cb = pool.c(), batch.c()
    n = lib().echo_attn_workspace_bytes(ctypes.byref(cp), ctypes.byref(cb), int(num_q_heads))
    if n == 0 and batch.num_rows:
        raise EchoError(ECHO_E_INVALID, "echo_attn_workspace_bytes", last_error())
    return int(n)


def host_workspace_bytes(pool: KVPool, batch: DeviceBatch, num_q_heads: int) -> int:
    cp, cb = pool.c(), batch.c()
    return int(lib().echo_attn_host_workspace_bytes(ctypes.byref(cp), ctypes.byref(cb),
                                                    int(num_q_heads)))


# hipHostMalloc flags: mapped into the device address space, and coherent
# (the device reads it uncached, so it sees what the host last wrote)
_HOST_MAPPED_COHERENT = 0x2 | 0x40000000


class HostWorkspace:
    """Caller-owned pinned host memory for the plans echo_attn_mixed packs
    and uploads.  A ring of buffers: a buffer is handed out again only after
    an event recorded behind the call that used it has completed, so the
    host never rewrites a plan the device has not read yet.  The HIP runtime
    is the one libecho.so is linked against (resolved through its handle)."""

    def __init__(self, slots: int = 4):
        self._bufs = [(None, 0)] * slots
        self._events = [None] * slots
        self._next = 0

    def acquire(self, nbytes: int):
        """(pointer, size, slot) of a buffer of at least ``nbytes`` bytes."""
        i = self._next
        self._next = (i + 1) % len(self._bufs)
        ev = self._events[i]
        if ev is not None:
            ev.synchronize()
            self._events[i] = None
        ptr, size = self._bufs[i]
        if size < nbytes:
            L = lib()
            if ptr:
                L.hipHostFree(ctypes.c_void_p(ptr))
                self._bufs[i] = (None, 0)
            size = max(int(nbytes * 1.5), 1 << 16)
            p = ctypes.c_void_p()
            rc = L.hipHostMalloc(ctypes.byref(p), ctypes.c_size_t(size),
                                 ctypes.c_uint(_HOST_MAPPED_COHERENT))
            if rc != 0:
                raise MemoryError(f"hipHostMalloc({size}) failed with HIP error {rc}")
            ptr = p.value
            self._bufs[i] = (ptr, size)
        return ptr, size, i

    def release(self, slot: int, stream) -> None:
        """Record that the work enqueued on ``stream`` so far reads ``slot``."""
        import torch
        ev = torch.cuda.Event()
        ev.record(stream)
        self._events[slot] = ev

    def close(self) -> None:
        for i, (ptr, _) in enumerate(self._bufs):
            if self._events[i] is not None:
                self._events[i].synchronize()
            if ptr:
                lib().hipHostFree(ctypes.c_void_p(ptr))
        self._bufs = [(None, 0)] * len(self._bufs)
        self._events = [None] * len(self._bufs)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


_default_host_ws = {}


def default_host_workspace() -> HostWorkspace:
    """One host-workspace ring per Python thread."""
    import threading
    k = threading.get_ident()
    if k not in _default_host_ws:
        _default_host_ws[k] = HostWorkspace()
    return _default_host_ws[k]


def attn_mixed(pool: KVPool, batch: DeviceBatch, q, num_q_heads: int, sm_scale: float, out,
               workspace, stream=None, host_workspace: HostWorkspace | None = None) -> None:
    """echo_attn_mixed.  With host mirrors the plan goes through a pinned
    host buffer of ``host_workspace`` (the calling thread's ring by default);
    without them the library plans on the device and no host buffer is used."""
    import torch
    cp, cb = pool.c(), batch.c()
    s = torch.cuda.current_stream() if stream is None else stream
    hptr, hsize, slot = None, 0, None
    if batch.mirrors and batch.num_rows:
        hw = host_workspace or default_host_workspace()
        need = host_workspace_bytes(pool, batch, num_q_heads)
        hptr, hsize, slot = hw.acquire(need)
    _check(lib().echo_attn_mixed(ctypes.byref(cp), ctypes.byref(cb), q.data_ptr(),
                                 int(num_q_heads), float(sm_scale), out.data_ptr(),
                                 workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                                 hptr, hsize, ctypes.c_void_p(s.cuda_stream)), "echo_attn_mixed")
    if slot is not None:
        hw.release(slot, s)


def attn_mixed_static(pool: KVPool, batch: DeviceBatch, q, num_q_heads: int, sm_scale: float,
                      out, stream=None) -> None:
    """echo_attn_mixed_static: no workspace, the library's static scratch."""
    cp, cb = pool.c(), batch.c()
    _check(lib().echo_attn_mixed_static(ctypes.byref(cp), ctypes.byref(cb), q.data_ptr(),
                                        int(num_q_heads), float(sm_scale), out.data_ptr(),
                                        _stream(stream)), "echo_attn_mixed_static")


def block_copy(pool: KVPool, pairs, h_pairs=None, stream=None) -> None:
    n = int(pairs.shape[0])
    hp = None if h_pairs is None else np.ascontiguousarray(h_pairs, np.int32)
    cp = pool.c()
    _check(lib().echo_block_copy(ctypes.byref(cp), pairs.data_ptr() if n else None, n,
                                 _np_ptr(hp), _stream(stream)), "echo_block_copy")


def plan_stats(cpool: CPool, cbatch: CBatch, num_q_heads: int) -> dict:
    st = CPlanStats()
    _check(lib().echo_attn_plan_stats(ctypes.byref(cpool), ctypes.byref(cbatch),
                                      int(num_q_heads), ctypes.byref(st)), "echo_attn_plan_stats")
    return {name: int(getattr(st, name)) for name, _ in CPlanStats._fields_}


def plan_pack(cpool: CPool, cbatch: CBatch, num_q_heads: int):
    """(layout dict, int32 words) of the plan echo_attn_mixed would upload."""
    lay = CPlanLayout()
    _check(lib().echo_attn_plan_pack(ctypes.byref(cpool), ctypes.byref(cbatch), int(num_q_heads),
                                     ctypes.byref(lay), None, 0), "echo_attn_plan_pack")
    words = np.full(max(int(lay.upload_words), 1), -1, np.int32)   # words the packer skips stay -1
    _check(lib().echo_attn_plan_pack(ctypes.byref(cpool), ctypes.byref(cbatch), int(num_q_heads),
                                     ctypes.byref(lay), words.ctypes.data, words.nbytes),
           "echo_attn_plan_pack")
    return {name: int(getattr(lay, name)) for name, _ in CPlanLayout._fields_}, words


def profile(enable: bool) -> bool:
    """Turn per-kernel event timing of echo_attn_mixed on or off (this thread)."""
    return bool(lib().echo_profile(int(enable)))


def attn_timing() -> dict:
    """Per-kernel milliseconds of this thread's last profiled echo_attn_mixed."""
    t = CAttnTiming()
    _check(lib().echo_attn_timing(ctypes.byref(t)), "echo_attn_timing")
    return {name: float(getattr(t, name)) for name, _ in CAttnTiming._fields_}


def validate(cpool: CPool, cbatch: CBatch, for_append: bool) -> int:
    return int(lib().echo_validate(ctypes.byref(cpool), ctypes.byref(cbatch), int(for_append)))


def host_structs(w, fake_device_ptr: int = 0x1000):
    """C structs of workload ``w`` for host-only calls (validation, plan
    statistics): device pointers are placeholders that are never touched."""
    bt = np.ascontiguousarray(w.batch.block_tables, np.int32)
    sl = np.ascontiguousarray(w.batch.seq_lens, np.int32)
    qs = np.ascontiguousarray(w.batch.q_start, np.int32)
    kd = np.ascontiguousarray(w.batch.row_kind, np.uint8)
    fp8 = w.kv_dtype != "bf16"
    p = fake_device_ptr
    cpool = CPool(p, p, p if fp8 else None, p if fp8 else None, w.num_blocks, w.num_kv_heads,
                  w.head_dim, 16, KV_FP8_E4M3 if fp8 else KV_BF16)
    q = np.diff(qs)
    cb = CBatch(int(sl.shape[0]), int(bt.shape[1]), int(qs[-1]),
                int(q.max()) if len(q) else 1, int(sl.max()) if len(sl) else 1,
                p, p, p, p, _np_ptr(bt), _np_ptr(sl), _np_ptr(qs), _np_ptr(kd))
    return cpool, cb, (bt, sl, qs, kd)
