"""Host-side checks of the C ABI: the library loads on a machine without a
GPU, exports every symbol the header declares, and its validation and
planning (pure host code) behave as documented.  No GPU work is enqueued:
every call here either fails validation or is a host-only entry point."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2504_03651_amd import echo
from paper_2504_03651_amd import workload as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    from paper_2504_03651_amd import kvm, layer
    lib = ctypes.CDLL(echo.LIB_PATH)
    for hdr, bound in (("echo.h", echo.SYMBOLS), ("echo_kvm.h", kvm.SYMBOLS),
                       ("echo_layer.h", layer.SYMBOLS)):
        header = open(os.path.join(ROOT, "include", hdr)).read()
        declared = set(re.findall(r"\b(echo_[a-z0-9_]+)\s*\(", header))
        assert declared >= set(bound), hdr
        assert declared, hdr
        for name in declared:
            assert hasattr(lib, name), name


def test_status_strings():
    for code, name in [(0, "ECHO_OK"), (-1, "ECHO_E_INVALID"), (-3, "ECHO_E_ALIAS_WRITE"),
                       (-6, "ECHO_E_HIP"), (-7, "ECHO_E_NOSPACE")]:
        assert echo.status_string(code) == name


def _structs(w):
    return echo.host_structs(w)


def test_valid_batches_pass_validation():
    for w in (W.config1(), W.random_case(1), W.random_case(2, kv_dtype=W.KV_FP8)):
        cp, cb, keep = _structs(w)
        assert echo.validate(cp, cb, True) == echo.ECHO_OK, echo.last_error()
        assert echo.validate(cp, cb, False) == echo.ECHO_OK


def test_block_id_out_of_range():
    w = W.config1()
    w.batch.block_tables[1, 0] = w.num_blocks
    cp, cb, keep = _structs(w)
    assert echo.validate(cp, cb, False) == echo.ECHO_E_RANGE
    assert "outside" in echo.last_error()


def test_decode_row_with_two_tokens():
    w = W.config1()
    w.batch.row_kind[1] = W.DECODE  # row 1 is a 32-token chunk
    cp, cb, keep = _structs(w)
    assert echo.validate(cp, cb, False) == echo.ECHO_E_INVALID


def test_append_into_aliased_block_is_rejected():
    w = W.config1()
    bt = w.batch.block_tables
    # row 2 (decode, context 37) appends into its block 2; alias it from row 0
    bt[0, 3] = bt[2, 2]
    cp, cb, keep = _structs(w)
    assert echo.validate(cp, cb, True) == echo.ECHO_E_ALIAS_WRITE
    assert echo.validate(cp, cb, False) == echo.ECHO_OK  # attention alone may alias


def test_two_rows_writing_one_block_is_rejected():
    w = W.config1()
    bt = w.batch.block_tables
    bt[1, 0] = bt[3, 3]  # both prefill rows would write the same block
    cp, cb, keep = _structs(w)
    assert echo.validate(cp, cb, True) == echo.ECHO_E_ALIAS_WRITE


def test_unsupported_head_dim_and_block_size():
    w = W.config1()
    cp, cb, keep = _structs(w)
    cp.head_dim = 96
    assert echo.validate(cp, cb, False) == echo.ECHO_E_UNSUPPORTED
    cp.head_dim = 64
    cp.block_size = 32
    assert echo.validate(cp, cb, False) == echo.ECHO_E_UNSUPPORTED


def test_fp8_pool_needs_scales():
    w = W.random_case(3, kv_dtype=W.KV_FP8)
    cp, cb, keep = _structs(w)
    cp.k_scale = None
    assert echo.validate(cp, cb, True) == echo.ECHO_E_INVALID


def test_q_start_must_start_at_zero_and_end_at_num_tokens():
    w = W.config1()
    cp, cb, (bt, sl, qs, kd) = _structs(w)
    cb.num_tokens = cb.num_tokens + 1
    assert echo.validate(cp, cb, False) == echo.ECHO_E_INVALID
    cb.num_tokens -= 1
    qs[0] = 1
    assert echo.validate(cp, cb, False) == echo.ECHO_E_INVALID


def test_extreme_q_start_and_lengths_are_rejected():
    # caller values at the ends of int32: rejected by the checks, with no
    # overflow on the way (the sanitized build runs this test too)
    w = W.config1()
    cp, cb, (bt, sl, qs, kd) = _structs(w)
    qs[2] = -2**31            # q of row 1 negative, row 2 huge
    assert echo.validate(cp, cb, False) == echo.ECHO_E_INVALID
    cp, cb, (bt, sl, qs, kd) = _structs(w)
    sl[0] = 2**31 - 1          # beyond max_seq_len
    assert echo.validate(cp, cb, False) == echo.ECHO_E_INVALID
    cp, cb, keep = _structs(w)
    cb.max_seq_len = 2**30 + 1
    cb.max_blocks_per_row = 2**27
    assert echo.validate(cp, cb, False) == echo.ECHO_E_UNSUPPORTED


def test_partial_mirrors_rejected():
    w = W.config1()
    cp, cb, keep = _structs(w)
    cb.h_row_kind = None
    assert echo.validate(cp, cb, False) == echo.ECHO_E_INVALID


def test_attention_without_mirrors_sizes_from_scalars():
    # without host mirrors the plan is built on the device: the workspace is a
    # bound from the scalar fields and no host workspace is needed
    w = W.config1()
    cp, cb, keep = _structs(w)
    L = echo.lib()
    with_mirrors = L.echo_attn_workspace_bytes(ctypes.byref(cp), ctypes.byref(cb), 4)
    assert L.echo_attn_host_workspace_bytes(ctypes.byref(cp), ctypes.byref(cb), 4) > 0
    cb.h_block_tables = cb.h_seq_lens = cb.h_q_start = cb.h_row_kind = None
    n = L.echo_attn_workspace_bytes(ctypes.byref(cp), ctypes.byref(cb), 4)
    assert n > 0 and n % 256 == 0 and with_mirrors > 0
    assert L.echo_attn_host_workspace_bytes(ctypes.byref(cp), ctypes.byref(cb), 4) == 0
    # the bound grows with the scalars it is taken from
    mbr, msl = cb.max_blocks_per_row, cb.max_seq_len
    cb.max_blocks_per_row, cb.max_seq_len = 64, 1000   # sizing only: no table is read
    assert L.echo_attn_workspace_bytes(ctypes.byref(cp), ctypes.byref(cb), 4) > n
    cb.max_blocks_per_row, cb.max_seq_len = mbr, msl
    cb.num_rows, cb.num_tokens = cb.num_rows * 2, cb.num_tokens * 2
    assert L.echo_attn_workspace_bytes(ctypes.byref(cp), ctypes.byref(cb), 4) > n


def _attn(L, cp, cb, hq, ws, ws_bytes, hws, hws_bytes):
    fake = ctypes.c_void_p(256)   # q / out: never dereferenced, a check fails first
    return L.echo_attn_mixed(ctypes.byref(cp), ctypes.byref(cb), fake, hq, 0.125, fake,
                             ws, ws_bytes, hws, hws_bytes, None)


def test_attention_workspace_errors_with_mirrors():
    w = W.config1()
    cp, cb, keep = _structs(w)
    L = echo.lib()
    n = L.echo_attn_workspace_bytes(ctypes.byref(cp), ctypes.byref(cb), 4)
    hn = L.echo_attn_host_workspace_bytes(ctypes.byref(cp), ctypes.byref(cb), 4)
    host = np.zeros(hn + 64, np.uint8)    # pageable memory: refused as host workspace
    hp = ctypes.c_void_p(host.ctypes.data + (-host.ctypes.data) % 16)
    dev = ctypes.c_void_p(1 << 20)        # a 256-byte aligned stand-in, never touched
    for args, what in [((None, n, hp, hn), "workspace of"),
                       ((dev, n - 4, hp, hn), "workspace of"),
                       ((ctypes.c_void_p((1 << 20) + 128), n, hp, hn), "256-byte aligned"),
                       ((dev, n, None, hn), "host workspace of"),
                       ((dev, n, hp, hn - 4), "host workspace of"),
                       ((dev, n, ctypes.c_void_p(hp.value + 4), hn), "16-byte aligned"),
                       ((dev, n, hp, hn), "not pinned")]:
        rc = _attn(L, cp, cb, 4, *args)
        assert rc == echo.ECHO_E_WORKSPACE and what in echo.last_error(), (what, echo.last_error())


def test_attention_workspace_errors_without_mirrors():
    w = W.config1()
    cp, cb, keep = _structs(w)
    cb.h_block_tables = cb.h_seq_lens = cb.h_q_start = cb.h_row_kind = None
    L = echo.lib()
    n = L.echo_attn_workspace_bytes(ctypes.byref(cp), ctypes.byref(cb), 4)
    for ws, nb, what in [(None, n, "workspace of"), (ctypes.c_void_p(1 << 20), n - 256, "workspace of"),
                         (ctypes.c_void_p((1 << 20) + 64), n, "256-byte aligned")]:
        rc = _attn(L, cp, cb, 4, ws, nb, None, 0)
        assert rc == echo.ECHO_E_WORKSPACE and what in echo.last_error(), echo.last_error()


@pytest.mark.parametrize("scale", [0.0, -0.125, float("nan"), float("inf")])
def test_attention_rejects_non_positive_scale(scale):
    # raw scores are reduced to a maximum before scaling, which needs scale > 0
    w = W.config1()
    cp, cb, keep = _structs(w)
    fake = ctypes.c_void_p(256)   # never dereferenced: validation fails first
    rc = echo.lib().echo_attn_mixed(ctypes.byref(cp), ctypes.byref(cb), fake, 4, scale, fake,
                                    None, 0, None, 0, None)
    assert rc == echo.ECHO_E_INVALID and "sm_scale" in echo.last_error()


def test_prefill_row_beyond_the_staging_limit():
    # a prefill workgroup stages its row's block ids in LDS: one block more
    # than fits (16,372 at head_dim 128) is refused before any work (GQA 8/4:
    # 264 workgroups, so the tile's key range is not cut into pieces)
    q = 8448
    w = W.build("pf-limit+1", [W.RowSpec(W.PREFILL, 16373 * 16 - q, q)], {}, 8, 4, 128, seed=31)
    cp, cb, keep = _structs(w)
    L = echo.lib()
    n = L.echo_attn_workspace_bytes(ctypes.byref(cp), ctypes.byref(cb), 8)
    assert n > 0
    fake = ctypes.c_void_p(256)   # never dereferenced: the check comes first
    rc = L.echo_attn_mixed(ctypes.byref(cp), ctypes.byref(cb), fake, 8, 0.088, fake, fake, n,
                           None, 0, None)
    assert rc == echo.ECHO_E_UNSUPPORTED
    assert "16373 blocks exceeds the 16372-block limit" in echo.last_error()


def test_block_copy_pair_rules():
    w = W.config1()
    cp, cb, keep = _structs(w)
    L = echo.lib()
    for pairs, code in [([[3, 3]], echo.ECHO_E_INVALID),
                        ([[1, 5], [2, 5]], echo.ECHO_E_INVALID),
                        ([[1, 5], [5, 6]], echo.ECHO_E_INVALID),
                        ([[1, 64]], echo.ECHO_E_RANGE),
                        ([[-1, 2]], echo.ECHO_E_RANGE)]:
        hp = np.ascontiguousarray(pairs, np.int32)
        rc = L.echo_block_copy(ctypes.byref(cp), 0x1000, len(pairs),
                               hp.ctypes.data_as(ctypes.c_void_p), None)
        assert rc == code, (pairs, echo.last_error())


def _unique_tokens(w):
    used = {}
    for r in range(w.batch.num_rows):
        L = int(w.batch.seq_lens[r])
        for j in range(0, L, 16):
            b = int(w.batch.block_tables[r, j // 16])
            used[b] = max(used.get(b, 0), min(16, L - j))
    return sum(used.values())


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_plan_statistics(cfg):
    w = W.config(cfg)
    cp, cb, keep = _structs(w)
    st = echo.plan_stats(cp, cb, w.num_q_heads)
    assert st["unique_kv_tokens"] == _unique_tokens(w)
    assert st["logical_kv_tokens"] == int(w.batch.seq_lens.sum())
    q = np.diff(w.batch.q_start)
    ctx = w.batch.seq_lens - q
    assert st["causal_pairs"] == int((q * ctx + q * (q + 1) // 2).sum())
    n_groups = len({r.group for r in w.rows if r.group >= 0 and r.kind == W.DECODE})
    assert st["shared_segments"] >= n_groups
    assert st["work_items"] == st["decode_items"] + st["prefill_items"]
    assert st["workspace_bytes"] >= st["partial_slots"] * (w.head_dim + 1) * 4


def test_plan_shares_prefix_blocks_in_config1():
    w = W.config1()
    cp, cb, keep = _structs(w)
    st = echo.plan_stats(cp, cb, w.num_q_heads)
    # the two decode rows share one 2-block segment
    assert st["shared_segments"] == 1
    dup = W.config1(duplicate_prefix=True)
    cp, cb, keep = _structs(dup)
    assert echo.plan_stats(cp, cb, dup.num_q_heads)["shared_segments"] == 0


def test_static_entry_refuses_batches_beyond_its_scratch():
    # the e4m3 mixed configuration's device-built plan needs about 100 MB of
    # partial results, more than the 32 MiB static scratch: refused before
    # any GPU work, with the sizes in the message
    w = W.config(5, values=False)
    cp, cb, keep = _structs(w)
    fake = ctypes.c_void_p(256)
    rc = echo.lib().echo_attn_mixed_static(ctypes.byref(cp), ctypes.byref(cb), fake,
                                           w.num_q_heads, w.sm_scale, fake, None)
    assert rc == echo.ECHO_E_WORKSPACE
    assert "static scratch holds 33554432" in echo.last_error()
