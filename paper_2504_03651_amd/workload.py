"""Seeded synthetic inputs for one mixed serving iteration over a paged KV cache.

This module only draws random numbers and lays them out; it computes nothing
that the iteration itself computes (no scatter, no quantisation, no attention).
Both the HIP path and the CPU oracle take their inputs from here.

What a workload holds (Echo, Section 2.1 "Prefill and decode", "Chunked
prefills"; Section 4.2 for fixed-size KV blocks; Section 6 for prefix reuse
through automatic prefix caching):

* ``batch``: the iteration's rows.  Decode rows add one token to a cached
  context; prefill rows add a chunk of prompt tokens to a (possibly empty)
  cached context.  ``seq_lens[r]`` counts the context plus this call's new
  tokens; ``q_start`` holds the prefix sums of new-token counts.
* ``ctx``: the context that earlier iterations already appended, expressed as
  an append batch with one pseudo-row per physical block (``fill`` tokens
  into a single-entry block table).  Each side builds its starting pool by
  running its own append over this batch on a pool poisoned with NaN.
* ``q``, ``k_new``, ``v_new``: bf16 bit patterns (uint16), token-major.
* ``cow_pairs``: (src, dst) block pairs copied before the append: one per
  prefix group, copying the group's last shared block into a block the batch
  never reads, as a copy-on-write fork would.

Rows that belong to a prefix group alias the group's leading blocks: a row
shares ``min(prefix_blocks, ctx // 16)`` full context blocks, never the block
it appends into.  Physical block ids come from a seeded permutation of the
pool.  Values are fp32 N(0, 1) draws rounded to nearest-even bf16.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
import os

import numpy as np

BLOCK = 16
DECODE = 0
PREFILL = 1
KV_BF16 = "bf16"
KV_FP8 = "fp8_e4m3"

BF16_NAN = 0x7FC0  # poison for unwritten bf16 slots
FP8_NAN = 0x7F     # poison for unwritten e4m3 slots

_CHUNK = 1 << 22


@dataclass
class Batch:
    block_tables: np.ndarray  # int32 [B][max_blocks_per_row], -1 past the valid entries
    seq_lens: np.ndarray      # int32 [B]
    q_start: np.ndarray       # int32 [B+1]
    row_kind: np.ndarray      # uint8 [B]

    @property
    def num_rows(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def num_tokens(self) -> int:
        return int(self.q_start[-1])

    @property
    def max_blocks_per_row(self) -> int:
        return int(self.block_tables.shape[1])

    @property
    def q_lens(self) -> np.ndarray:
        return np.diff(self.q_start).astype(np.int32)

    @property
    def max_q_len(self) -> int:
        return int(self.q_lens.max()) if self.num_rows else 0

    @property
    def max_seq_len(self) -> int:
        return int(self.seq_lens.max()) if self.num_rows else 0


@dataclass
class RowSpec:
    kind: int
    ctx: int          # tokens cached before this iteration
    q_len: int        # new tokens this iteration (1 for decode)
    group: int = -1   # prefix group, -1 for none


@dataclass
class Workload:
    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    num_blocks: int
    kv_dtype: str
    rows: list
    batch: Batch
    q: np.ndarray
    k_new: np.ndarray
    v_new: np.ndarray
    ctx: Batch
    ctx_k: np.ndarray
    ctx_v: np.ndarray
    cow_pairs: np.ndarray
    sm_scale: float
    seed: int
    # bookkeeping used by reports: physical ids that the batch reads
    used_blocks: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int32))
    free_blocks: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int32))

    @property
    def group_size(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def kv_bytes_per_elem(self) -> int:
        return 1 if self.kv_dtype == KV_FP8 else 2


# --------------------------------------------------------------------------
# random streams


def _normal_bf16(seed: int, stream: int, n: int, threads: int | None = None) -> np.ndarray:
    """n draws of fp32 N(0,1) rounded to nearest-even bf16 bit patterns.

    The draw is cut into fixed chunks, each with its own PCG64 stream keyed by
    (seed, stream, chunk), so the result does not depend on the thread count.
    """
    out = np.empty(n, dtype=np.uint16)
    nch = (n + _CHUNK - 1) // _CHUNK

    def work(i: int) -> None:
        lo = i * _CHUNK
        m = min(_CHUNK, n - lo)
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream, i])))
        x = g.standard_normal(m, dtype=np.float32)
        b = x.view(np.uint32)
        b += np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
        out[lo:lo + m] = (b >> np.uint32(16)).astype(np.uint16)

    if nch <= 1:
        for i in range(nch):
            work(i)
    else:
        threads = threads or min(16, os.cpu_count() or 1)
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(work, range(nch)))
    return out


# --------------------------------------------------------------------------
# layout of rows onto blocks


def build(name: str, rows: list, groups: dict, num_q_heads: int, num_kv_heads: int,
          head_dim: int, kv_dtype: str = KV_BF16, num_blocks: int | None = None,
          seed: int = 0, perm_seed: int | None = None, duplicate_prefix: bool = False,
          pool_factor: float = 1.25, values: bool = True) -> Workload:
    """Lay ``rows`` onto a paged pool and draw every value.

    ``groups`` maps a group id to its shared prefix length in tokens (a
    multiple of 16).  With ``duplicate_prefix`` every row gets private blocks
    holding the same values its group's shared blocks would hold, which is the
    physically duplicated twin of the aliased layout.  ``perm_seed`` reseeds
    only the placement of blocks in the pool.  With ``values=False`` only the
    layout is built (block tables, lengths, copy pairs): q, k_new, v_new,
    ctx_k and ctx_v are None.
    """
    assert num_q_heads % num_kv_heads == 0
    B = len(rows)
    # content blocks: (fill, owner tag); physical blocks map onto contents
    contents_fill = []          # tokens of context in each content block
    group_blocks = {}           # group -> list of content ids
    for gid, ptok in groups.items():
        assert ptok % BLOCK == 0
        used = 0
        for r in rows:
            if r.group == gid:
                used = max(used, min(ptok // BLOCK, r.ctx // BLOCK))
        ids = []
        for _ in range(used):
            ids.append(len(contents_fill))
            contents_fill.append(BLOCK)
        group_blocks[gid] = ids

    row_logical = []            # per row: list of (content id, is_shared)
    for r in rows:
        assert r.q_len >= 1 and r.ctx >= 0
        assert r.kind == PREFILL or r.q_len == 1
        L = r.ctx + r.q_len
        nblk = (L + BLOCK - 1) // BLOCK
        shared = 0
        if r.group >= 0:
            shared = min(len(group_blocks[r.group]), r.ctx // BLOCK)
        blocks = []
        for j in range(nblk):
            if j < shared:
                blocks.append((group_blocks[r.group][j], True))
            else:
                fill = max(0, min(BLOCK, r.ctx - BLOCK * j))
                blocks.append((len(contents_fill), False))
                contents_fill.append(fill)
        row_logical.append(blocks)

    # physical blocks: shared content gets one physical block, or one per row
    phys_content = []           # physical slot k -> content id
    shared_phys = {}
    row_phys_slots = []
    for blocks in row_logical:
        slots = []
        for cid, is_shared in blocks:
            if is_shared and not duplicate_prefix:
                if cid not in shared_phys:
                    shared_phys[cid] = len(phys_content)
                    phys_content.append(cid)
                slots.append(shared_phys[cid])
            else:
                slots.append(len(phys_content))
                phys_content.append(cid)
        row_phys_slots.append(slots)
    n_phys = len(phys_content)
    n_cow = len([g for g in groups if group_blocks[g]])
    if num_blocks is None:
        need = int(math.ceil(pool_factor * (n_phys + n_cow)))
        num_blocks = max(4096, ((need + 4095) // 4096) * 4096)
    assert num_blocks >= n_phys + n_cow, "pool too small"

    # draw order: lengths (given) -> pool permutation -> context K -> context V
    #             -> new K -> new V -> Q
    pg = np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [seed, 1 if perm_seed is None else 1000 + perm_seed])))
    perm = pg.permutation(num_blocks).astype(np.int32)
    phys_id = perm[:n_phys]

    MBR = max(len(s) for s in row_phys_slots) if B else 1
    bt = np.full((B, MBR), -1, dtype=np.int32)
    for i, slots in enumerate(row_phys_slots):
        bt[i, :len(slots)] = phys_id[np.asarray(slots, dtype=np.int64)]
    seq_lens = np.array([r.ctx + r.q_len for r in rows], dtype=np.int32)
    q_start = np.zeros(B + 1, dtype=np.int32)
    q_start[1:] = np.cumsum([r.q_len for r in rows])
    kind = np.array([r.kind for r in rows], dtype=np.uint8)
    batch = Batch(bt, seq_lens, q_start, kind)

    # context values per content block, then replicated onto physical blocks
    Hkv, D, Hq = num_kv_heads, head_dim, num_q_heads
    cfill = np.asarray(contents_fill, dtype=np.int64)
    coff = np.zeros(len(cfill) + 1, dtype=np.int64)
    coff[1:] = np.cumsum(cfill)
    ntok = int(coff[-1])
    if values:
        ck = _normal_bf16(seed, 2, ntok * Hkv * D).reshape(ntok, Hkv, D)
        cv = _normal_bf16(seed, 3, ntok * Hkv * D).reshape(ntok, Hkv, D)

    # one pseudo-row per physical block holding context, in content order
    holders = [[] for _ in range(len(cfill))]
    for k, c in enumerate(phys_content):
        holders[c].append(k)
    ctx_phys, ctx_cont = [], []
    for c in range(len(cfill)):
        if cfill[c] > 0:
            for k in holders[c]:
                ctx_phys.append(k)
                ctx_cont.append(c)
    nctx = len(ctx_phys)
    ctx_phys = np.asarray(ctx_phys, dtype=np.int64)
    ctx_cont = np.asarray(ctx_cont, dtype=np.int64)
    ctx_bt = phys_id[ctx_phys].reshape(nctx, 1).astype(np.int32)
    ctx_len = cfill[ctx_cont].astype(np.int32)
    ctx_qs = np.zeros(nctx + 1, dtype=np.int32)
    ctx_qs[1:] = np.cumsum(ctx_len)
    ctx = Batch(ctx_bt, ctx_len.copy(), ctx_qs, np.full(nctx, PREFILL, dtype=np.uint8))
    if not values:
        ctx_k = ctx_v = None
    elif nctx == int((cfill > 0).sum()):
        ctx_k, ctx_v = ck, cv
    else:
        idx = np.concatenate([np.arange(coff[c], coff[c] + cfill[c]) for c in ctx_cont])
        ctx_k, ctx_v = ck[idx], cv[idx]

    T = int(q_start[-1])
    k_new = v_new = q = None
    if values:
        k_new = _normal_bf16(seed, 4, T * Hkv * D).reshape(T, Hkv, D)
        v_new = _normal_bf16(seed, 5, T * Hkv * D).reshape(T, Hkv, D)
        q = _normal_bf16(seed, 6, T * Hq * D).reshape(T, Hq, D)

    # one copy-on-write fork per prefix group into a block nobody reads
    free = perm[n_phys:]
    cow = []
    for k, gid in enumerate(sorted(g for g in groups if group_blocks[g])):
        last = group_blocks[gid][-1]
        if duplicate_prefix:
            continue
        cow.append((int(phys_id[shared_phys[last]]), int(free[k])))
    cow_pairs = np.asarray(cow, dtype=np.int32).reshape(-1, 2)

    sm_scale = float(np.float32(1.0 / math.sqrt(D)))
    return Workload(name=name, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D,
                    num_blocks=int(num_blocks), kv_dtype=kv_dtype, rows=list(rows),
                    batch=batch, q=q, k_new=k_new, v_new=v_new, ctx=ctx,
                    ctx_k=ctx_k, ctx_v=ctx_v, cow_pairs=cow_pairs, sm_scale=sm_scale,
                    seed=seed, used_blocks=np.sort(phys_id), free_blocks=free[len(cow):])


# --------------------------------------------------------------------------
# the five serving-shaped configurations


def config(index: int, seed: int | None = None, **kw) -> Workload:
    """Configurations 1..5 (see the docstring of each builder), and 6, an
    extra shape: a late prefill chunk of a long prompt."""
    fn = {1: config1, 2: config2, 3: config3, 4: config4, 5: config5, 6: late_chunk}[index]
    return fn(seed=index if seed is None else seed, **kw)


def config1(seed: int = 1, share_with_prefill: bool = False, **kw) -> Workload:
    """Tiny mixed batch: MHA 4 heads, head_dim 64, pool of 64 blocks.

    Decode rows with contexts 100 and 37, prefill chunks of 32 new tokens on
    contexts 0 and 48.  The two decode rows alias a 2-block (32-token) prefix;
    with ``share_with_prefill`` the context-100 decode row shares it with the
    context-48 prefill row instead.
    """
    g_dec2 = -1 if share_with_prefill else 0
    g_pre2 = 0 if share_with_prefill else -1
    rows = [RowSpec(DECODE, 100, 1, 0),
            RowSpec(PREFILL, 0, 32, -1),
            RowSpec(DECODE, 37, 1, g_dec2),
            RowSpec(PREFILL, 48, 32, g_pre2)]
    return build("cfg1-tiny-mixed", rows, {0: 32}, 4, 4, 64, num_blocks=64, seed=seed, **kw)


def config2(seed: int = 2, **kw) -> Workload:
    """Decode-only offline batch: 256 rows, MHA 32x128, contexts U[512, 2048],
    groups of 16 rows alias a 1024-token prefix, pool of 40,000 blocks."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0])))
    ctx = g.integers(512, 2048, size=256, endpoint=True)
    rows = [RowSpec(DECODE, int(c), 1, i // 16) for i, c in enumerate(ctx)]
    groups = {k: 1024 for k in range(16)}
    return build("cfg2-decode-offline", rows, groups, 32, 32, 128, num_blocks=40000,
                 seed=seed, **kw)


def _mixed_rows(g, n_online, n_prefill, n_offline, group_size):
    online = np.clip(np.rint(1500.0 * np.exp(1.0 * g.standard_normal(n_online))), 1, 8192)
    offline = g.integers(256, 4096, size=n_offline, endpoint=True)
    rows = [RowSpec(DECODE, int(c), 1) for c in online]
    rows += [RowSpec(PREFILL, 1024, 2048) for _ in range(n_prefill)]
    rows += [RowSpec(DECODE, int(c), 1, i // group_size) for i, c in enumerate(offline)]
    groups = {k: 512 for k in range(n_offline // group_size)}
    return rows, groups


def config3(seed: int = 3, **kw) -> Workload:
    """Mixed online/offline iteration, GQA 32/8, head_dim 128: 8 online decode
    rows (context lognormal, median 1500, sigma 1, capped at 8192), one
    2048-token prefill chunk on a 1024-token context, 128 offline decode rows
    (context U[256, 4096]) sharing 512-token prefixes in groups of 32."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0])))
    rows, groups = _mixed_rows(g, 8, 1, 128, 32)
    return build("cfg3-mixed-gqa", rows, groups, 32, 8, 128, seed=seed, **kw)


def config4(seed: int = 4, **kw) -> Workload:
    """Long-context prefix-shared batch: 32 rows at 32,768-token contexts, GQA
    64/8, head_dim 128.  Groups of 8 rows share a 16,384-token prefix; the last
    row of each group is a 4,096-token prefill chunk, the rest decode."""
    rows = []
    for i in range(32):
        if i % 8 == 7:
            rows.append(RowSpec(PREFILL, 32768, 4096, i // 8))
        else:
            rows.append(RowSpec(DECODE, 32768, 1, i // 8))
    groups = {k: 16384 for k in range(4)}
    return build("cfg4-long-context", rows, groups, 64, 8, 128, seed=seed, **kw)


def config5(seed: int = 5, kv_dtype: str = KV_FP8, **kw) -> Workload:
    """Configuration 3 at four times the batch (32 online decode rows, two
    2048-token prefill chunks, 512 offline decode rows in 16 groups of 32) with
    the KV cache stored as fp8-e4m3 and one fp32 scale per block per KV head
    for K and for V.  ``kv_dtype=KV_BF16`` gives the same values in a bf16
    cache (the unquantised twin)."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0])))
    rows, groups = _mixed_rows(g, 32, 2, 512, 32)
    return build("cfg5-mixed-fp8", rows, groups, 32, 8, 128, kv_dtype=kv_dtype, seed=seed, **kw)


def late_chunk(seed: int = 6, **kw) -> Workload:
    """A late chunk of a long online prompt (64 new tokens on 30,000 cached
    ones) batched with 8 decode rows at 2,000-token contexts; GQA 64/8, head_dim
    128.  Chunked prefill (Section 2.1) reaches such chunks for every long
    prompt; its few query tiles span many keys."""
    rows = [RowSpec(PREFILL, 30000, 64)] + [RowSpec(DECODE, 2000, 1) for _ in range(8)]
    return build("late-chunk", rows, {}, 64, 8, 128, seed=seed, **kw)


def random_case(seed: int, num_rows: int = 6, num_q_heads: int = 8, num_kv_heads: int = 2,
                head_dim: int = 128, kv_dtype: str = KV_BF16, max_ctx: int = 600,
                max_q: int = 80, n_groups: int = 2, prefill_frac: float = 0.4,
                **kw) -> Workload:
    """A small random mix of decode and prefill rows, with random prefix
    groups, contexts that hit 16k, 16k+1 and 16k+15, and shuffled row kinds."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7])))
    rows = []
    for i in range(num_rows):
        c = int(g.integers(0, max_ctx, endpoint=True))
        pick = g.integers(0, 4)
        if pick == 1:
            c = 16 * (c // 16)
        elif pick == 2:
            c = 16 * (c // 16) + 1
        elif pick == 3:
            c = 16 * (c // 16) + 15
        c = min(c, max_ctx)
        if g.random() < prefill_frac:
            rows.append(RowSpec(PREFILL, c, int(g.integers(1, max_q, endpoint=True)),
                                int(g.integers(-1, n_groups)) if n_groups else -1))
        else:
            rows.append(RowSpec(DECODE, c, 1,
                                int(g.integers(-1, n_groups)) if n_groups else -1))
    groups = {k: 16 * int(g.integers(1, max(2, max_ctx // 16))) for k in range(n_groups)}
    return build(f"random-{seed}", rows, groups, num_q_heads, num_kv_heads, head_dim,
                 kv_dtype=kv_dtype, seed=seed, **kw)


# --------------------------------------------------------------------------
# decoder-layer inputs (random weights of a LLaMA-style layer)


def _scaled_bf16(seed: int, stream: int, n: int, scale: float, shift: float = 0.0) -> np.ndarray:
    """n draws of fp32 shift + scale * N(0,1), rounded to nearest-even bf16."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream])))
    x = (np.float32(shift) + np.float32(scale) * g.standard_normal(n, dtype=np.float32))
    b = x.astype(np.float32).view(np.uint32)
    b = b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return (b >> np.uint32(16)).astype(np.uint16)


@dataclass
class LayerWeights:
    hidden: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    intermediate: int
    rope_theta: float
    rms_eps: float
    attn_norm: np.ndarray   # [H] bf16 bits
    w_qkv: np.ndarray       # [(Hq + 2 Hkv) D][H]
    w_o: np.ndarray         # [H][Hq D]
    mlp_norm: np.ndarray    # [H]
    w_gate_up: np.ndarray   # [2 I][H] (gate rows, then up rows)
    w_down: np.ndarray      # [H][I]


def layer_weights(seed: int, hidden: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
                  intermediate: int, rope_theta: float = 500000.0,
                  rms_eps: float = 1e-5) -> LayerWeights:
    """Random weights: linear layers N(0, 1/fan_in), norms 1 + N(0, 0.1^2)."""
    H, I = hidden, intermediate
    qkv = (num_q_heads + 2 * num_kv_heads) * head_dim
    qd = num_q_heads * head_dim
    return LayerWeights(
        hidden, num_q_heads, num_kv_heads, head_dim, intermediate, rope_theta, rms_eps,
        _scaled_bf16(seed, 40, H, 0.1, 1.0),
        _scaled_bf16(seed, 41, qkv * H, 1.0 / math.sqrt(H)).reshape(qkv, H),
        _scaled_bf16(seed, 42, H * qd, 1.0 / math.sqrt(qd)).reshape(H, qd),
        _scaled_bf16(seed, 43, H, 0.1, 1.0),
        _scaled_bf16(seed, 44, 2 * I * H, 1.0 / math.sqrt(H)).reshape(2 * I, H),
        _scaled_bf16(seed, 45, H * I, 1.0 / math.sqrt(I)).reshape(H, I))


def layer_hidden(seed: int, num_tokens: int, hidden: int) -> np.ndarray:
    """The layer's input activations [T][H]: N(0,1) bf16 bits."""
    return _scaled_bf16(seed, 46, num_tokens * hidden, 1.0).reshape(num_tokens, hidden)
