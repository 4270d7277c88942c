"""Host-side invariants of the work plan that echo_attn_mixed uploads (CPU).

The plan is packed by the library's own code (echo_attn_plan_pack) and
decoded here word by word, so that a layout or planning mistake shows up on
the CPU instead of as a wrong address on the GPU:
  * the regions fit inside the workspace without overlapping;
  * every descriptor names valid rows, tokens, key ranges and partial slots;
  * for every new token, the key ranges of the work items that cover it tile
    [0, keys visible to it) exactly once, and a token with several items has
    one merge row whose entries are exactly those items;
  * partial-slot ranges of different items never overlap;
  * a prefill descriptor chained to another one (run next by the same
    workgroup) is named once and comes after every descriptor with a
    workgroup of its own; chains end.
"""
import numpy as np
import pytest

from paper_2504_03651_amd import echo
from paper_2504_03651_amd import workload as W

TILE = 64   # keys per prefill LDS tile


def _one_round_case(kv=W.KV_BF16):
    # 24 prefill tiles x 8 KV heads: one round of workgroups on 256 CUs, with
    # tiles of 1 to 40 64-key tiles
    rows = [W.RowSpec(W.PREFILL, 0, 1024), W.RowSpec(W.DECODE, 900, 1),
            W.RowSpec(W.PREFILL, 2000, 512), W.RowSpec(W.DECODE, 40, 1)]
    return W.build(f"one-round-{kv}", rows, {}, 32, 8, 128, kv_dtype=kv, seed=131)


def _cases():
    """(id, builder) pairs; workloads are built inside the test (layouts only
    for the full-size configurations, whose values the plan never reads)."""
    yield "cfg1", lambda: W.config1()
    yield "cfg1-share-prefill", lambda: W.config1(share_with_prefill=True)
    for seed in (201, 202, 203):
        yield f"random-{seed}", lambda seed=seed: W.random_case(
            seed, num_rows=9, num_q_heads=8, num_kv_heads=2, head_dim=128, max_ctx=2500,
            max_q=120, n_groups=3)
    yield "random-204", lambda: W.random_case(204, num_rows=7, num_q_heads=32, num_kv_heads=1,
                                              head_dim=64, max_ctx=3000, max_q=60, n_groups=2)
    for hq, hkv in ((32, 1), (8, 2), (4, 4)):
        rows = [W.RowSpec(W.PREFILL, 3000, 40), W.RowSpec(W.DECODE, 700, 1),
                W.RowSpec(W.PREFILL, 1500, 300), W.RowSpec(W.PREFILL, 64, 17)]
        yield f"split-{hq}-{hkv}", lambda hq=hq, hkv=hkv, rows=rows: W.build(
            f"split-{hq}-{hkv}", rows, {}, hq, hkv, 128, seed=118)
    # query heads per KV head that are not powers of two (3, 6, 12, 24)
    for g, hkv, d in ((3, 2, 128), (6, 2, 64), (12, 1, 128), (24, 2, 128)):
        yield f"gqa{g}", lambda g=g, hkv=hkv, d=d: W.random_case(
            210 + g, num_rows=9, num_q_heads=g * hkv, num_kv_heads=hkv, head_dim=d,
            max_ctx=2000, max_q=150, n_groups=2)
    for cfg in (2, 3, 4, 5):
        yield f"cfg{cfg}", lambda cfg=cfg: W.config(cfg, values=False)
    yield "one-round", lambda: _one_round_case()
    yield "random-205", lambda: W.random_case(205, num_rows=600, num_q_heads=4, num_kv_heads=2,
                                              head_dim=64, max_ctx=100, max_q=30, n_groups=3)


CASES = list(_cases())


def _decode(w):
    cp, cb, _keep = echo.host_structs(w)
    lay, words = echo.plan_pack(cp, cb, w.num_q_heads)
    return lay, words


@pytest.mark.parametrize("make", [m for _, m in CASES], ids=[n for n, _ in CASES])
def test_plan_invariants(make):
    w = make()
    lay, words = _decode(w)
    b = w.batch
    B, T = b.num_rows, b.num_tokens
    Hq, Hkv = w.num_q_heads, w.num_kv_heads
    G = Hq // Hkv
    hpc, nhc = lay["heads_per_chunk"], lay["head_chunks"]
    assert hpc == min(G, 16) and nhc == (G + 15) // 16

    # ---- regions in order, inside the workspace
    ends = [
        ("desc", lay["off_desc"], 8 * lay["n_desc"]),
        ("pdesc", lay["off_pdesc"], 8 * lay["n_pdesc"]),
        ("tok_list", lay["off_tok_list"], lay["n_tok_list"]),
        ("klim", lay["off_klim"], lay["n_tokens"]),
        ("merge_tok", lay["off_merge_tok"], lay["n_merge_rows"]),
        ("merge_ptr", lay["off_merge_ptr"], lay["n_merge_rows"] + 1),
        ("merge_ent", lay["off_merge_ent"], 2 * lay["n_merge_entries"]),
    ]
    pos = 0
    for name, off, n in ends:
        assert off >= pos, f"{name} overlaps the region before it"
        pos = off + n
    assert pos <= lay["upload_words"] <= lay["off_part_lse"]
    assert lay["off_part_lse"] + lay["n_slots"] <= lay["off_part_o"]
    assert lay["off_part_o"] + lay["n_slots"] * w.head_dim <= lay["total_words"]
    assert lay["n_tokens"] == T

    def region(off, n, width=1):
        return words[off:off + n * width].reshape(n, width) if width > 1 else words[off:off + n]

    desc = region(lay["off_desc"], lay["n_desc"], 8)
    pdesc = region(lay["off_pdesc"], lay["n_pdesc"], 8)
    tok_list = region(lay["off_tok_list"], lay["n_tok_list"])
    klim = region(lay["off_klim"], T)
    mtok = region(lay["off_merge_tok"], lay["n_merge_rows"])
    mptr = region(lay["off_merge_ptr"], lay["n_merge_rows"] + 1)
    ment = region(lay["off_merge_ent"], lay["n_merge_entries"], 2)

    # ---- chained prefill descriptors
    nxt = pdesc[:, 7].astype(np.int64) if len(pdesc) else np.zeros(0, np.int64)
    targets = (nxt[nxt > 0] - 1).tolist()
    assert len(set(targets)) == len(targets), "a descriptor is chained twice"
    n_grid = len(pdesc) - len(targets)
    assert all(n_grid <= t < len(pdesc) for t in targets)
    seen = 0
    for i in range(n_grid):   # each chain ends (targets are named once: no cycle)
        j = i
        while nxt[j] > 0:
            j = int(nxt[j]) - 1
            seen += 1
            assert pdesc[j][5] >= 0, "a chained piece writes partial states"
    assert seen == len(targets), "a chained descriptor is not reachable"

    # ---- per-token keys and rows
    q = np.diff(b.q_start)
    row_of = np.repeat(np.arange(B), q)
    pos_of = np.concatenate([b.seq_lens[r] - q[r] + np.arange(q[r]) for r in range(B)]) \
        if B else np.zeros(0, np.int64)
    assert np.array_equal(klim, pos_of + 1)

    ranges = [[] for _ in range(T)]        # (begin, end, part, slice size, index)
    slot_ranges = []
    for d in desc:
        tok_off, shape, bt_row, kb, ke, part, tok1, klim1 = (int(x) for x in d[:8])
        nt = shape & 0xFF
        if nt == 1:
            assert tok1 == tok_list[tok_off] and klim1 == klim[tok1]
        else:
            assert tok1 == -1
        assert 1 <= nt <= 16 // hpc
        assert 0 <= tok_off and tok_off + nt <= len(tok_list)
        assert 0 <= bt_row < B and b.row_kind[bt_row] == W.DECODE
        assert kb % 16 == 0 and 0 <= kb < ke <= b.seq_lens[bt_row]
        for i in range(nt):
            t = int(tok_list[tok_off + i])
            r = row_of[t]
            assert b.row_kind[r] == W.DECODE
            # the slice reads bt_row's blocks for these keys: they must be this row's too
            j0, j1 = kb // 16, (ke + 15) // 16
            assert ke <= b.seq_lens[r]
            assert np.array_equal(b.block_tables[r, j0:j1], b.block_tables[bt_row, j0:j1])
            ranges[t].append((kb, ke, part, nt, i))
        if part >= 0:
            slot_ranges.append((part, part + Hkv * nhc * nt * hpc))
    for d in pdesc:
        row, tok0, ntok, ke, kb, part, kfull = (int(x) for x in d[:7])
        assert b.row_kind[row] == W.PREFILL
        assert b.q_start[row] <= tok0 and tok0 + ntok <= b.q_start[row + 1]
        assert 1 <= ntok <= max(1, 256 // G)
        assert kb % TILE == 0 and 0 <= kb < ke <= b.seq_lens[row]
        assert kfull == klim[tok0]
        # every piece but a tile's last lies in keys all of its tokens see
        last = ke == klim[tok0 + ntok - 1]
        assert last or ke <= kfull
        for i in range(ntok):
            ranges[tok0 + i].append((kb, min(ke, int(klim[tok0 + i])), part, ntok, i))
        if part >= 0:
            slot_ranges.append((part, part + Hkv * nhc * ntok * hpc))

    # ---- coverage: exactly [0, klim) once per token
    for t in range(T):
        iv = sorted((kb, ke) for kb, ke, *_ in ranges[t])
        assert iv, f"token {t} has no work"
        cur = 0
        for kb, ke in iv:
            assert kb == cur, f"token {t}: keys {cur}..{kb} uncovered or overlapping"
            cur = ke
        assert cur == klim[t], f"token {t}: keys up to {cur}, visible {klim[t]}"

    # ---- merge rows: tokens with several items, entries exactly those items
    merged = {int(t): k for k, t in enumerate(mtok)}
    assert len(merged) == len(mtok), "a token has two merge rows"
    for t in range(T):
        items = ranges[t]
        if len(items) == 1:
            assert t not in merged and items[0][2] == -1
            continue
        assert t in merged, f"token {t} has {len(items)} items but no merge row"
        k = merged[t]
        ent = ment[mptr[k]:mptr[k + 1]]
        want = sorted((part, nt | (i << 10)) for _kb, _ke, part, nt, i in items)
        assert all(p >= 0 for p, _ in want)
        assert sorted(map(tuple, ent.tolist())) == want

    # ---- partial slots: disjoint ranges inside n_slots
    slot_ranges.sort()
    for (a0, a1), (b0, _b1) in zip(slot_ranges, slot_ranges[1:]):
        assert a1 <= b0, "two work items share partial slots"
    if slot_ranges:
        assert slot_ranges[0][0] >= 0 and slot_ranges[-1][1] <= lay["n_slots"]


def test_split_pieces_present():
    # the split shapes above must actually exercise pieces of key ranges
    w = W.build("split-check", [W.RowSpec(W.PREFILL, 3000, 40), W.RowSpec(W.DECODE, 700, 1)],
                {}, 8, 2, 128, seed=118)
    lay, words = _decode(w)
    pd = words[lay["off_pdesc"]:lay["off_pdesc"] + 8 * lay["n_pdesc"]].reshape(-1, 8)
    assert (pd[:, 5] >= 0).any() and (pd[:, 4] > 0).any()


def _prefill_work(w):
    """64-key tiles walked per prefill workgroup (own descriptor plus the
    chained one), and per tile before any balancing."""
    lay, words = _decode(w)
    pd = words[lay["off_pdesc"]:lay["off_pdesc"] + 8 * lay["n_pdesc"]].reshape(-1, 8)
    tiles = lambda d: (int(d[3]) - int(d[4]) + TILE - 1) // TILE
    n_grid = len(pd) - int((pd[:, 7] > 0).sum())
    work = []
    for i in range(n_grid):
        j, t = i, tiles(pd[i])
        while pd[j, 7] > 0:
            j = int(pd[j, 7]) - 1
            t += tiles(pd[j])
        work.append(t)
    orig = [(int(pd[i, 3]) + TILE - 1) // TILE for i in range(n_grid)]
    return work, orig, int((pd[:, 7] > 0).sum())


def test_one_round_prefill_balanced():
    # the mixed batch's 2,048-token chunk on 1,024 cached tokens: 32 tiles of
    # 17..48 64-key tiles per KV head, 256 workgroups; the longest workgroup
    # walks 34 (mean 32.5; a tile only 1 over the target of 33 keeps its keys)
    work, orig, chains = _prefill_work(W.config(3, values=False))
    assert max(orig) == 48 and chains == 14
    assert max(work) == 34 and sum(work) == sum(orig)
    # two chunks of unequal lengths (tiles of 1..16 and 33..40, mean 17.8): a
    # long tile gives pieces to several short ones and a short one takes
    # pieces of several long ones
    work, orig, chains = _prefill_work(_one_round_case())
    assert max(orig) == 40 and max(work) == 19 and sum(work) == sum(orig)
    # more than one round of workgroups: no chains
    assert _prefill_work(W.config(5, values=False))[2] == 0


def test_plan_pack_buffer_too_small():
    w = W.config1()
    cp, cb, _keep = echo.host_structs(w)
    import ctypes
    lay = echo.CPlanLayout()
    L = echo.lib()
    assert L.echo_attn_plan_pack(ctypes.byref(cp), ctypes.byref(cb), w.num_q_heads,
                                 ctypes.byref(lay), None, 0) == echo.ECHO_OK
    buf = np.zeros(4, np.int32)
    rc = L.echo_attn_plan_pack(ctypes.byref(cp), ctypes.byref(cb), w.num_q_heads,
                               ctypes.byref(lay), buf.ctypes.data, buf.nbytes)
    assert rc == echo.ECHO_E_WORKSPACE


def test_small_decode_batches_split_finer():
    # a late prefill chunk next to a few long decode rows: 48-block pieces
    # would give 24 descriptors; the planner shrinks them (not below 8 blocks)
    w = W.config(6, values=False)
    lay, words = _decode(w)
    d = words[lay["off_desc"]:lay["off_desc"] + 8 * lay["n_desc"]].reshape(-1, 8)
    blocks = (d[:, 4] - d[:, 3] + 15) // 16
    assert len(d) > 24 and blocks.max() <= 8
    # a large batch keeps the long pieces
    w2 = W.config(2, values=False)
    lay2, words2 = _decode(w2)
    d2 = words2[lay2["off_desc"]:lay2["off_desc"] + 8 * lay2["n_desc"]].reshape(-1, 8)
    assert ((d2[:, 4] - d2[:, 3] + 15) // 16).max() == 48
    # e4m3 pieces hold as many bytes: twice the blocks
    w5 = W.config(5, values=False)
    lay5, words5 = _decode(w5)
    d5 = words5[lay5["off_desc"]:lay5["off_desc"] + 8 * lay5["n_desc"]].reshape(-1, 8)
    assert ((d5[:, 4] - d5[:, 3] + 15) // 16).max() == 96


def _decode_pieces(w):
    lay, words = _decode(w)
    d = words[lay["off_desc"]:lay["off_desc"] + 8 * lay["n_desc"]].reshape(-1, 8)
    return lay, d


def test_equal_pieces_on_few_generation_launches():
    # the mixed batch's decode waves fill 1.2 generations of the resident
    # slots (12 waves x 256 CUs): a key range of n blocks cut into k pieces
    # gets pieces of ceil(n / k) blocks (the last one shorter by less than k);
    # the decode-only batch's 4.1 generations keep full 48-block pieces plus a
    # remainder
    for cfg, equal in ((3, True), (2, False)):
        w = W.config(cfg, values=False)
        lay, d = _decode_pieces(w)
        waves = len(d) * w.num_kv_heads * lay["head_chunks"]
        assert (waves <= 3 * 12 * 256) == equal
        # pieces of one key range: same bt_row and slice, consecutive ranges
        ranges = {}
        for tok_off, shape, bt_row, kb, ke, *_ in d.tolist():
            ranges.setdefault((bt_row, tok_off), []).append((kb, ke))
        split_ranges = 0
        for pieces in ranges.values():
            pieces.sort()
            if len(pieces) < 2:
                continue
            split_ranges += 1
            nblk = [(ke - kb + 15) // 16 for kb, ke in pieces]
            if equal:
                assert len(set(nblk[:-1])) == 1 and 0 <= nblk[0] - nblk[-1] < len(nblk), nblk
                assert nblk[0] == -(-sum(nblk) // len(nblk)), nblk
            else:
                assert all(n == 48 for n in nblk[:-1]), nblk
        assert split_ranges > 10


def test_pieces_stretch_to_fit_one_generation():
    # the long-context batch's decode (28 rows of 32k keys, GQA 64/8) needs
    # 2.5 generations of resident waves (12 per CU x 256 CUs) at the default
    # 48-block pieces; pieces of up to 4x that length fit it into one, and the
    # planner takes the shortest that does (equal lengths, 118-128 blocks).
    # The mixed batch cannot get under one generation (its ranges are short)
    # and keeps the default
    for cfg, longest in ((4, 128), (3, 48), (2, 48)):
        w = W.config(cfg, values=False)
        lay, d = _decode_pieces(w)
        waves = len(d) * w.num_kv_heads * lay["head_chunks"]
        nblk = (d[:, 4] - d[:, 3] + 15) // 16
        assert nblk.max() == longest
        if cfg == 4:   # one generation, and not stretched further than needed
            assert 0.9 * 12 * 256 < waves <= 12 * 256
