// plan.cpp -- host planner for echo_attn_mixed (see plan.hpp).
#include "plan.hpp"

#include <algorithm>
#include <cstring>

#include "echo.h"

namespace echo {
namespace {

struct Segment {
    int32_t rows_off;  // offset into seg_rows
    int32_t nrows;
    int32_t j0, j1;    // block index range in each member's table
    int32_t key_end;   // one past the last key
};

int64_t align_words(int64_t w, int64_t a) { return (w + a - 1) / a * a; }

// Prefix trie over the read-only full blocks of decode rows.  Rows in
// R[lo, hi) share blocks [0, d) of their tables.  Runs of rows that also share
// the block at depth d form a segment as long as all of them keep agreeing;
// a row that leaves every group reads the rest of its keys privately.
void build_trie(const HostBatch &b, const std::vector<int32_t> &nro, std::vector<int32_t> &R,
                std::vector<int32_t> &tail_start, std::vector<Segment> &segs,
                std::vector<int32_t> &seg_rows) {
    struct Frame { int32_t lo, hi, d; };
    std::vector<Frame> stack;
    if (!R.empty()) stack.push_back({0, (int32_t)R.size(), 0});
    auto blk = [&](int32_t r, int32_t j) { return b.bt[(size_t)r * b.mbr + j]; };
    while (!stack.empty()) {
        Frame f = stack.back();
        stack.pop_back();
        // rows with no read-only block at depth d end here
        int32_t *beg = R.data() + f.lo, *end = R.data() + f.hi;
        int32_t *mid = std::partition(beg, end, [&](int32_t r) { return nro[r] <= f.d; });
        for (int32_t *p = beg; p < mid; ++p) tail_start[*p] = f.d;
        std::sort(mid, end, [&](int32_t x, int32_t y) {
            int32_t bx = blk(x, f.d), by = blk(y, f.d);
            return bx != by ? bx < by : x < y;
        });
        for (int32_t *a = mid; a < end;) {
            int32_t *e = a + 1;
            while (e < end && blk(*e, f.d) == blk(*a, f.d)) ++e;
            if (e - a == 1) {
                tail_start[*a] = f.d;
            } else {
                int32_t dd = f.d + 1;
                for (;;) {
                    bool same = true;
                    for (int32_t *p = a; p < e && same; ++p)
                        same = nro[*p] > dd && blk(*p, dd) == blk(*a, dd);
                    if (!same) break;
                    ++dd;
                }
                Segment s;
                s.rows_off = (int32_t)seg_rows.size();
                s.nrows = (int32_t)(e - a);
                s.j0 = f.d;
                s.j1 = dd;
                s.key_end = kBlock * dd;
                seg_rows.insert(seg_rows.end(), a, e);
                segs.push_back(s);
                stack.push_back({(int32_t)(a - R.data()), (int32_t)(e - R.data()), dd});
            }
            a = e;
        }
    }
}

}  // namespace

int build_plan(const HostBatch &b, int32_t Hkv, int32_t Hq, int32_t D, const PlanOptions &opt,
               Plan &plan) {
    const int32_t B = b.num_rows, T = b.num_tokens;
    const int32_t G = Hq / Hkv;
    const int32_t hpc = G < kWaveQueries ? G : kWaveQueries;   // heads per chunk
    const int32_t nhc = (G + kWaveQueries - 1) / kWaveQueries; // head chunks
    const int32_t nt_max = kWaveQueries / hpc;                 // tokens per slice
    plan.head_chunks = nhc;
    plan.heads_per_chunk = hpc;
    plan.waves_per_desc = Hkv * nhc;

    plan.desc.clear();
    plan.tok_list.clear();
    plan.merge_tok.clear();
    plan.merge_ptr.clear();
    plan.merge_ent.clear();
    plan.klim.resize((size_t)T);
    plan.stats = PlanStats{};

    // keys visible to every new token: its position + 1
    for (int32_t r = 0; r < B; ++r) {
        const int32_t q = b.q_start[r + 1] - b.q_start[r];
        const int32_t c = b.seq_lens[r] - q;
        int32_t *kl = plan.klim.data() + b.q_start[r];
        for (int32_t i = 0; i < q; ++i) kl[i] = c + i + 1;
        plan.stats.logical_kv_tokens += b.seq_lens[r];
        plan.stats.causal_pairs += (int64_t)q * c + (int64_t)q * (q + 1) / 2;
        if (b.kind[r] == ECHO_ROW_PREFILL)
            plan.stats.prefill_causal_pairs += (int64_t)q * c + (int64_t)q * (q + 1) / 2;
    }

    // ---- decode rows: segments from the trie plus one private tail per row
    std::vector<int32_t> &nro = plan.nro, &R = plan.rows, &tail_start = plan.tail_start,
                         &seg_rows = plan.seg_rows;
    nro.assign((size_t)B, 0);
    tail_start.assign((size_t)B, 0);
    R.clear();
    seg_rows.clear();
    std::vector<Segment> segs;
    for (int32_t r = 0; r < B; ++r) {
        if (b.kind[r] != ECHO_ROW_DECODE) continue;
        nro[r] = (b.seq_lens[r] - 1) / kBlock;  // full blocks before the new token's block
        R.push_back(r);
    }
    build_trie(b, nro, R, tail_start, segs, seg_rows);
    plan.stats.shared_segments = (int64_t)segs.size();
    for (int32_t r : R) {
        Segment s;
        s.rows_off = (int32_t)seg_rows.size();
        s.nrows = 1;
        s.j0 = tail_start[r];
        s.j1 = (b.seq_lens[r] + kBlock - 1) / kBlock;
        s.key_end = b.seq_lens[r];
        seg_rows.push_back(r);
        segs.push_back(s);
    }

    // Key ranges are split into pieces of `split` blocks.  Long pieces keep
    // the partial results and the merge small; on a small decode batch they
    // would leave most of the GPU idle while a few waves walk long ranges one
    // latency-bound step after another, so the pieces shrink (to no fewer
    // than kMinSplitBlocks) until the batch has about kSplitTargetUnits
    // (piece, KV head, head chunk) units.
    int64_t seg_blocks = 0;
    for (const Segment &s : segs) seg_blocks += s.j1 - s.j0;
    const int32_t min_split = std::min<int32_t>(kMinSplitBlocks, std::max(2, opt.split_blocks));
    const int64_t units_cap = seg_blocks * Hkv * nhc / kSplitTargetUnits;
    int32_t split = (int32_t)std::max<int64_t>(min_split, std::min<int64_t>(opt.split_blocks, units_cap));
    auto waves_for = [&](int32_t sp) {
        int64_t n = 0;
        for (const Segment &s : segs)
            n += (int64_t)((s.j1 - s.j0 + sp - 1) / sp) * ((s.nrows + nt_max - 1) / nt_max);
        return n * plan.waves_per_desc;
    };
    // A launch that fits one generation of resident waves starts every wave
    // at once and has no partly filled last generation: when pieces up to
    // kOneGenerationStretch times longer (and no longer than the unit target
    // allows) bring the launch under that, take the shortest such length.
    const int64_t slots = (int64_t)kDecodeWavesPerCu * opt.num_cus;
    const int32_t stretch_cap = (int32_t)std::max<int64_t>(
        split, std::min<int64_t>((int64_t)kOneGenerationStretch * opt.split_blocks, units_cap));
    if (waves_for(split) > slots && waves_for(stretch_cap) <= slots) {
        int32_t lo = split + 1, hi = stretch_cap;
        while (lo < hi) {
            const int32_t mid = lo + (hi - lo) / 2;
            if (waves_for(mid) <= slots) hi = mid;
            else lo = mid + 1;
        }
        split = lo;
    }

    // contributions per decode row: sum over its segments of their splits
    std::vector<int32_t> &cnt = plan.cnt, &moff = plan.moff, &cursor = plan.cursor;
    cnt.assign((size_t)B, 0);
    auto n_splits = [&](const Segment &s) { return (s.j1 - s.j0 + split - 1) / split; };
    const int64_t n_waves = waves_for(split);
    const bool equal_pieces = n_waves <= (int64_t)kEqualPieceGenerations * slots;
    for (const Segment &s : segs)
        for (int32_t k = 0; k < s.nrows; ++k) cnt[seg_rows[s.rows_off + k]] += n_splits(s);

    // merge lists: rows with more than one contribution; entries
    // (first partial slot of the descriptor, nt | i << 10) for query i of a
    // slice of nt tokens
    moff.assign((size_t)B, -1);
    int64_t n_ent = 0;
    for (int32_t r : R) {
        if (cnt[r] < 2) continue;
        moff[r] = (int32_t)plan.merge_tok.size();
        plan.merge_tok.push_back(b.q_start[r]);
        plan.merge_ptr.push_back((int32_t)n_ent);
        n_ent += cnt[r];
    }
    plan.merge_ptr.push_back((int32_t)n_ent);
    plan.merge_ent.assign((size_t)(2 * n_ent), -1);
    cursor.assign(plan.merge_tok.size(), 0);

    int64_t n_slots = 0;
    const int64_t wpd = plan.waves_per_desc;
    plan.sibling_waves = 0;
    for (size_t si = 0; si < segs.size(); ++si) {
        const Segment &s = segs[si];
        const int32_t tok_base = (int32_t)plan.tok_list.size();
        for (int32_t k = 0; k < s.nrows; ++k)
            plan.tok_list.push_back(b.q_start[seg_rows[s.rows_off + k]]);
        const int32_t rep = seg_rows[s.rows_off];
        const bool direct = (s.nrows == 1 && cnt[rep] == 1);
        const bool shared = s.nrows > nt_max || nhc > 1;
        if (s.nrows > 1)   // slices x KV heads x head chunks read each piece
            plan.sibling_waves = (int32_t)std::max<int64_t>(
                plan.sibling_waves, (s.nrows + nt_max - 1) / nt_max * wpd);
        plan.stats.decode_kv_tokens += s.key_end - kBlock * s.j0;
        const int32_t ns = n_splits(s);
        const int32_t step = equal_pieces ? (s.j1 - s.j0 + ns - 1) / ns : split;
        for (int32_t j = s.j0; j < s.j1; j += step) {
            const int32_t jend = std::min(j + step, s.j1);
            for (int32_t k0 = 0; k0 < s.nrows; k0 += nt_max) {
                const int32_t ntk = std::min(nt_max, s.nrows - k0);
                WorkDesc d;
                d.tok_off = tok_base + k0;
                d.shape = ntk | (shared ? kItemShared : 0);
                d.bt_row = rep;
                d.key_begin = kBlock * j;
                d.key_end = std::min(kBlock * jend, s.key_end);
                d.part = -1;
                d.tok1 = ntk == 1 ? plan.tok_list[tok_base + k0] : -1;
                d.klim1 = ntk == 1 ? plan.klim[d.tok1] : 0;
                if (!direct) {
                    d.part = (int32_t)n_slots;
                    for (int32_t i = 0; i < ntk; ++i) {
                        const int32_t m = moff[seg_rows[s.rows_off + k0 + i]];
                        const int64_t e = plan.merge_ptr[m] + cursor[m]++;
                        plan.merge_ent[2 * e] = d.part;
                        plan.merge_ent[2 * e + 1] = ntk | (i << 10);
                    }
                    n_slots += wpd * ntk * hpc;
                }
                plan.desc.push_back(d);
                plan.stats.decode_items += wpd;
            }
        }
    }
    for (int32_t v : plan.merge_ent)
        if (v < 0) return ECHO_E_INVALID;  // every merged result must have all its parts

    // ---- prefill rows: tiles of consecutive tokens, all heads of a KV head
    plan.pdesc.clear();
    const int32_t bt_tok = std::max(1, kPrefillQueries / G);
    plan.prefill_tokens_per_tile = bt_tok;
    int64_t pf_work = 0, pf_tiles = 0;   // 64-key tiles summed over the prefill tiles
    for (int32_t r = 0; r < B; ++r) {
        if (b.kind[r] != ECHO_ROW_PREFILL) continue;
        const int32_t q = b.q_start[r + 1] - b.q_start[r];
        const int32_t c = b.seq_lens[r] - q;
        const int32_t ntiles = (q + bt_tok - 1) / bt_tok;
        for (int32_t k = ntiles - 1; k >= 0; --k) {  // longest key ranges first
            PrefillDesc d;
            d.row = r;
            d.tok0 = b.q_start[r] + k * bt_tok;
            d.ntok = std::min(bt_tok, q - k * bt_tok);
            d.key_end = c + k * bt_tok + d.ntok;
            d.key_begin = 0;
            d.part = -1;
            d.kfull = d.key_end - d.ntok + 1;
            d.next = 0;
            plan.pdesc.push_back(d);
            pf_work += (d.key_end + kPrefillTileKeys - 1) / kPrefillTileKeys;
            ++pf_tiles;
        }
    }
    // Workgroups for at most half the CUs leave the rest idle (a late chunk
    // of a long prompt is a handful of tiles over tens of thousands of keys):
    // cut key ranges longer than the average share of a CU into pieces at
    // tile boundaries that every token of the tile sees unmasked.  Pieces
    // write partial softmax states that the merge kernel combines.  (With
    // about one workgroup per CU, cutting every long range costs in the
    // merge what it gains; the branch below moves only the excess.)
    int32_t grid_pdesc = -1;   // descriptors that get workgroups (chained ones follow)
    if (pf_tiles > 0 && 2 * pf_tiles * Hkv <= (int64_t)opt.num_cus) {
        const int64_t share = (pf_work * Hkv + opt.num_cus - 1) / opt.num_cus;
        const int32_t piece = (int32_t)std::max<int64_t>(kPrefillMinPieceTiles, share);
        std::vector<PrefillDesc> &out = plan.pdesc_split;
        out.clear();
        if (!plan.merge_ptr.empty()) plan.merge_ptr.pop_back();   // reopen the list
        for (const PrefillDesc &d : plan.pdesc) {
            const int32_t nt = (d.key_end + kPrefillTileKeys - 1) / kPrefillTileKeys;
            const int32_t unmasked = d.kfull / kPrefillTileKeys;   // whole tiles every token sees
            int32_t cut = 0;
            std::vector<int32_t> &bounds = plan.bounds;
            bounds.assign(1, 0);
            while (nt - cut > piece && cut + piece <= unmasked) {
                cut += piece;
                bounds.push_back(cut);
            }
            if (bounds.size() == 1) {
                out.push_back(d);
                continue;
            }
            bounds.push_back(nt);
            const int32_t slots = Hkv * nhc * d.ntok * hpc;
            for (int32_t i = 0; i < d.ntok; ++i) {
                plan.merge_tok.push_back(d.tok0 + i);
                plan.merge_ptr.push_back((int32_t)(plan.merge_ent.size() / 2));
                for (size_t p = 0; p + 1 < bounds.size(); ++p) {
                    plan.merge_ent.push_back((int32_t)(n_slots + (int64_t)p * slots));
                    plan.merge_ent.push_back(d.ntok | (i << 10));
                }
            }
            for (size_t p = 0; p + 1 < bounds.size(); ++p) {
                PrefillDesc e = d;
                e.key_begin = bounds[p] * kPrefillTileKeys;
                e.key_end = p + 2 < bounds.size() ? bounds[p + 1] * kPrefillTileKeys : d.key_end;
                e.part = (int32_t)(n_slots + (int64_t)p * slots);
                out.push_back(e);
            }
            n_slots += (int64_t)(bounds.size() - 1) * slots;
        }
        plan.merge_ptr.push_back((int32_t)(plan.merge_ent.size() / 2));
        // longest pieces first
        std::stable_sort(out.begin(), out.end(), [](const PrefillDesc &x, const PrefillDesc &y) {
            return x.key_end - x.key_begin > y.key_end - y.key_begin;
        });
        plan.pdesc.swap(out);
    } else if (pf_tiles > 1 && pf_tiles * Hkv <= (int64_t)opt.num_cus) {
        // One round of workgroups takes as long as its longest tile, and the
        // causal tiles of a chunk span from its context to its full length.
        // Short tiles' workgroups take over the leading keys of long tiles
        // (keys every token of such a tile sees) as further descriptors
        // chained to their own, so that every workgroup walks about the mean
        // number of 64-key tiles.  All pieces of a long tile write partial
        // states that the merge kernel combines.
        const int32_t n = (int32_t)plan.pdesc.size();
        std::vector<int32_t> &wk = plan.bounds;   // 64-key tiles per workgroup
        std::vector<int32_t> &order = plan.bucket;
        wk.resize(n);
        order.resize(n);
        int64_t total = 0;
        for (int32_t i = 0; i < n; ++i) {
            wk[i] = (plan.pdesc[i].key_end + kPrefillTileKeys - 1) / kPrefillTileKeys;
            total += wk[i];
            order[i] = i;
        }
        const int32_t target = (int32_t)((total + n - 1) / n);
        std::stable_sort(order.begin(), order.end(),
                         [&](int32_t x, int32_t y) { return wk[x] > wk[y]; });
        std::vector<PrefillDesc> &chained = plan.pdesc_split;
        chained.clear();
        if (!plan.merge_ptr.empty()) plan.merge_ptr.pop_back();   // reopen the list
        int32_t lo = n - 1;   // shortest tile that may still take a piece
        std::vector<int32_t> &cuts = plan.cuts, &takers = plan.takers, &last = plan.ctail;
        last.resize(n);   // last descriptor of each workgroup's chain
        for (int32_t i = 0; i < n; ++i) last[i] = i;
        for (int32_t hi = 0; hi < lo; ++hi) {
            PrefillDesc &dj = plan.pdesc[order[hi]];
            int32_t excess = wk[order[hi]] - target;
            if (excess < kPrefillMinChainTiles) break;   // the rest have less
            // leading pieces [cuts[k], cuts[k+1]) go to short tiles' workgroups
            const int32_t unmasked = dj.kfull / kPrefillTileKeys;
            cuts.assign(1, 0);
            takers.clear();
            while (excess >= kPrefillMinChainTiles) {
                while (lo > hi && target - wk[order[lo]] < kPrefillMinChainTiles) --lo;
                if (lo <= hi) break;
                const int32_t i = order[lo];
                const int32_t x = std::min(std::min(excess, target - wk[i]), unmasked - cuts.back());
                if (x < kPrefillMinChainTiles) break;
                cuts.push_back(cuts.back() + x);
                takers.push_back(i);
                wk[i] += x;
                excess -= x;
            }
            if (takers.empty()) continue;
            const int32_t np = (int32_t)takers.size() + 1;   // pieces of this tile
            const int32_t slots = Hkv * nhc * dj.ntok * hpc;
            for (int32_t t = 0; t < dj.ntok; ++t) {
                plan.merge_tok.push_back(dj.tok0 + t);
                plan.merge_ptr.push_back((int32_t)(plan.merge_ent.size() / 2));
                for (int32_t p = 0; p < np; ++p) {
                    plan.merge_ent.push_back((int32_t)(n_slots + (int64_t)p * slots));
                    plan.merge_ent.push_back(dj.ntok | (t << 10));
                }
            }
            for (int32_t p = 0; p + 1 < np; ++p) {
                PrefillDesc head = dj;
                head.key_begin = cuts[p] * kPrefillTileKeys;
                head.key_end = cuts[p + 1] * kPrefillTileKeys;
                head.part = (int32_t)(n_slots + (int64_t)p * slots);
                const int32_t idx = n + (int32_t)chained.size();
                int32_t &tail = last[takers[p]];
                (tail < n ? plan.pdesc[tail] : chained[tail - n]).next = idx + 1;
                tail = idx;
                chained.push_back(head);
            }
            dj.key_begin = cuts.back() * kPrefillTileKeys;
            dj.part = (int32_t)(n_slots + (int64_t)(np - 1) * slots);
            wk[order[hi]] -= cuts.back();
            n_slots += (int64_t)np * slots;
        }
        plan.merge_ptr.push_back((int32_t)(plan.merge_ent.size() / 2));
        plan.pdesc.insert(plan.pdesc.end(), chained.begin(), chained.end());
        grid_pdesc = n;
    }
    plan.pdesc_grid = grid_pdesc >= 0 ? grid_pdesc : (int32_t)plan.pdesc.size();
    plan.stats.prefill_items = (int64_t)plan.pdesc.size() * Hkv;
    n_ent = (int64_t)plan.merge_ent.size() / 2;

    // heavy descriptors first (counting sort on 32-key steps, stable)
    {
        const int32_t nb = 1024;
        std::vector<int32_t> &count = plan.bucket;
        count.assign(nb + 1, 0);
        auto bucket = [&](const WorkDesc &d) {
            int32_t steps = (d.key_end - d.key_begin + 31) / 32;
            return nb - 1 - std::min(steps, nb - 1);
        };
        for (const WorkDesc &d : plan.desc) ++count[bucket(d) + 1];
        for (int32_t i = 0; i < nb; ++i) count[i + 1] += count[i];
        // (merge entries name partial slots, which do not move with the order)
        plan.desc_sorted.resize(plan.desc.size());
        for (size_t i = 0; i < plan.desc.size(); ++i)
            plan.desc_sorted[count[bucket(plan.desc[i])]++] = plan.desc[i];
        plan.desc.swap(plan.desc_sorted);
    }

    PlanLayout &L = plan.layout;
    L = PlanLayout{};
    L.head_dim = D;
    L.n_desc = (int64_t)plan.desc.size();
    L.n_tok_list = (int64_t)plan.tok_list.size();
    L.n_tokens = T;
    L.n_merge_rows = (int64_t)plan.merge_tok.size();
    L.n_merge_entries = n_ent;
    L.n_slots = n_slots;
    int64_t w = 0;
    L.n_pdesc = (int64_t)plan.pdesc.size();
    static_assert(sizeof(WorkDesc) % 4 == 0 && sizeof(PrefillDesc) % 4 == 0, "word-sized descriptors");
    L.off_desc = w;       w += L.n_desc * (int64_t)(sizeof(WorkDesc) / 4);
    L.off_pdesc = w;      w += L.n_pdesc * (int64_t)(sizeof(PrefillDesc) / 4);
    L.off_tok_list = w;   w += L.n_tok_list;
    L.off_klim = w;       w += L.n_tokens;
    L.off_merge_tok = w;  w += L.n_merge_rows;
    L.off_merge_ptr = w;  w += L.n_merge_rows + 1;
    L.off_merge_ent = w;  w += 2 * n_ent;
    L.upload_words = w;
    w = align_words(w, 64);
    L.off_part_lse = w;   w += n_slots;
    w = align_words(w, 64);
    L.off_part_o = w;     w += n_slots * D;
    L.total_words = align_words(w, 64);
    return ECHO_OK;
}

void pack_plan(const Plan &plan, void *dst) {
    const PlanLayout &L = plan.layout;
    int32_t *w = static_cast<int32_t *>(dst);
    if (L.n_desc) std::memcpy(w + L.off_desc, plan.desc.data(), L.n_desc * sizeof(WorkDesc));
    if (L.n_pdesc)
        std::memcpy(w + L.off_pdesc, plan.pdesc.data(), L.n_pdesc * sizeof(PrefillDesc));
    if (L.n_tok_list)
        std::memcpy(w + L.off_tok_list, plan.tok_list.data(), L.n_tok_list * 4);
    if (L.n_tokens) std::memcpy(w + L.off_klim, plan.klim.data(), L.n_tokens * 4);
    if (L.n_merge_rows)
        std::memcpy(w + L.off_merge_tok, plan.merge_tok.data(), L.n_merge_rows * 4);
    std::memcpy(w + L.off_merge_ptr, plan.merge_ptr.data(), (L.n_merge_rows + 1) * 4);
    if (L.n_merge_entries)
        std::memcpy(w + L.off_merge_ent, plan.merge_ent.data(), L.n_merge_entries * 8);
}

}  // namespace echo
