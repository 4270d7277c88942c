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
    const int32_t nh_full = G < kWaveQueries ? G : kWaveQueries;
    const int32_t n_head_chunks = (G + kWaveQueries - 1) / kWaveQueries;
    const int32_t split = opt.split_blocks > 0 ? opt.split_blocks : 32;

    plan.items.clear();
    plan.tok_list.clear();
    plan.merge_q.clear();
    plan.merge_ptr.clear();
    plan.merge_slot.clear();
    plan.klim.assign((size_t)T, 0);
    plan.stats = PlanStats{};

    // keys visible to every new token: its position + 1
    for (int32_t r = 0; r < B; ++r) {
        const int32_t q = b.q_start[r + 1] - b.q_start[r];
        const int32_t c = b.seq_lens[r] - q;
        for (int32_t i = 0; i < q; ++i) plan.klim[(size_t)b.q_start[r] + i] = c + i + 1;
        plan.stats.logical_kv_tokens += b.seq_lens[r];
        plan.stats.causal_pairs += (int64_t)q * c + (int64_t)q * (q + 1) / 2;
    }

    // ---- decode rows: segments from the trie plus one private tail per row
    std::vector<int32_t> nro((size_t)B, 0), R, tail_start((size_t)B, 0), seg_rows;
    std::vector<Segment> segs;
    for (int32_t r = 0; r < B; ++r) {
        if (b.kind[r] != ECHO_ROW_DECODE) continue;
        nro[r] = (b.seq_lens[r] - 1) / kBlock;  // full blocks before the new token's block
        R.push_back(r);
    }
    build_trie(b, nro, R, tail_start, segs, seg_rows);
    plan.stats.shared_segments = (int64_t)segs.size();
    const size_t n_shared = segs.size();
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

    // contributions per decode row: sum over its segments of their splits
    std::vector<int32_t> cnt((size_t)B, 0);
    auto n_splits = [&](const Segment &s) { return (s.j1 - s.j0 + split - 1) / split; };
    for (const Segment &s : segs)
        for (int32_t k = 0; k < s.nrows; ++k) cnt[seg_rows[s.rows_off + k]] += n_splits(s);

    // merge list layout: rows with more than one contribution, all heads
    std::vector<int32_t> moff((size_t)B, -1), cursor;
    int64_t n_merge_slots = 0;
    for (int32_t r : R) {
        if (cnt[r] < 2) continue;
        moff[r] = (int32_t)plan.merge_q.size();
        for (int32_t h = 0; h < Hq; ++h) {
            plan.merge_q.push_back(b.q_start[r] * Hq + h);
            plan.merge_ptr.push_back((int32_t)n_merge_slots);
            n_merge_slots += cnt[r];
        }
    }
    plan.merge_ptr.push_back((int32_t)n_merge_slots);
    plan.merge_slot.assign((size_t)n_merge_slots, -1);
    cursor.assign(plan.merge_q.size(), 0);

    int64_t n_slots = 0;
    for (size_t si = 0; si < segs.size(); ++si) {
        const Segment &s = segs[si];
        const int32_t tok_base = (int32_t)plan.tok_list.size();
        for (int32_t k = 0; k < s.nrows; ++k)
            plan.tok_list.push_back(b.q_start[seg_rows[s.rows_off + k]]);
        const int32_t rep = seg_rows[s.rows_off];
        const bool direct = (s.nrows == 1 && cnt[rep] == 1);
        for (int32_t j = s.j0; j < s.j1; j += split) {
            const int32_t kb = kBlock * j;
            const int32_t jend = std::min(j + split, s.j1);
            const int32_t ke = std::min(kBlock * jend, s.key_end);
            for (int32_t g = 0; g < Hkv; ++g) {
                for (int32_t hc = 0; hc < n_head_chunks; ++hc) {
                    const int32_t h0 = g * G + hc * kWaveQueries;
                    const int32_t nh = std::min(nh_full, G - hc * kWaveQueries);
                    const int32_t nt = kWaveQueries / nh;
                    for (int32_t k0 = 0; k0 < s.nrows; k0 += nt) {
                        const int32_t ntk = std::min(nt, s.nrows - k0);
                        AttnItem it;
                        it.tok_off = tok_base + k0;
                        it.shape = ntk | (nh << 8);
                        it.h0 = h0;
                        it.kvh = g;
                        it.bt_row = rep;
                        it.key_begin = kb;
                        it.key_end = ke;
                        it.part = -1;
                        if (!direct) {
                            it.part = (int32_t)n_slots;
                            for (int32_t i = 0; i < ntk; ++i) {
                                const int32_t r = seg_rows[s.rows_off + k0 + i];
                                for (int32_t jh = 0; jh < nh; ++jh) {
                                    const int32_t m = moff[r] + h0 + jh;
                                    plan.merge_slot[(size_t)plan.merge_ptr[m] + cursor[m]++] =
                                        (int32_t)(n_slots + i * nh + jh);
                                }
                            }
                            n_slots += (int64_t)ntk * nh;
                        }
                        plan.items.push_back(it);
                        ++plan.stats.decode_items;
                    }
                }
            }
        }
        if (si < n_shared) plan.stats.unique_kv_tokens += (int64_t)kBlock * (s.j1 - s.j0);
        else plan.stats.unique_kv_tokens += s.key_end - kBlock * s.j0;
    }

    for (int32_t v : plan.merge_slot)
        if (v < 0) return ECHO_E_INVALID;  // every merged result must have all its parts

    // ---- prefill rows: consecutive token slices, whole causal key range
    for (int32_t r = 0; r < B; ++r) {
        if (b.kind[r] != ECHO_ROW_PREFILL) continue;
        const int32_t q = b.q_start[r + 1] - b.q_start[r];
        const int32_t c = b.seq_lens[r] - q;
        plan.stats.unique_kv_tokens += b.seq_lens[r];
        for (int32_t g = 0; g < Hkv; ++g) {
            for (int32_t hc = 0; hc < n_head_chunks; ++hc) {
                const int32_t h0 = g * G + hc * kWaveQueries;
                const int32_t nh = std::min(nh_full, G - hc * kWaveQueries);
                const int32_t nt = kWaveQueries / nh;
                for (int32_t i0 = 0; i0 < q; i0 += nt) {
                    const int32_t ntk = std::min(nt, q - i0);
                    AttnItem it;
                    it.tok_off = b.q_start[r] + i0;
                    it.shape = ntk | (nh << 8) | kItemConsecutive;
                    it.h0 = h0;
                    it.kvh = g;
                    it.bt_row = r;
                    it.key_begin = 0;
                    it.key_end = c + i0 + ntk;
                    it.part = -1;
                    plan.items.push_back(it);
                    ++plan.stats.prefill_items;
                }
            }
        }
    }

    // heavy items first (counting sort on 32-key steps, stable)
    {
        const int32_t nb = 1024;
        std::vector<int32_t> count(nb + 1, 0);
        auto bucket = [&](const AttnItem &it) {
            int32_t steps = (it.key_end - it.key_begin + 31) / 32;
            return nb - 1 - std::min(steps, nb - 1);
        };
        for (const AttnItem &it : plan.items) ++count[bucket(it) + 1];
        for (int32_t i = 0; i < nb; ++i) count[i + 1] += count[i];
        std::vector<AttnItem> sorted(plan.items.size());
        for (const AttnItem &it : plan.items) sorted[count[bucket(it)]++] = it;
        plan.items.swap(sorted);
    }

    PlanLayout &L = plan.layout;
    L = PlanLayout{};
    L.head_dim = D;
    L.n_items = (int64_t)plan.items.size();
    L.n_tok_list = (int64_t)plan.tok_list.size();
    L.n_tokens = T;
    L.n_merge = (int64_t)plan.merge_q.size();
    L.n_merge_slots = n_merge_slots;
    L.n_slots = n_slots;
    int64_t w = 0;
    L.off_items = w;      w += L.n_items * 8;
    L.off_tok_list = w;   w += L.n_tok_list;
    L.off_klim = w;       w += L.n_tokens;
    L.off_merge_q = w;    w += L.n_merge;
    L.off_merge_ptr = w;  w += L.n_merge + 1;
    L.off_merge_slot = w; w += L.n_merge_slots;
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
    if (L.n_items) std::memcpy(w + L.off_items, plan.items.data(), L.n_items * sizeof(AttnItem));
    if (L.n_tok_list)
        std::memcpy(w + L.off_tok_list, plan.tok_list.data(), L.n_tok_list * 4);
    if (L.n_tokens) std::memcpy(w + L.off_klim, plan.klim.data(), L.n_tokens * 4);
    if (L.n_merge) std::memcpy(w + L.off_merge_q, plan.merge_q.data(), L.n_merge * 4);
    std::memcpy(w + L.off_merge_ptr, plan.merge_ptr.data(), (L.n_merge + 1) * 4);
    if (L.n_merge_slots)
        std::memcpy(w + L.off_merge_slot, plan.merge_slot.data(), L.n_merge_slots * 4);
}

}  // namespace echo
