// abi.cpp -- the extern "C" entry points declared in include/echo.h:
// validation, planning, plan upload and kernel launches.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "echo.h"
#include "kernels.hpp"
#include "plan.hpp"
#include "status.hpp"

namespace echo {

thread_local std::string g_error;

int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_error = buf;
    return code;
}

void clear_error() { g_error.clear(); }

}  // namespace echo

using namespace echo;

namespace {

int hip_fail(hipError_t e, const char *what) {
    return fail(ECHO_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool has_mirrors(const echo_batch_t *b) {
    return b->h_block_tables && b->h_seq_lens && b->h_q_start && b->h_row_kind;
}

int check_pool(const echo_kv_pool_t *p) {
    if (!p) return fail(ECHO_E_INVALID, "pool is NULL");
    if (p->dtype != ECHO_KV_BF16 && p->dtype != ECHO_KV_FP8_E4M3)
        return fail(ECHO_E_UNSUPPORTED, "kv dtype %d not supported", p->dtype);
    if (p->block_size != kBlock)
        return fail(ECHO_E_UNSUPPORTED, "block_size %d (only 16)", p->block_size);
    if (p->head_dim != 64 && p->head_dim != 128)
        return fail(ECHO_E_UNSUPPORTED, "head_dim %d (only 64, 128)", p->head_dim);
    if (p->num_blocks <= 0 || p->num_kv_heads <= 0)
        return fail(ECHO_E_INVALID, "num_blocks %d / num_kv_heads %d", p->num_blocks,
                    p->num_kv_heads);
    if (!p->k || !p->v) return fail(ECHO_E_INVALID, "pool k/v is NULL");
    if (p->dtype == ECHO_KV_FP8_E4M3 && (!p->k_scale || !p->v_scale))
        return fail(ECHO_E_INVALID, "e4m3 pool needs k_scale and v_scale");
    return ECHO_OK;
}

// Scalar checks, then (with host mirrors) per-row checks.
int check_batch(const echo_kv_pool_t *p, const echo_batch_t *b, bool for_append) {
    if (!b) return fail(ECHO_E_INVALID, "batch is NULL");
    const int32_t B = b->num_rows;
    if (B < 0) return fail(ECHO_E_INVALID, "num_rows %d", B);
    const bool any = b->h_block_tables || b->h_seq_lens || b->h_q_start || b->h_row_kind;
    if (any && !has_mirrors(b)) return fail(ECHO_E_INVALID, "host mirrors: give all four or none");
    if (B == 0) return ECHO_OK;
    if (b->max_blocks_per_row <= 0) return fail(ECHO_E_INVALID, "max_blocks_per_row <= 0");
    if (b->num_tokens < B) return fail(ECHO_E_INVALID, "num_tokens %d < num_rows %d",
                                       b->num_tokens, B);
    if (b->max_q_len < 1 || b->max_seq_len < 1)
        return fail(ECHO_E_INVALID, "max_q_len / max_seq_len must be >= 1");
    if ((int64_t)b->max_seq_len > (int64_t)b->max_blocks_per_row * kBlock)
        return fail(ECHO_E_INVALID, "max_seq_len %d exceeds the block table width", b->max_seq_len);
    if (!b->block_tables || !b->seq_lens || !b->q_start || !b->row_kind)
        return fail(ECHO_E_INVALID, "device metadata pointer is NULL");
    if (!has_mirrors(b)) return ECHO_OK;

    const int32_t *qs = b->h_q_start, *sl = b->h_seq_lens, *bt = b->h_block_tables;
    if (qs[0] != 0) return fail(ECHO_E_INVALID, "q_start[0] = %d", qs[0]);
    if (qs[B] != b->num_tokens)
        return fail(ECHO_E_INVALID, "q_start[num_rows] = %d != num_tokens %d", qs[B],
                    b->num_tokens);
    for (int32_t r = 0; r < B; ++r) {
        const int32_t q = qs[r + 1] - qs[r], L = sl[r];
        const uint8_t kind = b->h_row_kind[r];
        if (kind != ECHO_ROW_DECODE && kind != ECHO_ROW_PREFILL)
            return fail(ECHO_E_INVALID, "row %d: kind %d", r, kind);
        if (q < 1) return fail(ECHO_E_INVALID, "row %d: %d new tokens", r, q);
        if (kind == ECHO_ROW_DECODE && q != 1)
            return fail(ECHO_E_INVALID, "row %d: decode row with %d new tokens", r, q);
        if (q > b->max_q_len) return fail(ECHO_E_INVALID, "row %d: q %d > max_q_len", r, q);
        if (L < q) return fail(ECHO_E_INVALID, "row %d: seq_len %d < new tokens %d", r, L, q);
        if (L > b->max_seq_len) return fail(ECHO_E_INVALID, "row %d: seq_len > max_seq_len", r);
        const int32_t nb = (L + kBlock - 1) / kBlock;
        for (int32_t j = 0; j < nb; ++j) {
            const int32_t blk = bt[(size_t)r * b->max_blocks_per_row + j];
            if (blk < 0 || blk >= p->num_blocks)
                return fail(ECHO_E_RANGE, "row %d: block_tables[%d] = %d outside [0, %d)", r, j,
                            blk, p->num_blocks);
        }
    }
    if (!for_append) return ECHO_OK;

    // every block written by this append is referenced exactly once
    thread_local std::vector<uint32_t> stamp;
    thread_local std::vector<int32_t> owner_row, owner_j;
    thread_local uint32_t epoch = 0;
    if (stamp.size() < (size_t)p->num_blocks) {
        stamp.assign((size_t)p->num_blocks, 0);
        owner_row.assign((size_t)p->num_blocks, -1);
        owner_j.assign((size_t)p->num_blocks, -1);
        epoch = 0;
    }
    if (++epoch == 0) {
        std::fill(stamp.begin(), stamp.end(), 0u);
        epoch = 1;
    }
    for (int32_t r = 0; r < B; ++r) {
        const int32_t q = qs[r + 1] - qs[r], L = sl[r], p0 = L - q;
        for (int32_t j = p0 / kBlock; j <= (L - 1) / kBlock; ++j) {
            const int32_t blk = bt[(size_t)r * b->max_blocks_per_row + j];
            if (stamp[blk] == epoch)
                return fail(ECHO_E_ALIAS_WRITE, "block %d written by rows %d and %d", blk,
                            owner_row[blk], r);
            stamp[blk] = epoch;
            owner_row[blk] = r;
            owner_j[blk] = j;
        }
    }
    for (int32_t r = 0; r < B; ++r) {
        const int32_t nb = (sl[r] + kBlock - 1) / kBlock;
        for (int32_t j = 0; j < nb; ++j) {
            const int32_t blk = bt[(size_t)r * b->max_blocks_per_row + j];
            if (stamp[blk] == epoch && (owner_row[blk] != r || owner_j[blk] != j))
                return fail(ECHO_E_ALIAS_WRITE,
                            "row %d appends into block %d, which row %d also references",
                            owner_row[blk], blk, r);
        }
    }
    return ECHO_OK;
}

HostBatch host_batch(const echo_batch_t *b) {
    HostBatch h;
    h.num_rows = b->num_rows;
    h.mbr = b->max_blocks_per_row;
    h.num_tokens = b->num_tokens;
    h.max_q_len = b->max_q_len;
    h.max_seq_len = b->max_seq_len;
    h.bt = b->h_block_tables;
    h.seq_lens = b->h_seq_lens;
    h.q_start = b->h_q_start;
    h.kind = b->h_row_kind;
    return h;
}

PlanOptions plan_options(const echo_kv_pool_t *pool) {
    PlanOptions o;
    static const int split = [] {   // override for tuning sweeps
        const char *e = getenv("ECHO_SPLIT_BLOCKS");
        int v = e ? atoi(e) : 0;
        return v > 0 ? v : 0;
    }();
    const int64_t block_bytes = 2 * (int64_t)kBlock * pool->head_dim *
                                (pool->dtype == ECHO_KV_FP8_E4M3 ? 1 : 2);
    o.split_blocks = split > 0 ? split : (int)std::max<int64_t>(1, kSplitBytes / block_bytes);
    // compute units of the current device (256 on MI355X; also the value
    // used by host-only calls made where no device is present)
    static std::atomic<int> cus[64];
    int dev = 0;
    if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < 64) {
        int v = cus[dev].load(std::memory_order_relaxed);
        if (v == 0) {
            if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
                v <= 0)
                v = 256;
            cus[dev].store(v, std::memory_order_relaxed);
        }
        o.num_cus = v;
    } else {
        (void)hipGetLastError();
        o.num_cus = 256;
    }
    return o;
}

int plan_for(const echo_kv_pool_t *pool, const echo_batch_t *batch, int32_t num_q_heads,
             Plan &plan) {
    int rc = check_pool(pool);
    if (rc) return rc;
    rc = check_batch(pool, batch, false);
    if (rc) return rc;
    if (batch->num_rows > 0 && !has_mirrors(batch))
        return fail(ECHO_E_INVALID, "echo_attn_mixed needs the host mirrors of the batch");
    if (num_q_heads <= 0 || num_q_heads % pool->num_kv_heads != 0)
        return fail(ECHO_E_INVALID, "num_q_heads %d is not a multiple of num_kv_heads %d",
                    num_q_heads, pool->num_kv_heads);
    if (num_q_heads / pool->num_kv_heads > kPrefillQueries)
        return fail(ECHO_E_UNSUPPORTED, "more than %d query heads per KV head", kPrefillQueries);
    if (batch->num_rows == 0) {
        plan.desc.clear();
        plan.merge_ptr.assign(1, 0);
        plan.layout = PlanLayout{};
        plan.layout.upload_words = 1;
        plan.layout.total_words = 64;
        return ECHO_OK;
    }
    return build_plan(host_batch(batch), pool->num_kv_heads, num_q_heads, pool->head_dim,
                      plan_options(pool), plan);
}

// Shortest XCD run (log2 of decode workgroups) for a plan: the waves that
// read one shared key range are consecutive in the work order, and a run
// twice their span keeps most such groups inside one XCD's L2 (a group that
// straddles two runs is fetched from HBM by both XCDs).
int run_log2_for(int32_t sibling_waves) {
    const int64_t wgs = 2 * (((int64_t)sibling_waves + 3) / 4);
    int l = 0;
    while (l < 5 && ((int64_t)1 << l) < wgs) ++l;
    return l;
}

// Pinned host staging for plan uploads: a small ring per device, each slot
// guarded by an event so that a buffer is refilled only after the kernel
// that copies it to the workspace has completed.
struct StagingSlot {
    void *host = nullptr;
    void *dev = nullptr;   // the same memory as the device sees it
    size_t cap = 0;
    hipEvent_t ev = nullptr;
    bool pending = false;
};
struct Staging {
    std::mutex mu;
    StagingSlot slots[4];
    int next = 0;
};
Staging g_staging[64];

// Opt-in per-kernel timing (echo_profile / echo_attn_timing).
struct Profile {
    bool on = false;
    bool valid = false;
    int device = -1;
    hipEvent_t ev[8] = {};          // upload pair, then one pair per kernel
    bool launched[4] = {};          // upload, prefill, decode, merge
};
thread_local Profile g_prof;

}  // namespace

bool echo::profile_enabled() { return g_prof.on; }

namespace {

int profile_events(hipEvent_t **out) {
    *out = nullptr;
    if (!g_prof.on) return ECHO_OK;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (g_prof.device != dev) {
        for (hipEvent_t &x : g_prof.ev) {
            if (x) (void)hipEventDestroy(x);
            x = nullptr;
        }
        g_prof.device = dev;
    }
    for (hipEvent_t &x : g_prof.ev) {
        if (!x && (e = hipEventCreate(&x)) != hipSuccess) return hip_fail(e, "hipEventCreate");
    }
    *out = g_prof.ev;
    return ECHO_OK;
}

int upload_plan(const Plan &plan, void *workspace, hipStream_t stream) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= 64) return fail(ECHO_E_HIP, "device index %d", dev);
    Staging &st = g_staging[dev];
    std::lock_guard<std::mutex> lock(st.mu);
    StagingSlot &s = st.slots[st.next];
    st.next = (st.next + 1) % 4;
    if (!s.ev) {
        e = hipEventCreateWithFlags(&s.ev, hipEventDisableTiming);
        if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
    }
    if (s.pending) {
        e = hipEventSynchronize(s.ev);
        if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
        s.pending = false;
    }
    const size_t bytes = (size_t)plan.layout.upload_words * 4;
    if (s.cap < bytes) {
        if (s.host) (void)hipHostFree(s.host);
        s.host = s.dev = nullptr;
        s.cap = 0;
        const size_t cap = std::max<size_t>(bytes + bytes / 2, 1 << 20);
        // coherent: the upload kernel reads what the host wrote, uncached
        e = hipHostMalloc(&s.host, cap, hipHostMallocMapped | hipHostMallocCoherent);
        if (e != hipSuccess) return hip_fail(e, "hipHostMalloc (plan staging)");
        e = hipHostGetDevicePointer(&s.dev, s.host, 0);
        if (e != hipSuccess) return hip_fail(e, "hipHostGetDevicePointer (plan staging)");
        s.cap = cap;
    }
    pack_plan(plan, s.host);
    e = launch_plan_upload(s.dev, workspace, plan.layout.upload_words, stream);
    if (e != hipSuccess) return hip_fail(e, "plan upload launch");
    e = hipEventRecord(s.ev, stream);
    if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
    s.pending = true;
    return ECHO_OK;
}

}  // namespace

extern "C" {

const char *echo_status_string(int status) {
    switch (status) {
        case ECHO_OK: return "ECHO_OK";
        case ECHO_E_INVALID: return "ECHO_E_INVALID";
        case ECHO_E_RANGE: return "ECHO_E_RANGE";
        case ECHO_E_ALIAS_WRITE: return "ECHO_E_ALIAS_WRITE";
        case ECHO_E_WORKSPACE: return "ECHO_E_WORKSPACE";
        case ECHO_E_UNSUPPORTED: return "ECHO_E_UNSUPPORTED";
        case ECHO_E_HIP: return "ECHO_E_HIP";
        case ECHO_E_NOSPACE: return "ECHO_E_NOSPACE";
        default: return "ECHO_E_UNKNOWN";
    }
}

const char *echo_last_error(void) { return g_error.c_str(); }

int echo_profile(int enable) {
    const int prev = g_prof.on ? 1 : 0;
    g_prof.on = enable != 0;
    return prev;
}

int echo_attn_timing(echo_attn_timing_t *t) {
    g_error.clear();
    if (!t) return fail(ECHO_E_INVALID, "timing is NULL");
    if (!g_prof.valid) return fail(ECHO_E_INVALID, "no profiled echo_attn_mixed call on this thread");
    float ms[4] = {0.f, 0.f, 0.f, 0.f};
    for (int k = 0; k < 4; ++k) {
        if (!g_prof.launched[k]) continue;
        hipError_t e = hipEventSynchronize(g_prof.ev[2 * k + 1]);
        if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
        e = hipEventElapsedTime(&ms[k], g_prof.ev[2 * k], g_prof.ev[2 * k + 1]);
        if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    }
    t->upload_ms = ms[0];
    t->prefill_ms = ms[1];
    t->decode_ms = ms[2];
    t->merge_ms = ms[3];
    return ECHO_OK;
}

int echo_validate(const echo_kv_pool_t *pool, const echo_batch_t *batch, int32_t for_append) {
    g_error.clear();
    int rc = check_pool(pool);
    if (rc) return rc;
    return check_batch(pool, batch, for_append != 0);
}

int echo_kv_append(const echo_kv_pool_t *pool, const echo_batch_t *batch, const void *k_new,
                   const void *v_new, void *stream) {
    g_error.clear();
    int rc = check_pool(pool);
    if (rc) return rc;
    rc = check_batch(pool, batch, true);
    if (rc) return rc;
    if (batch->num_rows == 0) return ECHO_OK;
    if (!k_new || !v_new) return fail(ECHO_E_INVALID, "k_new / v_new is NULL");
    AppendArgs a;
    a.k = pool->k;
    a.v = pool->v;
    a.k_scale = pool->k_scale;
    a.v_scale = pool->v_scale;
    a.k_new = (const uint16_t *)k_new;
    a.v_new = (const uint16_t *)v_new;
    a.block_tables = batch->block_tables;
    a.seq_lens = batch->seq_lens;
    a.q_start = batch->q_start;
    a.num_blocks = pool->num_blocks;
    a.num_kv_heads = pool->num_kv_heads;
    a.max_blocks_per_row = batch->max_blocks_per_row;
    a.num_rows = batch->num_rows;
    // a row of q new tokens writes at most q / 16 + 2 blocks
    a.n_units = ((int64_t)batch->num_tokens / kBlock + 2 * (int64_t)batch->num_rows) *
                pool->num_kv_heads;
    // direct form when a padded grid (every row given the most blocks a row
    // can write: q tokens span at most (q + 14) / 16 + 1 blocks) is at most
    // twice the compact bound: no scan, no LDS
    const int64_t bpr =
        std::min<int64_t>((batch->max_q_len + kBlock - 2) / kBlock + 1, batch->max_blocks_per_row);
    a.blocks_per_row =
        (int64_t)batch->num_rows * bpr * pool->num_kv_heads <= 2 * a.n_units ? (int32_t)bpr : 0;
    hipError_t e = launch_append(a, pool->head_dim, pool->dtype == ECHO_KV_FP8_E4M3,
                                 (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "append launch");
    return ECHO_OK;
}

int echo_block_copy(const echo_kv_pool_t *pool, const int32_t *pairs, int32_t n_pairs,
                    const int32_t *h_pairs, void *stream) {
    g_error.clear();
    int rc = check_pool(pool);
    if (rc) return rc;
    if (n_pairs < 0) return fail(ECHO_E_INVALID, "n_pairs %d", n_pairs);
    if (n_pairs == 0) return ECHO_OK;
    if (!pairs) return fail(ECHO_E_INVALID, "pairs is NULL");
    if (h_pairs) {
        std::vector<int32_t> srcs, dsts;
        srcs.reserve(n_pairs);
        dsts.reserve(n_pairs);
        for (int32_t i = 0; i < n_pairs; ++i) {
            const int32_t s = h_pairs[2 * i], d = h_pairs[2 * i + 1];
            if (s < 0 || s >= pool->num_blocks || d < 0 || d >= pool->num_blocks)
                return fail(ECHO_E_RANGE, "pair %d: (%d, %d) outside [0, %d)", i, s, d,
                            pool->num_blocks);
            if (s == d) return fail(ECHO_E_INVALID, "pair %d copies block %d onto itself", i, s);
            srcs.push_back(s);
            dsts.push_back(d);
        }
        std::sort(srcs.begin(), srcs.end());
        std::sort(dsts.begin(), dsts.end());
        if (std::adjacent_find(dsts.begin(), dsts.end()) != dsts.end())
            return fail(ECHO_E_INVALID, "a destination block appears twice");
        for (int32_t d : dsts)
            if (std::binary_search(srcs.begin(), srcs.end(), d))
                return fail(ECHO_E_INVALID, "block %d is both a source and a destination", d);
    }
    BlockCopyArgs a;
    a.k = pool->k;
    a.v = pool->v;
    const bool fp8 = pool->dtype == ECHO_KV_FP8_E4M3;
    a.k_scale = fp8 ? pool->k_scale : nullptr;
    a.v_scale = fp8 ? pool->v_scale : nullptr;
    a.pairs = pairs;
    a.n_pairs = n_pairs;
    a.num_blocks = pool->num_blocks;
    a.num_kv_heads = pool->num_kv_heads;
    a.block_bytes = (int64_t)pool->num_kv_heads * kBlock * pool->head_dim * (fp8 ? 1 : 2);
    a.chunks = (int32_t)((a.block_bytes / 16 + 1023) / 1024);
    hipError_t e = launch_block_copy(a, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "block copy launch");
    return ECHO_OK;
}

size_t echo_attn_workspace_bytes(const echo_kv_pool_t *pool, const echo_batch_t *batch,
                                 int32_t num_q_heads) {
    g_error.clear();
    thread_local Plan plan;
    if (plan_for(pool, batch, num_q_heads, plan) != ECHO_OK) return 0;
    return (size_t)plan.layout.total_words * 4;
}

int echo_attn_plan_stats(const echo_kv_pool_t *pool, const echo_batch_t *batch,
                         int32_t num_q_heads, echo_plan_stats_t *stats) {
    g_error.clear();
    if (!stats) return fail(ECHO_E_INVALID, "stats is NULL");
    thread_local Plan plan;
    int rc = plan_for(pool, batch, num_q_heads, plan);
    if (rc) return rc;
    std::memset(stats, 0, sizeof *stats);
    stats->work_items = plan.stats.decode_items + plan.stats.prefill_items;
    stats->decode_items = plan.stats.decode_items;
    stats->prefill_items = plan.stats.prefill_items;
    stats->shared_segments = plan.stats.shared_segments;
    stats->partial_slots = plan.layout.n_slots;
    stats->merged_queries = plan.layout.n_merge_rows * num_q_heads;
    stats->logical_kv_tokens = plan.stats.logical_kv_tokens;
    stats->causal_pairs = plan.stats.causal_pairs;
    stats->decode_kv_tokens = plan.stats.decode_kv_tokens;
    stats->prefill_causal_pairs = plan.stats.prefill_causal_pairs;
    stats->workspace_bytes = plan.layout.total_words * 4;
    // distinct (block, slot) pairs that the batch reads
    std::vector<uint8_t> used((size_t)pool->num_blocks, 0);
    for (int32_t r = 0; r < batch->num_rows; ++r) {
        const int32_t L = batch->h_seq_lens[r];
        for (int32_t j = 0; j * kBlock < L; ++j) {
            const int32_t blk = batch->h_block_tables[(size_t)r * batch->max_blocks_per_row + j];
            const int32_t n = std::min(kBlock, L - j * kBlock);
            if (n > used[blk]) used[blk] = (uint8_t)n;
        }
    }
    for (uint8_t n : used) stats->unique_kv_tokens += n;
    return ECHO_OK;
}

int echo_attn_plan_pack(const echo_kv_pool_t *pool, const echo_batch_t *batch,
                        int32_t num_q_heads, echo_plan_layout_t *layout, void *words,
                        size_t bytes) {
    g_error.clear();
    if (!layout) return fail(ECHO_E_INVALID, "layout is NULL");
    thread_local Plan plan;
    int rc = plan_for(pool, batch, num_q_heads, plan);
    if (rc) return rc;
    const PlanLayout &L = plan.layout;
    layout->n_desc = L.n_desc;
    layout->n_pdesc = L.n_pdesc;
    layout->n_tok_list = L.n_tok_list;
    layout->n_tokens = L.n_tokens;
    layout->n_merge_rows = L.n_merge_rows;
    layout->n_merge_entries = L.n_merge_entries;
    layout->n_slots = L.n_slots;
    layout->off_desc = L.off_desc;
    layout->off_pdesc = L.off_pdesc;
    layout->off_tok_list = L.off_tok_list;
    layout->off_klim = L.off_klim;
    layout->off_merge_tok = L.off_merge_tok;
    layout->off_merge_ptr = L.off_merge_ptr;
    layout->off_merge_ent = L.off_merge_ent;
    layout->upload_words = L.upload_words;
    layout->off_part_lse = L.off_part_lse;
    layout->off_part_o = L.off_part_o;
    layout->total_words = L.total_words;
    layout->head_chunks = plan.head_chunks;
    layout->heads_per_chunk = plan.heads_per_chunk;
    if (!words) return ECHO_OK;
    if (bytes < (size_t)L.upload_words * 4)
        return fail(ECHO_E_WORKSPACE, "plan buffer of %zu bytes, need %lld", bytes,
                    (long long)L.upload_words * 4);
    pack_plan(plan, words);
    return ECHO_OK;
}

int echo_attn_mixed(const echo_kv_pool_t *pool, const echo_batch_t *batch, const void *q,
                    int32_t num_q_heads, float sm_scale, float *out, void *workspace,
                    size_t workspace_bytes, void *stream) {
    g_error.clear();
    thread_local Plan plan;
    int rc = plan_for(pool, batch, num_q_heads, plan);
    if (rc) return rc;
    if (batch->num_rows == 0) return ECHO_OK;
    if (!q || !out) return fail(ECHO_E_INVALID, "q / out is NULL");
    if (!(sm_scale > 0.f) || !std::isfinite(sm_scale))
        return fail(ECHO_E_INVALID, "sm_scale must be positive and finite");
    const size_t need = (size_t)plan.layout.total_words * 4;
    if (!workspace || workspace_bytes < need)
        return fail(ECHO_E_WORKSPACE, "workspace of %zu bytes, need %zu", workspace_bytes, need);
    if (((uintptr_t)workspace & 255u) != 0)
        return fail(ECHO_E_WORKSPACE, "workspace must be 256-byte aligned");
    int32_t pf_blocks = 0;
    for (const PrefillDesc &d : plan.pdesc)
        pf_blocks = std::max(pf_blocks, (d.key_end + kBlock - 1) / kBlock - d.key_begin / kBlock);
    if (pf_blocks > prefill_max_blocks(pool->head_dim))
        return fail(ECHO_E_UNSUPPORTED, "prefill row of %d blocks exceeds the %d-block limit",
                    pf_blocks, prefill_max_blocks(pool->head_dim));
    hipStream_t s = (hipStream_t)stream;
    hipEvent_t *ev = nullptr;
    rc = profile_events(&ev);
    if (rc) return rc;
    g_prof.valid = false;
    if (ev) {
        hipError_t e0 = hipEventRecord(ev[0], s);
        if (e0 != hipSuccess) return hip_fail(e0, "hipEventRecord");
    }
    rc = upload_plan(plan, workspace, s);
    if (rc) return rc;
    if (ev) {
        hipError_t e0 = hipEventRecord(ev[1], s);
        if (e0 != hipSuccess) return hip_fail(e0, "hipEventRecord");
    }

    const PlanLayout &L = plan.layout;
    int32_t *w = (int32_t *)workspace;
    AttnArgs a;
    a.desc = (const WorkDesc *)(w + L.off_desc);
    a.n_waves = L.n_desc * plan.waves_per_desc;
    a.waves_per_desc = plan.waves_per_desc;
    a.run_log2 = run_log2_for(plan.sibling_waves);
    a.head_chunks = plan.head_chunks;
    a.heads_per_chunk = plan.heads_per_chunk;
    a.group = num_q_heads / pool->num_kv_heads;
    a.tok_list = w + L.off_tok_list;
    a.klim = w + L.off_klim;
    a.q = (const uint16_t *)q;
    a.num_q_heads = num_q_heads;
    a.num_kv_heads = pool->num_kv_heads;
    a.k = pool->k;
    a.v = pool->v;
    a.k_scale = pool->k_scale;
    a.v_scale = pool->v_scale;
    a.block_tables = batch->block_tables;
    a.max_blocks_per_row = batch->max_blocks_per_row;
    a.scale_log2 = (float)((double)sm_scale * 1.4426950408889634);
    a.out = out;
    a.part_o = (float *)(w + L.off_part_o);
    a.part_lse = (float *)(w + L.off_part_lse);
    MergeArgs m;
    m.n_waves = L.n_merge_rows * ((num_q_heads + 3) / 4);
    m.num_q_heads = num_q_heads;
    m.head_chunks = plan.head_chunks;
    m.heads_per_chunk = plan.heads_per_chunk;
    m.group = a.group;
    m.merge_tok = w + L.off_merge_tok;
    m.merge_ptr = w + L.off_merge_ptr;
    m.merge_ent = w + L.off_merge_ent;
    m.part_o = a.part_o;
    m.part_lse = a.part_lse;
    m.out = out;
    PrefillArgs pf;
    pf.pdesc = (const PrefillDesc *)(w + L.off_pdesc);
    pf.n_pdesc = plan.pdesc_grid;   // chained descriptors follow these
    pf.n_logical = (int32_t)((int64_t)plan.pdesc_grid * pool->num_kv_heads);
    pf.per_xcd = (pf.n_logical + 7) / 8;
    pf.group = a.group;
    pf.klim = a.klim;
    pf.q = a.q;
    pf.num_q_heads = num_q_heads;
    pf.num_kv_heads = pool->num_kv_heads;
    pf.k = pool->k;
    pf.v = pool->v;
    pf.k_scale = pool->k_scale;
    pf.v_scale = pool->v_scale;
    pf.block_tables = batch->block_tables;
    pf.max_blocks_per_row = batch->max_blocks_per_row;
    pf.scale_log2 = a.scale_log2;
    pf.out = out;
    pf.max_blocks = pf_blocks;
    pf.head_chunks = plan.head_chunks;
    pf.heads_per_chunk = plan.heads_per_chunk;
    pf.part_o = a.part_o;
    pf.part_lse = a.part_lse;
    const int D = pool->head_dim;
    const bool fp8 = pool->dtype == ECHO_KV_FP8_E4M3;
    hipError_t e;
    // prefill, decode and merge in that order on the caller's stream; with
    // profiling on, an event pair around each kernel that launches (an empty
    // pair still costs GPU time between the two records)
    if (pf.n_logical > 0) {
        if (ev && (e = hipEventRecord(ev[2], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
        if ((e = launch_prefill(pf, D, fp8, s)) != hipSuccess) return hip_fail(e, "prefill launch");
        if (ev && (e = hipEventRecord(ev[3], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    }
    if (a.n_waves > 0) {
        if (ev && (e = hipEventRecord(ev[4], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
        if ((e = launch_decode(a, D, fp8, s)) != hipSuccess) return hip_fail(e, "decode launch");
        if (ev && (e = hipEventRecord(ev[5], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    }
    if (m.n_waves > 0) {
        if (ev && (e = hipEventRecord(ev[6], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
        if ((e = launch_merge(m, D, s)) != hipSuccess) return hip_fail(e, "merge launch");
        if (ev && (e = hipEventRecord(ev[7], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    }
    g_prof.valid = ev != nullptr;
    g_prof.launched[0] = true;
    g_prof.launched[1] = pf.n_logical > 0;
    g_prof.launched[2] = a.n_waves > 0;
    g_prof.launched[3] = m.n_waves > 0;
    return ECHO_OK;
}

}  // extern "C"
