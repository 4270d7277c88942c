// abi.cpp -- the extern "C" entry points declared in include/echo.h:
// validation, planning, plan upload and kernel launches.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
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
    if (b->max_seq_len > kMaxSeqLen)
        return fail(ECHO_E_UNSUPPORTED, "max_seq_len %d above %d", b->max_seq_len, kMaxSeqLen);
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
        // differences of caller values in 64 bits: no overflow before the checks
        const int64_t q = (int64_t)qs[r + 1] - qs[r], L = sl[r];
        const uint8_t kind = b->h_row_kind[r];
        if (kind != ECHO_ROW_DECODE && kind != ECHO_ROW_PREFILL)
            return fail(ECHO_E_INVALID, "row %d: kind %d", r, kind);
        if (q < 1) return fail(ECHO_E_INVALID, "row %d: %lld new tokens", r, (long long)q);
        if (kind == ECHO_ROW_DECODE && q != 1)
            return fail(ECHO_E_INVALID, "row %d: decode row with %lld new tokens", r, (long long)q);
        if (q > b->max_q_len)
            return fail(ECHO_E_INVALID, "row %d: q %lld > max_q_len", r, (long long)q);
        if (L < q)
            return fail(ECHO_E_INVALID, "row %d: seq_len %lld < new tokens %lld", r, (long long)L,
                        (long long)q);
        if (L > b->max_seq_len) return fail(ECHO_E_INVALID, "row %d: seq_len > max_seq_len", r);
        const int32_t nb = (int32_t)((L + kBlock - 1) / kBlock);
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
        const int32_t nb = (int32_t)(((int64_t)sl[r] + kBlock - 1) / kBlock);
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

// The plan goes to the device through the caller's pinned host workspace:
// packed there on the host, then copied into the device workspace by a
// kernel on the caller's stream.  The caller keeps the host workspace
// untouched until that kernel has run (it is read on the device, not here).
int check_host_workspace(void *host_ws, size_t bytes, size_t need, void **dev_ptr) {
    if (!host_ws || bytes < need)
        return fail(ECHO_E_WORKSPACE, "host workspace of %zu bytes, need %zu", bytes, need);
    if (((uintptr_t)host_ws & 15u) != 0)
        return fail(ECHO_E_WORKSPACE, "host workspace must be 16-byte aligned");
    hipError_t e = hipHostGetDevicePointer(dev_ptr, host_ws, 0);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(ECHO_E_WORKSPACE, "host workspace is not pinned host memory mapped for the "
                                      "device (%s)", hipGetErrorString(e));
    }
    return ECHO_OK;
}

// Scalar bounds of the device-built plan for a batch without host mirrors.
struct DevLayout {
    int32_t split_keys = 0, tile_tokens = 0, slots_per_desc = 0, head_chunks = 1,
            heads_per_chunk = 1, waves_per_desc = 1, pf_max_blocks = 0;
    int64_t cap_desc = 0, cap_pdesc = 0, cap_mrows = 0, cap_ent = 0, cap_slots = 0;
    int64_t off_row_info = 0, off_desc = 0, off_pdesc = 0, off_mtok = 0, off_mptr = 0,
            off_ment = 0, off_lse = 0, off_o = 0, total_words = 0;
};

int64_t align_up(int64_t w, int64_t a) { return (w + a - 1) / a * a; }

int dev_layout(const echo_kv_pool_t *pool, const echo_batch_t *b, int32_t Hq, DevLayout &L) {
    const int64_t B = b->num_rows, Hkv = pool->num_kv_heads, G = Hq / Hkv;
    L.heads_per_chunk = (int32_t)std::min<int64_t>(G, kWaveQueries);
    L.head_chunks = (int32_t)((G + kWaveQueries - 1) / kWaveQueries);
    L.waves_per_desc = (int32_t)(Hkv * L.head_chunks);
    L.slots_per_desc = L.waves_per_desc * L.heads_per_chunk;
    // decode pieces: the host planner's rule, with every row taken at the
    // longest length the scalars allow
    const PlanOptions o = plan_options(pool);
    const int64_t seg_blocks = B * (((int64_t)b->max_seq_len + kBlock - 1) / kBlock);
    const int64_t split = std::max<int64_t>(
        std::min(kMinSplitBlocks, std::max(2, o.split_blocks)),
        std::min<int64_t>(o.split_blocks, seg_blocks * Hkv * L.head_chunks / kSplitTargetUnits));
    L.split_keys = (int32_t)(split * kBlock);
    L.tile_tokens = (int32_t)std::max<int64_t>(1, kPrefillQueries / G);
    const int64_t P = ((int64_t)b->max_seq_len + L.split_keys - 1) / L.split_keys;
    L.cap_desc = B * P;
    L.cap_ent = B * P;
    L.cap_mrows = B;
    L.cap_slots = B * P * L.slots_per_desc;
    L.cap_pdesc = std::min(B * (((int64_t)b->max_q_len + L.tile_tokens - 1) / L.tile_tokens),
                           ((int64_t)b->num_tokens + L.tile_tokens - 1) / L.tile_tokens + B);
    if (L.cap_desc * L.waves_per_desc > ((int64_t)1 << 31) - (1 << 20) ||
        L.cap_pdesc * Hkv > ((int64_t)1 << 31) - (1 << 20) || L.cap_slots > ((int64_t)1 << 31) - 1)
        return fail(ECHO_E_UNSUPPORTED, "batch too large for a plan built on the device");
    L.pf_max_blocks = (int32_t)std::min<int64_t>(((int64_t)b->max_seq_len + kBlock - 1) / kBlock,
                                                 prefill_max_blocks(pool->head_dim));
    int64_t w = kHdrWords;
    L.off_row_info = w;  w = align_up(w + B, 8);
    L.off_desc = w;      w += L.cap_desc * (int64_t)(sizeof(WorkDesc) / 4);
    L.off_pdesc = w;     w += L.cap_pdesc * (int64_t)(sizeof(PrefillDesc) / 4);
    L.off_mtok = w;      w += L.cap_mrows;
    L.off_mptr = w;      w += L.cap_mrows + 1;
    L.off_ment = w;      w += 2 * L.cap_ent;
    w = align_up(w, 64);
    L.off_lse = w;       w += L.cap_slots;
    w = align_up(w, 64);
    L.off_o = w;         w += L.cap_slots * pool->head_dim;
    L.total_words = align_up(w, 64);
    return ECHO_OK;
}

// Everything echo_attn_mixed launches after the plan is in the workspace.
struct AttnLaunch {
    const WorkDesc *desc = nullptr;
    const PrefillDesc *pdesc = nullptr;
    const int32_t *tok_list = nullptr, *klim = nullptr, *merge_tok = nullptr,
                  *merge_ptr = nullptr, *merge_ent = nullptr, *counts = nullptr;
    float *part_lse = nullptr, *part_o = nullptr;
    int64_t n_desc = 0, n_merge_rows = 0;
    int32_t n_pdesc_grid = 0;     // prefill descriptors that get workgroups (a capacity with counts)
    int32_t head_chunks = 1, heads_per_chunk = 1, waves_per_desc = 1, run_log2 = 0,
            pf_max_blocks = 0;
};

int launch_attention(const echo_kv_pool_t *pool, const echo_batch_t *batch, const void *q,
                     int32_t num_q_heads, float sm_scale, float *out, const AttnLaunch &w,
                     hipStream_t s, hipEvent_t *ev) {
    AttnArgs a;
    a.desc = w.desc;
    a.n_waves = w.n_desc * w.waves_per_desc;
    a.waves_per_desc = w.waves_per_desc;
    a.run_log2 = w.run_log2;
    a.head_chunks = w.head_chunks;
    a.heads_per_chunk = w.heads_per_chunk;
    a.group = num_q_heads / pool->num_kv_heads;
    a.tok_list = w.tok_list;
    a.klim = w.klim;
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
    a.part_o = w.part_o;
    a.part_lse = w.part_lse;
    a.counts = w.counts;
    MergeArgs m;
    m.n_waves = w.n_merge_rows * ((num_q_heads + 3) / 4);
    m.counts = w.counts;
    m.num_q_heads = num_q_heads;
    m.head_chunks = w.head_chunks;
    m.heads_per_chunk = w.heads_per_chunk;
    m.group = a.group;
    m.merge_tok = w.merge_tok;
    m.merge_ptr = w.merge_ptr;
    m.merge_ent = w.merge_ent;
    m.part_o = a.part_o;
    m.part_lse = a.part_lse;
    m.out = out;
    PrefillArgs pf;
    pf.pdesc = w.pdesc;
    pf.n_pdesc = w.n_pdesc_grid;   // chained descriptors follow these
    pf.n_logical = (int32_t)((int64_t)w.n_pdesc_grid * pool->num_kv_heads);
    pf.per_xcd = (pf.n_logical + 7) / 8;
    pf.group = a.group;
    pf.seq_lens = batch->seq_lens;
    pf.q_start = batch->q_start;
    pf.counts = w.counts;
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
    pf.max_blocks = w.pf_max_blocks;
    pf.head_chunks = w.head_chunks;
    pf.heads_per_chunk = w.heads_per_chunk;
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

// Checks shared by both planning modes.
int check_attn_args(const echo_kv_pool_t *pool, const echo_batch_t *batch, int32_t num_q_heads) {
    int rc = check_pool(pool);
    if (rc) return rc;
    rc = check_batch(pool, batch, false);
    if (rc) return rc;
    if (num_q_heads <= 0 || num_q_heads % pool->num_kv_heads != 0)
        return fail(ECHO_E_INVALID, "num_q_heads %d is not a multiple of num_kv_heads %d",
                    num_q_heads, pool->num_kv_heads);
    if (num_q_heads / pool->num_kv_heads > kPrefillQueries)
        return fail(ECHO_E_UNSUPPORTED, "more than %d query heads per KV head", kPrefillQueries);
    return ECHO_OK;
}

// The device-built plan (no host mirrors): two planning kernels, then the
// attention kernels reading their counts from the plan's header.
int attn_device_planned(const echo_kv_pool_t *pool, const echo_batch_t *batch, const void *q,
                        int32_t num_q_heads, float sm_scale, float *out, void *workspace,
                        size_t workspace_bytes, hipStream_t s, bool allow_profile = true) {
    DevLayout L;
    int rc = dev_layout(pool, batch, num_q_heads, L);
    if (rc) return rc;
    const size_t need = (size_t)L.total_words * 4;
    if (!workspace || workspace_bytes < need)
        return fail(ECHO_E_WORKSPACE, "workspace of %zu bytes, need %zu", workspace_bytes, need);
    if (((uintptr_t)workspace & 255u) != 0)
        return fail(ECHO_E_WORKSPACE, "workspace must be 256-byte aligned");
    hipEvent_t *ev = nullptr;
    if (allow_profile) {
        rc = profile_events(&ev);
        if (rc) return rc;
    }
    g_prof.valid = false;
    int32_t *w = (int32_t *)workspace;
    DevPlanArgs d;
    d.block_tables = batch->block_tables;
    d.seq_lens = batch->seq_lens;
    d.q_start = batch->q_start;
    d.row_kind = batch->row_kind;
    d.num_rows = batch->num_rows;
    d.num_tokens = batch->num_tokens;
    d.max_blocks_per_row = batch->max_blocks_per_row;
    d.num_blocks = pool->num_blocks;
    d.max_seq_len = batch->max_seq_len;
    d.split_keys = L.split_keys;
    d.tile_tokens = L.tile_tokens;
    d.slots_per_desc = L.slots_per_desc;
    d.prefill_max_keys = prefill_max_blocks(pool->head_dim) * kBlock;
    d.cap_desc = L.cap_desc;
    d.cap_pdesc = L.cap_pdesc;
    d.cap_merge_rows = L.cap_mrows;
    d.cap_ent = L.cap_ent;
    d.cap_slots = L.cap_slots;
    d.row_info = w + L.off_row_info;
    d.hdr = w;
    d.desc = (WorkDesc *)(w + L.off_desc);
    d.pdesc = (PrefillDesc *)(w + L.off_pdesc);
    d.merge_tok = w + L.off_mtok;
    d.merge_ptr = w + L.off_mptr;
    d.merge_ent = w + L.off_ment;
    hipError_t e;
    if (ev && (e = hipEventRecord(ev[0], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    if ((e = launch_dev_plan(d, s)) != hipSuccess) return hip_fail(e, "device plan launch");
    if (ev && (e = hipEventRecord(ev[1], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    AttnLaunch a;
    a.desc = d.desc;
    a.pdesc = d.pdesc;
    a.merge_tok = d.merge_tok;
    a.merge_ptr = d.merge_ptr;
    a.merge_ent = d.merge_ent;
    a.counts = w;
    a.part_lse = (float *)(w + L.off_lse);
    a.part_o = (float *)(w + L.off_o);
    a.n_desc = L.cap_desc;
    a.n_merge_rows = L.cap_mrows;
    a.n_pdesc_grid = (int32_t)L.cap_pdesc;
    a.head_chunks = L.head_chunks;
    a.heads_per_chunk = L.heads_per_chunk;
    a.waves_per_desc = L.waves_per_desc;
    a.run_log2 = 0;
    a.pf_max_blocks = L.pf_max_blocks;
    return launch_attention(pool, batch, q, num_q_heads, sm_scale, out, a, s, ev);
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
    if (check_attn_args(pool, batch, num_q_heads) != ECHO_OK) return 0;
    if (batch->num_rows == 0) return 256;
    if (!has_mirrors(batch)) {
        DevLayout L;
        if (dev_layout(pool, batch, num_q_heads, L) != ECHO_OK) return 0;
        return (size_t)L.total_words * 4;
    }
    thread_local Plan plan;
    if (plan_for(pool, batch, num_q_heads, plan) != ECHO_OK) return 0;
    return (size_t)plan.layout.total_words * 4;
}

size_t echo_attn_host_workspace_bytes(const echo_kv_pool_t *pool, const echo_batch_t *batch,
                                      int32_t num_q_heads) {
    g_error.clear();
    if (check_attn_args(pool, batch, num_q_heads) != ECHO_OK) return 0;
    if (batch->num_rows == 0 || !has_mirrors(batch)) return 0;
    thread_local Plan plan;
    if (plan_for(pool, batch, num_q_heads, plan) != ECHO_OK) return 0;
    return (size_t)plan.layout.upload_words * 4;
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
                    size_t workspace_bytes, void *host_workspace, size_t host_workspace_bytes,
                    void *stream) {
    g_error.clear();
    int rc = check_attn_args(pool, batch, num_q_heads);
    if (rc) return rc;
    if (batch->num_rows == 0) return ECHO_OK;
    if (!q || !out) return fail(ECHO_E_INVALID, "q / out is NULL");
    if (!(sm_scale > 0.f) || !std::isfinite(sm_scale))
        return fail(ECHO_E_INVALID, "sm_scale must be positive and finite");
    hipStream_t s = (hipStream_t)stream;
    if (!has_mirrors(batch))
        return attn_device_planned(pool, batch, q, num_q_heads, sm_scale, out, workspace,
                                   workspace_bytes, s);

    thread_local Plan plan;
    rc = plan_for(pool, batch, num_q_heads, plan);
    if (rc) return rc;
    const PlanLayout &L = plan.layout;
    int32_t pf_blocks = 0;
    for (const PrefillDesc &d : plan.pdesc)
        pf_blocks = std::max(pf_blocks, (d.key_end + kBlock - 1) / kBlock - d.key_begin / kBlock);
    if (pf_blocks > prefill_max_blocks(pool->head_dim))
        return fail(ECHO_E_UNSUPPORTED, "prefill row of %d blocks exceeds the %d-block limit",
                    pf_blocks, prefill_max_blocks(pool->head_dim));
    const size_t need = (size_t)L.total_words * 4;
    if (!workspace || workspace_bytes < need)
        return fail(ECHO_E_WORKSPACE, "workspace of %zu bytes, need %zu", workspace_bytes, need);
    if (((uintptr_t)workspace & 255u) != 0)
        return fail(ECHO_E_WORKSPACE, "workspace must be 256-byte aligned");
    void *staged = nullptr;
    rc = check_host_workspace(host_workspace, host_workspace_bytes, (size_t)L.upload_words * 4,
                              &staged);
    if (rc) return rc;
    hipEvent_t *ev = nullptr;
    rc = profile_events(&ev);
    if (rc) return rc;
    g_prof.valid = false;
    // every check is done: pack the plan into the host workspace and enqueue
    pack_plan(plan, host_workspace);
    hipError_t e;
    if (ev && (e = hipEventRecord(ev[0], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    if ((e = launch_plan_upload(staged, workspace, L.upload_words, s)) != hipSuccess)
        return hip_fail(e, "plan upload launch");
    if (ev && (e = hipEventRecord(ev[1], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");

    int32_t *w = (int32_t *)workspace;
    AttnLaunch a;
    a.desc = (const WorkDesc *)(w + L.off_desc);
    a.pdesc = (const PrefillDesc *)(w + L.off_pdesc);
    a.tok_list = w + L.off_tok_list;
    a.klim = w + L.off_klim;
    a.merge_tok = w + L.off_merge_tok;
    a.merge_ptr = w + L.off_merge_ptr;
    a.merge_ent = w + L.off_merge_ent;
    a.part_lse = (float *)(w + L.off_part_lse);
    a.part_o = (float *)(w + L.off_part_o);
    a.n_desc = L.n_desc;
    a.n_merge_rows = L.n_merge_rows;
    a.n_pdesc_grid = plan.pdesc_grid;
    a.head_chunks = plan.head_chunks;
    a.heads_per_chunk = plan.heads_per_chunk;
    a.waves_per_desc = plan.waves_per_desc;
    a.run_log2 = run_log2_for(plan.sibling_waves);
    a.pf_max_blocks = pf_blocks;
    return launch_attention(pool, batch, q, num_q_heads, sm_scale, out, a, s, ev);
}

int echo_attn_mixed_static(const echo_kv_pool_t *pool, const echo_batch_t *batch, const void *q,
                           int32_t num_q_heads, float sm_scale, float *out, void *stream) {
    g_error.clear();
    int rc = check_attn_args(pool, batch, num_q_heads);
    if (rc) return rc;
    if (batch->num_rows == 0) return ECHO_OK;
    if (!q || !out) return fail(ECHO_E_INVALID, "q / out is NULL");
    if (!(sm_scale > 0.f) || !std::isfinite(sm_scale))
        return fail(ECHO_E_INVALID, "sm_scale must be positive and finite");
    DevLayout L;
    rc = dev_layout(pool, batch, num_q_heads, L);
    if (rc) return rc;
    const size_t need = (size_t)L.total_words * 4;
    if (need > kScratchBytes)
        return fail(ECHO_E_WORKSPACE,
                    "batch needs %zu bytes of scratch; the static scratch holds %zu (use "
                    "echo_attn_mixed with a workspace)", need, kScratchBytes);
    void *ptr = nullptr;
    hipError_t e = scratch_region(&ptr);
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress (static scratch)");
    return attn_device_planned(pool, batch, q, num_q_heads, sm_scale, out, ptr, kScratchBytes,
                               (hipStream_t)stream, false);
}

}  // extern "C"
