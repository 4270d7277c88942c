/*
 * echo.h -- C ABI of the MI355X (gfx950) mixed paged-attention iteration.
 *
 * One serving iteration of the Echo paper (arXiv 2504.03651) over a paged KV
 * cache: the new keys/values of every scheduled token are appended into
 * fixed-size cache blocks, then the new tokens of chunked-prefill rows and
 * decode rows attend causally to their row's cached and new tokens through
 * per-row block tables, where rows of a prefix group alias the same blocks
 * (Section 2.1 "Prefill and decode" and "Chunked prefills"; Section 4.2, KV
 * cache divided into fixed-size blocks; Section 6, prefix reuse by automatic
 * prefix caching).  Block copy duplicates whole blocks (copy-on-write).
 *
 * Conventions shared by every entry point
 *   - Pointers named h_* are host memory; every other pointer is device
 *     memory on the current HIP device.  All buffers belong to the caller and
 *     must outlive the work enqueued on `stream` (a hipStream_t, NULL for the
 *     default stream).  Calls return after enqueueing; they do not
 *     synchronise and allocate no device or pinned host memory; nothing a
 *     call leaves behind affects a later call (per-thread host buffers for
 *     validation and planning are reused, and echo_profile's opt-in events
 *     are kept per thread).
 *   - Validation happens before anything is enqueued: a call that returns an
 *     error has enqueued nothing and changed nothing.
 *   - Return values are echo_status_t codes (0 on success, negative on error);
 *     echo_status_string() names a code and echo_last_error() gives the
 *     calling thread's most recent error detail.
 *   - Nothing throws across the ABI.  Calls from several host threads are
 *     safe; work enqueued on the same stream runs in call order.
 *
 * Pool layout (block_size 16; head_dim 64 or 128):
 *   K codes  [num_blocks][num_kv_heads][16][head_dim]
 *   V codes  [num_blocks][num_kv_heads][head_dim][16]   (block-transposed)
 *   bf16 pools store bf16; e4m3 pools store OCP e4m3fn bytes plus fp32 scales
 *   k_scale / v_scale [num_blocks][num_kv_heads]: the value of a code is
 *   e4m3(code) * scale of its (block, head).  Chunked-prefill attention over
 *   an e4m3 pool carries V values in fp16, so they must lie within +-65504
 *   (finite results are not guaranteed beyond).
 * Token-major tensors: q [T][Hq][head_dim] bf16, k_new / v_new
 *   [T][Hkv][head_dim] bf16, out [T][Hq][head_dim] fp32, where token t of row
 *   r is q_start[r] + i for its i-th new token, at position
 *   seq_lens[r] - (q_start[r+1] - q_start[r]) + i of the row.
 */
#ifndef ECHO_H
#define ECHO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    ECHO_OK = 0,
    ECHO_E_INVALID = -1,      /* malformed argument or metadata */
    ECHO_E_RANGE = -2,        /* a block id outside [0, num_blocks) */
    ECHO_E_ALIAS_WRITE = -3,  /* an append would write a block another row also reads */
    ECHO_E_WORKSPACE = -4,    /* workspace missing or smaller than required */
    ECHO_E_UNSUPPORTED = -5,  /* head_dim, block_size or dtype not supported */
    ECHO_E_HIP = -6,          /* the HIP runtime reported an error */
    ECHO_E_NOSPACE = -7       /* KV block manager: not enough free blocks, or
                                 the limit for offline sequences (echo_kvm.h) */
} echo_status_t;

typedef enum { ECHO_KV_BF16 = 0, ECHO_KV_FP8_E4M3 = 1 } echo_kv_dtype_t;
typedef enum { ECHO_ROW_DECODE = 0, ECHO_ROW_PREFILL = 1 } echo_row_kind_t;

/* The paged KV cache of one layer (Section 4.2: fixed-size blocks allocated
 * non-contiguously).  Device memory owned by the caller. */
typedef struct {
    void *k;                  /* K codes, layout above */
    void *v;                  /* V codes, layout above */
    float *k_scale;           /* e4m3 only: [num_blocks][num_kv_heads]; else NULL */
    float *v_scale;
    int32_t num_blocks;
    int32_t num_kv_heads;
    int32_t head_dim;         /* 64 or 128 */
    int32_t block_size;       /* must be 16 */
    int32_t dtype;            /* echo_kv_dtype_t */
} echo_kv_pool_t;

/* The rows of one iteration (Section 2.1: decode batching and chunked
 * prefill in one batch).  Device arrays, plus optional host mirrors with the
 * same contents.  With the mirrors, validation is complete (block ranges,
 * aliased writes) and echo_attn_mixed plans on the host, grouping the rows
 * that share prefix blocks (Section 6) so that those blocks are read once.
 * Without them only the scalar fields are checked on the host and
 * echo_attn_mixed builds a plan without prefix grouping on the device. */
typedef struct {
    int32_t num_rows;             /* B */
    int32_t max_blocks_per_row;   /* row stride of block_tables */
    int32_t num_tokens;           /* T = q_start[B] */
    int32_t max_q_len;            /* >= every row's new-token count */
    int32_t max_seq_len;          /* >= every seq_lens[r]; at most 2^30 (else ECHO_E_UNSUPPORTED) */
    const int32_t *block_tables;  /* [B][max_blocks_per_row]; entry j holds positions
                                     16j..16j+15; entries at or past ceil(L/16) unused */
    const int32_t *seq_lens;      /* [B] L_r: cached tokens + this call's new tokens */
    const int32_t *q_start;       /* [B+1] prefix sums of new-token counts, q_start[0]=0 */
    const uint8_t *row_kind;      /* [B] echo_row_kind_t; decode rows add exactly one token */
    const int32_t *h_block_tables;  /* optional host mirrors (all four or none) */
    const int32_t *h_seq_lens;
    const int32_t *h_q_start;
    const uint8_t *h_row_kind;
} echo_batch_t;

/* Append (Section 2.1: decode appends the new token's KV state to the cache;
 * prefill generates and caches it).  For token i of row r at position p,
 * writes k_new[t] / v_new[t] (bf16 [T][Hkv][head_dim]) into slot p % 16 of
 * block block_tables[r][p / 16].  e4m3 pools: a block whose slot 0 is written
 * by this call gets, per KV head, scale fp32(amax / 448) over the values this
 * call writes into it (1 when amax is 0); other blocks keep their scale; each
 * code is the round-to-nearest-even, saturating e4m3 encoding of the
 * correctly rounded fp32 quotient value / scale.  Every block written must be
 * referenced by exactly one row (copy-on-write first with echo_block_copy);
 * with host mirrors a violation returns ECHO_E_ALIAS_WRITE.  Without mirrors
 * only scalar checks run and the caller guarantees the metadata. */
int echo_kv_append(const echo_kv_pool_t *pool, const echo_batch_t *batch, const void *k_new,
                   const void *v_new, void *stream);

/* Mixed attention (Section 2.1: prefill chunks and decode rows batched in
 * one iteration; Section 6: rows of a prefix group reuse the same cached
 * blocks).  For every new token t of row r at position p and query head h,
 *   out[t][h] = sum_{j<=p} softmax_j(sm_scale * q[t][h] . K_r[j][g]) V_r[j][g],
 * with g = h / (num_q_heads / num_kv_heads) and K_r/V_r the row's logical
 * sequence read through its block table.  Run echo_kv_append for the same
 * iteration first: attention reads the new tokens from the pool.
 * q: bf16 [T][num_q_heads][head_dim]; out: fp32 [T][num_q_heads][head_dim].
 * sm_scale must be positive and finite (ECHO_E_INVALID otherwise).
 * workspace: device scratch of at least echo_attn_workspace_bytes() bytes,
 * 256-byte aligned, not used by another call until this call's work on
 * `stream` has completed (calls on one stream may share it).
 *
 * Two planning modes, chosen by the host mirrors:
 *   - with mirrors, the work plan is built on the host: decode rows whose
 *     leading full blocks are the same physical blocks are grouped and those
 *     blocks are read once per KV head for all of them; long key ranges are
 *     split and prefill tiles balanced.  The plan is packed into
 *     host_workspace -- pinned host memory the device reads coherently
 *     (hipHostMalloc with hipHostMallocMapped | hipHostMallocCoherent), at
 *     least echo_attn_host_workspace_bytes() bytes, 16-byte aligned -- and
 *     copied into `workspace` by a kernel on `stream`.  The call does not
 *     wait for that copy: the caller must not change or reuse host_workspace
 *     until this call's work on `stream` has run past it (for example, wait
 *     on an event recorded after the call, or rotate several buffers).
 *     Memory that is not pinned host memory returns ECHO_E_WORKSPACE;
 *   - without mirrors, host_workspace is ignored (may be NULL) and two small
 *     kernels build the plan in `workspace` from the device metadata: no
 *     prefix grouping (shared blocks are read once per row), decode rows cut
 *     into equal key pieces, prefill rows into tiles, grids sized from the
 *     scalar fields.  The results are the same within rounding.  Rows whose
 *     metadata is inconsistent (the checks the mirrors would have run) get
 *     no work and leave their outputs unchanged; nothing is read outside the
 *     buffers described by the scalar fields.
 * All checks run before anything is enqueued; a HIP launch failure (ECHO_E_HIP)
 * can leave the kernels launched before it enqueued. */
int echo_attn_mixed(const echo_kv_pool_t *pool, const echo_batch_t *batch, const void *q,
                    int32_t num_q_heads, float sm_scale, float *out, void *workspace,
                    size_t workspace_bytes, void *host_workspace, size_t host_workspace_bytes,
                    void *stream);

/* Device workspace bytes echo_attn_mixed needs for this batch (the planning
 * mode follows from the host mirrors; without them the size is a bound from
 * the scalar fields), or 0 if the arguments are invalid. */
size_t echo_attn_workspace_bytes(const echo_kv_pool_t *pool, const echo_batch_t *batch,
                                 int32_t num_q_heads);

/* Pinned host workspace bytes echo_attn_mixed needs (the packed plan): 0
 * without host mirrors, or when the arguments are invalid. */
size_t echo_attn_host_workspace_bytes(const echo_kv_pool_t *pool, const echo_batch_t *batch,
                                      int32_t num_q_heads);

/* Mixed attention that allocates nothing and takes no workspace, for
 * callers that cannot allocate device memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation.  Same arguments,
 * results and checks as echo_attn_mixed, always with the plan built on the
 * device (host mirrors, when given, are used for validation only).  The plan
 * and the partial results live in a static device array of the library
 * (32 MiB, held by each GPU the library runs on until the process ends);
 * a batch whose device-built plan needs more returns ECHO_E_WORKSPACE before
 * anything is enqueued.  Every call on a GPU uses that GPU's one array and
 * leaves its contents behind; every word a call reads is written earlier in
 * the same call, so nothing needs clearing, but calls that overlap on one
 * GPU (other streams, other host threads) race and must be serialised by
 * the caller. */
int echo_attn_mixed_static(const echo_kv_pool_t *pool, const echo_batch_t *batch, const void *q,
                           int32_t num_q_heads, float sm_scale, float *out, void *stream);

/* Block copy (copy-on-write of blocks that prefix-sharing rows alias; the
 * paper's automatic prefix caching, Section 6, implies it).  For each pair
 * (src, dst) of pairs (device int32 [n][2]) copies K, V and, for e4m3 pools,
 * both scales of block src into block dst, byte for byte.  Requires src !=
 * dst, distinct dst, and no dst that is also a src (ECHO_E_INVALID, checked
 * when the host mirror h_pairs is given; ids are range-checked then too, and
 * on the device always, where out-of-range pairs are skipped). */
int echo_block_copy(const echo_kv_pool_t *pool, const int32_t *pairs, int32_t n_pairs,
                    const int32_t *h_pairs, void *stream);

/* What the planner made of a batch: a host-only call (no GPU work). */
typedef struct {
    int64_t work_items;         /* decode_items + prefill_items */
    int64_t decode_items;       /* decode waves: (key range, query slice, KV head) */
    int64_t prefill_items;      /* prefill workgroups: (token tile, KV head) */
    int64_t shared_segments;    /* block runs read once for several decode rows */
    int64_t partial_slots;      /* split results merged after the main pass */
    int64_t merged_queries;     /* (token, head) pairs that need the merge */
    int64_t unique_kv_tokens;   /* per KV head: distinct (block, slot) pairs read */
    int64_t logical_kv_tokens;  /* per KV head: sum over rows of seq_lens */
    int64_t causal_pairs;       /* per query head: sum over queries of visible keys */
    int64_t decode_kv_tokens;   /* per KV head: keys the decode items read (shared runs once) */
    int64_t prefill_causal_pairs; /* per query head: causal_pairs of the prefill rows only */
    int64_t workspace_bytes;
} echo_plan_stats_t;

/* Validates the batch (host mirrors required) and fills *stats. */
int echo_attn_plan_stats(const echo_kv_pool_t *pool, const echo_batch_t *batch,
                         int32_t num_q_heads, echo_plan_stats_t *stats);

/* The work plan echo_attn_mixed uploads for a batch (host-only; for tests
 * and tools that inspect plans).  Regions are in 32-bit words from the start
 * of the workspace; everything below upload_words is the packed plan:
 *   desc      [n_desc][8]   decode work: tok_off, nt | 1 << 16 when other
 *                           waves read the same keys, bt_row, key_begin,
 *                           key_end, part (first partial slot or -1), and
 *                           for nt == 1 the token and its key limit (else -1, 0)
 *   pdesc     [n_pdesc][8]  prefill work: row, tok0, ntok, key_end,
 *                           key_begin, part, kfull (keys every token of the
 *                           tile sees), next (1 + index of a descriptor the
 *                           same workgroup runs afterwards, or 0; descriptors
 *                           named this way come last and get no workgroup
 *                           of their own)
 *   tok_list  [n_tok_list]  tokens of the decode slices
 *   klim      [n_tokens]    keys visible to each token
 *   merge_tok [n_merge_rows], merge_ptr [n_merge_rows + 1]
 *   merge_ent [n_merge_entries][2]  (first slot, nt | i << 10): query i of a
 *                           slice of nt tokens; the (token, head h) result of
 *                           an entry sits in slot first + (h / G * head_chunks
 *                           + (h % G) / 16) * nt * heads_per_chunk + i * nh
 *                           + (h % G) % 16, nh = min(heads_per_chunk, G - 16 *
 *                           ((h % G) / 16)), G = Hq / Hkv
 * Decode descriptor d expands to waves (d, KV head k, head chunk c), whose
 * partial slots start at part + (k * head_chunks + c) * nt * heads_per_chunk. */
typedef struct {
    int64_t n_desc, n_pdesc, n_tok_list, n_tokens, n_merge_rows, n_merge_entries, n_slots;
    int64_t off_desc, off_pdesc, off_tok_list, off_klim, off_merge_tok, off_merge_ptr,
        off_merge_ent;
    int64_t upload_words, off_part_lse, off_part_o, total_words;
    int32_t head_chunks, heads_per_chunk;
} echo_plan_layout_t;

/* Fills *layout and, when words is not NULL, packs the plan into the host
 * buffer words (at least layout->upload_words * 4 bytes, else
 * ECHO_E_WORKSPACE).  Validates like echo_attn_mixed; no GPU work. */
int echo_attn_plan_pack(const echo_kv_pool_t *pool, const echo_batch_t *batch,
                        int32_t num_q_heads, echo_plan_layout_t *layout, void *words,
                        size_t bytes);

/* Host-only validation of pool and batch as echo_kv_append (for_append = 1)
 * or echo_attn_mixed (for_append = 0) would do it; no GPU work. */
int echo_validate(const echo_kv_pool_t *pool, const echo_batch_t *batch, int32_t for_append);

/* Per-kernel GPU time of the calling thread's most recent echo_attn_mixed
 * call, measured with HIP events recorded on that call's stream around the
 * plan upload and each kernel launch.  Recording is off unless enabled with
 * echo_profile(1) on the same thread; kernels not launched report 0. */
typedef struct {
    float upload_ms;    /* plan upload from the host workspace, or the two device
                           planning kernels when there are no host mirrors */
    float prefill_ms;   /* prefill_kernel: chunked-prefill tiles */
    float decode_ms;    /* attn_kernel: decode split-KV / shared-prefix items */
    float merge_ms;     /* merge_kernel: log-sum-exp merge of partial results */
} echo_attn_timing_t;

/* Turns event recording on (1) or off (0) for this thread; returns the
 * previous setting.  Recording adds a few events per call, nothing else. */
int echo_profile(int enable);

/* Waits for the last profiled call's events and fills *timing. */
int echo_attn_timing(echo_attn_timing_t *timing);

/* Static name of a status code. */
const char *echo_status_string(int status);

/* The calling thread's most recent error detail ("" when none). */
const char *echo_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* ECHO_H */
