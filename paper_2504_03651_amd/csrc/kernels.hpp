// kernels.hpp -- argument blocks and launchers of the gfx950 kernels.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "plan.hpp"

namespace echo {

struct AppendArgs {
    void *k, *v;
    float *k_scale, *v_scale;
    const uint16_t *k_new, *v_new;  // [T][Hkv][D] bf16 bits
    const int32_t *block_tables, *seq_lens, *q_start;
    int32_t num_rows, num_blocks, num_kv_heads, max_blocks_per_row;
    int64_t n_units;                // upper bound of (row, written block, head) units
    int32_t blocks_per_row;         // > 0: direct form, written blocks per row bound
};

struct BlockCopyArgs {
    void *k, *v;
    float *k_scale, *v_scale;       // NULL unless e4m3
    const int32_t *pairs;
    int32_t n_pairs, num_blocks, num_kv_heads;
    int64_t block_bytes;            // bytes of one block of K (same for V)
    int32_t chunks;                 // 16 KiB chunks per block
};

struct AttnArgs {
    const WorkDesc *desc;
    int64_t n_waves;                // n_desc * waves_per_desc
    int32_t waves_per_desc;         // num_kv_heads * head_chunks
    int32_t head_chunks, heads_per_chunk, group;  // group = Hq / Hkv
    const int32_t *tok_list, *klim;
    const uint16_t *q;              // [T][Hq][D] bf16 bits
    int32_t num_q_heads, num_kv_heads;
    const void *k, *v;
    const float *k_scale, *v_scale;
    const int32_t *block_tables;
    int32_t max_blocks_per_row;
    float scale_log2;               // sm_scale * log2(e)
    float *out, *part_o, *part_lse;
    int32_t run_log2;               // XCD run length: the caller's minimum, set by the launcher
    const int32_t *counts;          // device-built plan: its header (word 0 = descriptors);
                                    // NULL when n_waves is exact
};

struct PrefillArgs {
    const PrefillDesc *pdesc;
    int32_t n_pdesc;                // descriptors that get workgroups (chained ones follow);
                                    // with `counts`, the capacity of the descriptor region
    int32_t n_logical;              // n_pdesc * num_kv_heads
    int32_t per_xcd;                // logical tiles per XCD slot
    int32_t group;                  // Hq / Hkv (<= 128)
    const int32_t *seq_lens, *q_start;   // a token's visible keys follow from its row's
    const int32_t *counts;          // device-built plan: its header (word 1 = descriptors)
    const uint16_t *q;
    int32_t num_q_heads, num_kv_heads;
    const void *k, *v;
    const float *k_scale, *v_scale;
    const int32_t *block_tables;
    int32_t max_blocks_per_row;
    float scale_log2;
    float *out;
    int32_t max_blocks;             // most blocks any piece reads (ids staged in LDS)
    int32_t head_chunks, heads_per_chunk;   // partial-slot layout shared with decode
    float *part_o, *part_lse;       // partial results of pieces of split key ranges
};

struct MergeArgs {
    int64_t n_waves;                // merged rows * ceil(Hq / 4)
    const int32_t *counts;          // device-built plan: its header (word 2 = merged rows)
    int32_t num_q_heads, head_chunks, heads_per_chunk, group;
    const int32_t *merge_tok, *merge_ptr;
    const int32_t *merge_ent;       // per entry: first slot of its descriptor, nt | i << 10
    const float *part_o, *part_lse;
    float *out;
};

// The plan of a batch without host mirrors, built on the device into the
// workspace: no prefix grouping; decode rows cut into pieces of split_keys,
// prefill rows into tiles of tile_tokens tokens.  Regions have capacities
// from the host's scalar bounds; the header holds the counts the attention
// kernels read (DevPlanHeader).
struct DevPlanArgs {
    const int32_t *block_tables, *seq_lens, *q_start;
    const uint8_t *row_kind;
    int32_t num_rows, num_tokens, max_blocks_per_row, num_blocks, max_seq_len;
    int32_t split_keys;             // keys per decode piece (multiple of 16)
    int32_t tile_tokens;            // tokens per prefill tile
    int32_t slots_per_desc;         // partial slots per decode piece (one token)
    int32_t prefill_max_keys;       // longest key range the prefill kernel can stage
    int64_t cap_desc, cap_pdesc, cap_merge_rows, cap_ent, cap_slots;
    int32_t *row_info;              // [num_rows] scratch: decode pieces | prefill tiles << 16, or -1
    int32_t *hdr;                   // DevPlanHeader words
    WorkDesc *desc;
    PrefillDesc *pdesc;
    int32_t *merge_tok, *merge_ptr, *merge_ent;
};
// words of the header of a device-built plan
enum DevPlanHeader {
    kHdrDesc = 0,       // decode descriptors
    kHdrPdesc = 1,      // prefill descriptors
    kHdrMergeRows = 2,  // merged tokens
    kHdrSlots = 3,      // partial slots used
    kHdrBadRows = 4,    // rows skipped because their metadata is inconsistent
    kHdrWords = 64
};
hipError_t launch_dev_plan(const DevPlanArgs &a, hipStream_t s);

// Static device scratch of echo_attn_mixed_static (a file-scope __device__
// array in kernels.hip): its size, and this device's address of it.
constexpr size_t kScratchBytes = (size_t)32 << 20;
hipError_t scratch_region(void **ptr);

hipError_t launch_append(const AppendArgs &a, int head_dim, bool fp8, hipStream_t s);
hipError_t launch_block_copy(const BlockCopyArgs &a, hipStream_t s);
// Copies `words` 32-bit words from device-visible pinned host memory to dst.
hipError_t launch_plan_upload(const void *src, void *dst, int64_t words, hipStream_t s);
// Largest number of block ids the prefill kernel can stage for one row.
int prefill_max_blocks(int head_dim);

// Attention launchers; each returns hipSuccess without launching when it
// has no work.  The merge reads the partial results of both others, so it
// runs after them.
hipError_t launch_prefill(const PrefillArgs &p, int head_dim, bool fp8, hipStream_t s);
hipError_t launch_decode(const AttnArgs &a, int head_dim, bool fp8, hipStream_t s);
hipError_t launch_merge(const MergeArgs &m, int head_dim, hipStream_t s);

}  // namespace echo
