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
};

struct PrefillArgs {
    const PrefillDesc *pdesc;
    int32_t n_pdesc;                // descriptors that get workgroups (chained ones follow)
    int32_t n_logical;              // n_pdesc * num_kv_heads
    int32_t per_xcd;                // logical tiles per XCD slot
    int32_t group;                  // Hq / Hkv (<= 128)
    const int32_t *klim;
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
    int32_t num_q_heads, head_chunks, heads_per_chunk, group;
    const int32_t *merge_tok, *merge_ptr;
    const int32_t *merge_ent;       // per entry: first slot of its descriptor, nt | i << 10
    const float *part_o, *part_lse;
    float *out;
};

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
