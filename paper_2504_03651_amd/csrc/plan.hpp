// plan.hpp -- work plan of one mixed attention call, built on the host from
// the batch's host mirrors and uploaded into the caller's workspace.
//
// A work item is what one 64-lane wave computes: up to 16 query vectors
// (tokens x query heads of one KV head) against one contiguous key range of
// one row's block table.  Decode rows whose leading blocks are the same
// physical blocks (a prefix group, Section 6 of the paper: prefix reuse via
// automatic prefix caching) are found with a trie over their block ids; each
// shared run of blocks becomes one segment whose keys are read once for the
// query vectors of every row in it.  Long key ranges are cut into splits;
// split and segment results are partial softmax states merged afterwards.
#pragma once
#include <cstddef>
#include <cstdint>
#include <vector>

namespace echo {

constexpr int kBlock = 16;
constexpr int32_t kMaxSeqLen = 1 << 30;   // longest row accepted (key positions stay far from int overflow)
constexpr int kWaveQueries = 16;   // query vectors per wave (MFMA N dimension)
constexpr int kWavesPerGroup = 4;  // waves per workgroup

// flags in WorkDesc::shape
// The descriptor's keys are also read by other waves (sibling query slices of
// a shared segment, or other head chunks of the same KV head): load them
// through the L2 so the siblings hit there, instead of streaming them.
constexpr int32_t kItemShared = 1 << 16;

// One key range of one block table against one slice of query tokens.  On
// the GPU it expands into num_kv_heads * head_chunks waves (a head chunk is
// up to 16 query heads of one KV head), so the host never enumerates heads.
struct WorkDesc {      // 32 bytes
    int32_t tok_off;   // offset of the slice's first token in the plan's token list
    int32_t shape;     // nt | flags: nt tokens in the slice
    int32_t bt_row;    // row whose block table supplies the block ids
    int32_t key_begin; // first key position, a multiple of 16
    int32_t key_end;   // one past the last key position
    int32_t part;      // first partial slot, or -1: write `out` directly
    int32_t tok1;      // nt == 1: the slice's token (saves the token-list load)
    int32_t klim1;     // nt == 1: keys visible to that token
};
static_assert(sizeof(WorkDesc) == 32, "descriptor layout");

// One tile of a prefill chunk: up to kPrefillQueries query vectors (ntok
// consecutive tokens x all query heads of one KV head) for one workgroup.  On
// the GPU it expands over the KV heads.
#ifndef ECHO_PF_WAVES
#define ECHO_PF_WAVES 8
#endif
constexpr int kPrefillQueries = 32 * ECHO_PF_WAVES;
struct PrefillDesc {   // 32 bytes
    int32_t row;
    int32_t tok0;      // first token of the tile
    int32_t ntok;      // tokens in the tile
    int32_t key_end;   // one past the last key of this piece of the tile's keys
    int32_t key_begin; // first key of the piece, a multiple of the 64-key tile
    int32_t part;      // first partial slot of the piece, or -1: write `out`
    int32_t kfull;     // keys every token of the tile sees (unmasked below)
    int32_t next;      // 1 + index of a descriptor the same workgroup runs
                       // after this one, or 0
};
static_assert(sizeof(PrefillDesc) == 32, "prefill descriptor layout");
constexpr int kPrefillTileKeys = 64;      // keys per LDS tile of the prefill kernel
constexpr int kPrefillMinPieceTiles = 8;  // shortest piece a long key range is cut into
constexpr int kPrefillMinChainTiles = 2;  // fewest 64-key tiles moved to a chained piece
// Decode key ranges are cut into pieces of about kSplitBytes of K+V per KV
// head: 48 blocks of bf16 at head_dim 128, 96 of e4m3, whose waves move half
// the bytes per block (a sweep of 16-128 blocks on the decode-only, mixed and
// e4m3 batches).
constexpr int64_t kSplitBytes = 384 * 1024;
constexpr int kMinSplitBlocks = 8;        // shortest decode piece on small batches
constexpr int kSplitTargetUnits = 2048;   // decode units below which pieces shrink
#ifndef ECHO_EQ_GENS
#define ECHO_EQ_GENS 3
#endif
// Decode launches of at most this many generations of resident waves (3 per
// SIMD, 12 per CU) cut each key range into pieces of equal length rather
// than full pieces and a remainder: with few generations the longest waves of
// the last one end the kernel, and equal pieces shorten them; with more, the
// short remainders fill the slots that the long pieces leave
// (measured on MI355X: mixed batch, 1.2 generations, decode 3.6% faster;
// decode-only and e4m3 batches, 4.1 and 3.4 generations, 3-4% slower)
constexpr int kEqualPieceGenerations = ECHO_EQ_GENS;
constexpr int kDecodeWavesPerCu = 12;
#ifndef ECHO_ONE_GEN_STRETCH
#define ECHO_ONE_GEN_STRETCH 4
#endif
// Decode pieces may grow up to this many times the default length when that
// lets the whole launch fit one generation of resident waves (measured on
// MI355X: the long-context batch goes from 2.5 generations at 48 blocks to
// one at 128, decode 0.442 -> 0.386 ms; batches that cannot get there keep
// the default)
constexpr int kOneGenerationStretch = ECHO_ONE_GEN_STRETCH;

// Wave w of the attention grid handles descriptor w / (Hkv * head_chunks),
// KV head (w % (Hkv * head_chunks)) / head_chunks and head chunk
// w % head_chunks; its partial slots start at
// part + (w % (Hkv * head_chunks)) * nt * heads_per_chunk.

// Offsets (in 4-byte words from the start of the workspace) of each region.
struct PlanLayout {
    int64_t n_desc = 0;
    int64_t n_tok_list = 0;
    int64_t n_tokens = 0;
    int64_t n_merge_rows = 0;
    int64_t n_merge_entries = 0;
    int64_t n_slots = 0;
    int32_t head_dim = 0;
    int64_t n_pdesc = 0;
    int64_t off_desc = 0;       // WorkDesc[n_desc]
    int64_t off_pdesc = 0;      // PrefillDesc[n_pdesc]
    int64_t off_tok_list = 0;   // int32[n_tok_list]
    int64_t off_klim = 0;       // int32[n_tokens]: keys visible to each token
    int64_t off_merge_tok = 0;  // int32[n_merge_rows]: the row's token
    int64_t off_merge_ptr = 0;  // int32[n_merge_rows + 1]
    int64_t off_merge_ent = 0;  // int32[2 * n_merge_entries]: (first slot, nt | i << 10)
    int64_t upload_words = 0;   // everything above is uploaded
    int64_t off_part_lse = 0;   // float[n_slots]
    int64_t off_part_o = 0;     // float[n_slots][head_dim]
    int64_t total_words = 0;
};

struct PlanStats {
    int64_t decode_items = 0, prefill_items = 0, shared_segments = 0;
    int64_t logical_kv_tokens = 0, causal_pairs = 0;
    int64_t decode_kv_tokens = 0, prefill_causal_pairs = 0;
};

struct HostBatch {
    int32_t num_rows, mbr, num_tokens, max_q_len, max_seq_len;
    const int32_t *bt, *seq_lens, *q_start;
    const uint8_t *kind;
};

struct PlanOptions {
    int split_blocks = 48;  // key blocks per decode split (set from kSplitBytes)
    int num_cus = 256;      // compute units: prefill key ranges are cut into
                            // pieces when workgroups would fill at most half of them
};

// Host plan under construction (reused between calls on the same thread).
struct Plan {
    std::vector<WorkDesc> desc, desc_sorted;
    std::vector<PrefillDesc> pdesc, pdesc_split;
    int32_t pdesc_grid = 0;       // leading descriptors of pdesc that get workgroups
    std::vector<int32_t> bounds;
    int32_t prefill_tokens_per_tile = 1;
    std::vector<int32_t> tok_list, klim, merge_tok, merge_ptr, merge_ent;
    // scratch
    std::vector<int32_t> nro, rows, tail_start, seg_rows, cnt, moff, cursor, bucket, cuts, takers, ctail;
    PlanLayout layout;
    PlanStats stats;
    int32_t waves_per_desc = 1;   // num_kv_heads * head_chunks
    int32_t sibling_waves = 0;    // most decode waves that read one shared key range
    int32_t head_chunks = 1;
    int32_t heads_per_chunk = 1;  // min(G, 16)
};

// Builds the plan for a validated batch.  Returns 0 or an echo_status_t.
int build_plan(const HostBatch &b, int32_t num_kv_heads, int32_t num_q_heads,
               int32_t head_dim, const PlanOptions &opt, Plan &plan);

// Serialises the uploaded regions of `plan` into `dst` (layout.upload_words
// words).
void pack_plan(const Plan &plan, void *dst);

}  // namespace echo
