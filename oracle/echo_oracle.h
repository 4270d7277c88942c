/*
 * echo_oracle.h -- plain fp64 CPU reference for one mixed serving iteration
 * over a paged KV cache.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The product path never
 * calls it, and it shares no code with the HIP library.
 *
 * What it computes (Echo, Section 2.1 "Prefill and decode" and "Chunked
 * prefills"; Section 4.2 on fixed-size KV blocks; Section 6 on prefix reuse):
 *   append  -- every new K/V vector goes into the slot of the block its
 *              position falls in, through the row's block table;
 *   attend  -- each new token of a row attends causally to every cached and
 *              new token of that row at or before its own position;
 *   copy    -- whole blocks are duplicated byte for byte (copy-on-write).
 * The paper prints no attention formula; the oracle uses textbook scaled
 * dot-product attention with a causal mask aligned so that the query at
 * position p sees keys 0..p.
 *
 * Pool layout (shared with the library as an interface, not as code):
 *   K codes [num_blocks][num_kv_heads][16][head_dim]
 *   V codes [num_blocks][num_kv_heads][head_dim][16]   (block-transposed)
 *   codes are bf16 bit patterns (uint16) or OCP e4m3fn bytes (uint8);
 *   e4m3 pools carry fp32 scales [num_blocks][num_kv_heads] for K and for V.
 */
#ifndef ECHO_ORACLE_H
#define ECHO_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    void *k;            /* K codes, layout above */
    void *v;            /* V codes, layout above */
    float *k_scale;     /* [num_blocks][num_kv_heads], e4m3 only */
    float *v_scale;
    int32_t num_blocks;
    int32_t num_kv_heads;
    int32_t head_dim;
    int32_t kv_fp8;     /* 0: bf16 codes, 1: e4m3 codes */
} orc_pool;

typedef struct {
    int32_t num_rows;
    int32_t max_blocks_per_row;
    const int32_t *block_tables;   /* [num_rows][max_blocks_per_row] */
    const int32_t *seq_lens;       /* [num_rows], context + new tokens */
    const int32_t *q_start;        /* [num_rows + 1] */
    const uint8_t *row_kind;       /* [num_rows], 0 decode, 1 prefill */
} orc_batch;

/* Scatter new K/V [T][Hkv][D] (bf16 bits) into the pool.  e4m3 pools: a
 * block whose slot 0 is written by this call gets scale fp32(amax/448) over
 * the values written into it (1 when amax is 0); other blocks keep theirs;
 * codes are round-to-nearest-even, saturated to +-448, of fp32(x/scale).
 * Returns 0, or -1 on malformed metadata. */
int orc_kv_append(const orc_pool *pool, const orc_batch *batch,
                  const uint16_t *k_new, const uint16_t *v_new);

/* Copy K, V (and scales) of block src to block dst for each (src, dst) pair,
 * in list order.  Returns 0, or -1 on an out-of-range id. */
int orc_block_copy(const orc_pool *pool, const int32_t *pairs, int32_t n_pairs);

/* Causal attention of the iteration's new tokens.  q is [T][Hq][D] bf16
 * bits.  sel lists query indices t*Hq + h to evaluate (NULL: all T*Hq in
 * order); out receives [n][D] doubles.  Query head h reads KV head
 * h / (Hq / Hkv).  Returns 0, or -1 on malformed input. */
int orc_attention(const orc_pool *pool, const orc_batch *batch, const uint16_t *q,
                  int32_t num_q_heads, float sm_scale, const int32_t *sel, int32_t n_sel,
                  double *out, int32_t n_threads);

/* Codec helpers, exported so that tests can pin them on their own. */
double orc_bf16_value(uint16_t bits);
double orc_e4m3_value(uint8_t code);
uint8_t orc_e4m3_encode(float x);
float orc_e4m3_fresh_scale(float amax);

#ifdef __cplusplus
}
#endif
#endif
