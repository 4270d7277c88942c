/*
 * echo_layer.h -- one decoder layer around the mixed iteration (GPU).
 *
 * A LLaMA-style layer whose attention is the iteration of echo.h, so that the
 * attention's share of a serving iteration can be measured in context
 * (Section 7 runs a LLaMA-3.1-8B-class model; the paper's time equations of
 * Section 5.2 split each iteration into attention, quadratic in the sequence
 * length, and the layers that are linear in it):
 *
 *   y  = RMSNorm(x) * attn_norm                       bf16
 *   qkv = y W_qkv^T                                    bf16 (hipBLASLt, fp32 accumulate)
 *   q, k, v = split(qkv); q, k = RoPE(q, k, position) bf16
 *   echo_kv_append(k, v); o = echo_attn_mixed(q)       fp32 -> bf16
 *   h  = x + o W_o^T                                   bf16
 *   y2 = RMSNorm(h) * mlp_norm
 *   x' = h + (SiLU(y2 W_gate^T) * (y2 W_up^T)) W_down^T
 *
 * RoPE rotates each head's pair (i, i + D/2) by position * theta^(-2i/D)
 * (angles in fp64).  The position of the i-th new token of row r is
 * seq_lens[r] - q_len[r] + i, as for the append.  Row-major bf16 weights in
 * device memory, out_features x in_features: w_qkv [(Hq + 2 Hkv) D][H] (query
 * rows, then key rows, then value rows), w_o [H][Hq D], w_gate_up [2 I][H]
 * (gate rows, then up rows), w_down [H][I]; norms [H].
 *
 * The pool and batch follow echo.h.  hidden [T][H] bf16 is read and
 * overwritten with the layer's output; all other device buffers come from the
 * caller's workspace (echo_layer_workspace_bytes, 256-byte aligned), and the
 * attention's plan goes through host_workspace exactly as in
 * echo_attn_mixed (echo_attn_host_workspace_bytes; not used, and may be
 * NULL, without host mirrors).
 * The GEMMs run through hipBLASLt on `stream`, with a handle per host thread
 * and device created on first use.
 */
#ifndef ECHO_LAYER_H
#define ECHO_LAYER_H

#include <stddef.h>
#include <stdint.h>

#include "echo.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t hidden;        /* H, a multiple of 8 */
    int32_t num_q_heads, num_kv_heads, head_dim;
    int32_t intermediate;  /* I, a multiple of 8 */
    float rope_theta;      /* e.g. 500000 */
    float rms_eps;         /* e.g. 1e-5 */
    const void *attn_norm, *w_qkv, *w_o, *mlp_norm, *w_gate_up, *w_down;
} echo_layer_t;

/* Workspace bytes that echo_layer_forward needs for this batch (0 and an
 * error status via echo_last_error() when the arguments are invalid). */
size_t echo_layer_workspace_bytes(const echo_layer_t *layer, const echo_kv_pool_t *pool,
                                  const echo_batch_t *batch);

/* One forward step of the layer for the batch's new tokens (see above).  The
 * pool receives the new tokens' K/V.  Arguments, pool and batch are validated
 * before anything is enqueued, as in echo.h; a HIP or hipBLASLt failure
 * afterwards (ECHO_E_HIP) can leave the stages before it enqueued, with
 * hidden and the pool then undefined. */
int echo_layer_forward(const echo_layer_t *layer, const echo_kv_pool_t *pool,
                       const echo_batch_t *batch, void *hidden, void *workspace,
                       size_t workspace_bytes, void *host_workspace,
                       size_t host_workspace_bytes, void *stream);

/* Per-stage GPU times of the calling thread's last echo_layer_forward while
 * echo_profile(1) is on: norms, qkv GEMM, RoPE, append, attention, o GEMM,
 * MLP GEMMs (gate_up + down) and the element-wise rest, in milliseconds. */
typedef struct {
    float norm_ms, qkv_ms, rope_ms, append_ms, attention_ms, o_ms, mlp_ms, other_ms;
} echo_layer_timing_t;

int echo_layer_timing(echo_layer_timing_t *timing);

#ifdef __cplusplus
}
#endif

#endif /* ECHO_LAYER_H */
