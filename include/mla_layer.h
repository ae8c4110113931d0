/*
 * mla_layer.h -- C ABI of the projections around the mixed-step attention
 * (libmlastep.so), which together with it make one attention layer of the
 * model the paper serves (DeepSeek-V2-Lite, section 6 of the paper:
 * multi-head latent attention, hidden width 2048, 16 heads, no query
 * compression).
 *
 * For each row t of the step (rows and requests as in mla_step.h), with
 * position pos_t = p_r + (t - cu_q[r]) for the request r that owns it:
 *
 *   q[t]       = W_q  x[t]                        [16][192]: per head 128 dims
 *                                                 without position, 64 rope dims
 *   kv[t]      = W_dkv x[t]                       [576]: 512 compressed + 64 rope
 *   latent[t]  = ( RMSNorm(kv[t][0:512]) * gain , RoPE(kv[t][512:576], pos_t) )
 *   q_abs[t][h]= ( W_UK[h]^T q[t][h][0:128]       (the key up-projection folded
 *                                                  into the query: 512 dims),
 *                  RoPE(q[t][h][128:192], pos_t) )
 *   ... mixed-step attention over the cache (mla_step.h) gives o_lat[t][h][512]
 *   o[t][h]    = W_UV[h] o_lat[t][h]              [128] per head
 *   out[t]     = W_o concat_h o[t][h]             [2048]
 *
 * RMSNorm(v) = v / sqrt(mean(v^2) + eps).  RoPE rotates each pair of dims
 * (2i, 2i + 1), i < 32, by the angle pos * base^(-2i / 64).  Scoring the
 * absorbed query against the latent equals scoring the per-head query
 * against the per-head key (W_UK[h] c, rope part): the 1/sqrt(192) softmax
 * scale is the caller's argument to the attention as before.
 *
 * Precision: bf16 inputs and weights, fp32 accumulation; intermediates are
 * kept in fp32 except where a bf16 MFMA operand or a bf16 output is stored:
 * q[t][h][0:128], q_abs, latent, o_lat (rounded to bf16 before W_UV when it
 * is fp32) and o, each rounded to nearest even once.
 *
 * Weights (DEVICE, bf16 bits, contiguous, 16-byte aligned), row-major with
 * the reduction dimension contiguous, as the model stores its linear layers:
 *   w_q     [16 * 192][2048]  row h * 192 + j: head h, query dim j
 *   w_dkv   [576][2048]       rows 0..511 compressed latent, 512..575 rope key
 *   kv_gain [512]             RMSNorm gain of the compressed latent
 *   w_uk_t  [16][512][128]    w_uk_t[h][c][d] = W_UK[h][d][c]: the key
 *                             up-projection of head h, transposed once when
 *                             weights are loaded
 *   w_uv    [16][128][512]    w_uv[h][d][c] = W_UV[h][d][c]
 *   w_uk    [16][128][512]    w_uk[h][d][c] = W_UK[h][d][c], the model's own
 *                             layout (mla_attention_layer only; may be NULL
 *                             when no chunk request takes the multi-head path)
 *   w_o     [2048][16 * 128]  output projection
 *
 * Conventions, errors and streams are those of mla_step.h.  Workspaces are
 * caller-allocated device memory; their contents on entry are ignored except
 * where stated.
 */
#ifndef MLA_LAYER_H
#define MLA_LAYER_H

#include "mla_step.h"

#ifdef __cplusplus
extern "C" {
#endif

#define MLA_HIDDEN 2048
#define MLA_QK_NOPE 128
#define MLA_QK_ROPE 64
#define MLA_V_HEAD 128

typedef struct mla_proj_weights {
    const uint16_t *w_q;
    const uint16_t *w_dkv;
    const uint16_t *kv_gain;
    const uint16_t *w_uk_t;
    const uint16_t *w_uv;
    const uint16_t *w_uk;
    const uint16_t *w_o;
    float rms_eps;   /* > 0 and finite (1e-6 for the served model) */
    float rope_base; /* > 1 and finite (10000) */
} mla_proj_weights;

/* Workspace bytes of mla_pre_attn / mla_post_attn for T rows (0 if T <= 0).
 * The same buffer serves both. */
size_t mla_proj_workspace_bytes(int32_t num_rows);

/* Projections before attention.
 *   hidden       DEVICE bf16 [T][2048], T = rows of the batch.
 *   q_abs        DEVICE bf16 [T][16][576]: absorbed queries, the q of mixed_step.
 *   new_latents  DEVICE bf16 [T][576]: the step's latents, the new_latents of
 *                mixed_step / append_latent_kv.
 * Positions come from batch->cu_q_dev and batch->prefix_lens_dev.
 * Errors: MLA_ERR_INVALID_ARG (null pointer with T > 0, bad eps or base, a
 * negative length), MLA_ERR_WORKSPACE, MLA_ERR_HIP. */
int mla_pre_attn(const mla_batch *batch, const uint16_t *hidden, const mla_proj_weights *w, uint16_t *q_abs,
                 uint16_t *new_latents, void *workspace, size_t workspace_bytes, void *stream);

/* Projections after attention, for T rows.
 *   attn_out     DEVICE [T][16][512] fp32 (MLA_OUT_F32) or bf16 (MLA_OUT_BF16):
 *                the out of mixed_step_attn.
 *   out          DEVICE [T][2048] fp32 or bf16 (out_dtype).
 * Errors: MLA_ERR_INVALID_ARG, MLA_ERR_WORKSPACE, MLA_ERR_HIP. */
int mla_post_attn(int32_t num_rows, const void *attn_out, int32_t attn_dtype, const mla_proj_weights *w,
                  void *out, int32_t out_dtype, void *workspace, size_t workspace_bytes, void *stream);

/* Workspace bytes of mla_attention_layer for this batch (0 on invalid
 * arguments, then mla_last_error says why; an empty batch needs 0).  Its
 * first 256 bytes are the attention's work-queue counters: zero them once
 * before the workspace is first used (see mixed_step_workspace_bytes). */
size_t mla_layer_workspace_bytes(const mla_batch *batch);

/* Tuning overrides, process-wide (for tuning and tests; every later call on
 * any thread sees them).  value -1 restores the library's own choice.
 *   MLA_TUNE_GEMM_BM / _BN / _DEPTH  GEMM tile rows, columns, LDS stages (a
 *       shape that is not instantiated fails the launch with MLA_ERR_HIP);
 *   MLA_TUNE_MHA_MIN_ROWS (>= 2)  chunk requests of at least this many rows
 *       take the layer's multi-head path (off by default);
 *   MLA_TUNE_MHA_PAIRS (>= 0)  and only those whose query-key pairs per key,
 *       c (p + c / 2) / (p + c), reach this many.
 * The first values come from the environment variables MLA_GEMM_BM,
 * MLA_GEMM_BN, MLA_GEMM_D, MLA_LAYER_MHA_MIN and MLA_LAYER_MHA_PAIRS, read
 * once.  Errors: MLA_ERR_INVALID_ARG (unknown knob, value < -1). */
typedef enum {
    MLA_TUNE_GEMM_BM = 0,
    MLA_TUNE_GEMM_BN = 1,
    MLA_TUNE_GEMM_DEPTH = 2,
    MLA_TUNE_MHA_MIN_ROWS = 3,
    MLA_TUNE_MHA_PAIRS = 4,
    MLA_TUNE_COUNT = 5
} mla_tune_knob;
int mla_layer_tune(int32_t knob, int32_t value);

/* One attention layer of the step: mla_pre_attn, mixed_step (append of the
 * new latents + attention, output rounded to bf16, which is where the value
 * up-projection rounds it anyway) and mla_post_attn, enqueued on one stream.
 * Optionally (MLA_TUNE_MHA_MIN_ROWS) a long chunk request takes the
 * multi-head form instead of the absorbed one (same result up to rounding;
 * about 30% of the flops per query-key pair): its keys 0 .. p + c - 1 are
 * up-projected once to per-head keys W_UK c and values W_UV c, stored in
 * fp16 (|values| must stay below 65504), then causal attention runs per head
 * over 128 + 64 query / key dims and 128 value dims with fp16 probabilities;
 * the other rows run on the absorbed kernel.
 *   hidden    DEVICE bf16 [T][2048]
 *   kv_cache  DEVICE bf16 [num_pages][P][576], updated with the step's latents
 *   out       DEVICE [T][2048] fp32 or bf16 (out_dtype)
 * Errors: as the three calls. */
int mla_attention_layer(const mla_batch *batch, const uint16_t *hidden, const mla_proj_weights *w,
                        uint16_t *kv_cache, float softmax_scale, void *out, int32_t out_dtype, void *workspace,
                        size_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* MLA_LAYER_H */
