/*
 * mla_step.h -- C ABI of the MI355X (gfx950) mixed-step latent-attention
 * library (libmlastep.so).
 *
 * One decode-node step of the serving scheme in the paper: in-flight decode
 * rows (one new token per request) mixed with the chunked-prefill rows of
 * deflected requests (section 2.3 "Chunked Prefill"; section 4.3.1, Eq. 4:
 * a step carries B_n decode tokens plus chi - B_n prefill tokens over a node
 * whose cache holds K_n tokens; section 4.3.2, Eq. 5: chunk i of a request
 * starts after the sum of its earlier chunks).  The attention is the absorbed
 * multi-head latent attention of the model the paper serves (DeepSeek-V2-Lite,
 * section 6): 16 query heads share one cached 576-dim latent per token (512
 * compressed dims + 64 rope dims); the value is the latent's first 512 dims.
 *
 * Per request r: p_r = prefix_lens[r] tokens are already cached, c_r =
 * q_lens[r] >= 1 tokens are new this step (a decode row has c_r = 1).  The
 * rows of all requests are concatenated in request order: request r owns rows
 * cu_q[r] .. cu_q[r+1]-1, cu_q[0] = 0, T = cu_q[R].
 *
 *   append_latent_kv:  for t in [p_r, p_r + c_r):
 *       kv_cache[bt[r][t / P]][t % P][:] = new_latents[cu_q[r] + t - p_r][:]
 *   mixed_step_attn:   row i of request r (0 <= i < c_r) attends the keys
 *       j = 0 .. p_r + i of its pages (bottom-right causal), for each head h:
 *       s_j = scale * <q[row][h][0:576], k_j[0:576]>,
 *       out[row][h][e] = sum_j softmax(s)_j * k_j[e]  (e < 512),
 *       lse[row][h] = log sum_j exp(s_j)  (natural log).
 *   Attention reads the appended latents from the cache: call append first,
 *   on the same stream, or call mixed_step, which does both in one launch.
 *
 * Conventions
 *   - bf16 values travel as uint16_t bit patterns.  All pointers are plain
 *     device or host addresses as marked; device arrays are contiguous and
 *     16-byte aligned.  The caller allocates and frees everything; the
 *     library keeps no pointer after a call returns and allocates no device
 *     memory.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream).  Entry
 *     points only enqueue work and never synchronise; a device fault shows up
 *     at the caller's next synchronisation.
 *   - Every entry point returns MLA_OK or a negative mla_status and, on error,
 *     sets a thread-local message (mla_last_error).  All arguments are checked
 *     on the host before anything is enqueued; nothing is launched on error.
 *   - Device arrays must hold the same values as their host twins (q_lens /
 *     prefix_lens).  Block-table entries are not read on the host; kernels
 *     guard every page id (an id outside [0, num_pages) is never dereferenced:
 *     append skips that slot, attention reads page 0 in its place) so a bad
 *     table gives wrong numbers, not a memory fault, and raises the device
 *     flag MLA_FLAG_BAD_PAGE (see mla_device_flags).
 *   - Two requests must not map the same written slot, nor may a request
 *     read a slot another request writes in the same step (undefined result).
 *   - Check mode (mla_debug_set(MLA_DEBUG_CHECK, 1), or MLASTEP_CHECK=1 in the
 *     environment when the library first runs): before launching, every entry
 *     point synchronises the stream and checks on the host that the device
 *     lengths equal the host ones, that every block-table entry a request uses
 *     lies in [0, num_pages) and that no written slot is aliased as above
 *     (MLA_ERR_INVALID_ARG); after launching it synchronises again and turns
 *     the device flags into MLA_ERR_INVALID_ARG (bad page) or MLA_ERR_HIP
 *     (an expired wait).  For debugging: it makes every call synchronous.
 *   - Chunk rows (c_r > 1) carry the value dims through fp16 for their
 *     probability x value products: value dims of magnitude up to 65504 are
 *     exact, larger ones are clamped to +-65504 (wrong results); magnitudes
 *     below 2^-14 keep the fp16 subnormal spacing of 2^-24.  Decode rows keep
 *     bf16 values as they are.
 *   - Reentrant; concurrent calls on different streams need distinct
 *     workspaces.
 */
#ifndef MLA_STEP_H
#define MLA_STEP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MLA_ABI_VERSION 5
#define MLA_NUM_HEADS 16
#define MLA_D_QK 576 /* latent width: 512 compressed + 64 rope dims */
#define MLA_D_V 512  /* value width: the first 512 latent dims */

typedef enum {
    MLA_OK = 0,
    MLA_ERR_INVALID_ARG = -1, /* null pointer, negative or inconsistent size */
    MLA_ERR_UNSUPPORTED = -2, /* page size not a power of two in [1, 1024] */
    MLA_ERR_WORKSPACE = -3,   /* workspace pointer null or too small */
    MLA_ERR_HIP = -4          /* a HIP runtime call failed (message has details) */
} mla_status;

typedef enum { MLA_OUT_F32 = 0, MLA_OUT_BF16 = 1 } mla_out_dtype;

/* One step's batch; the same for every layer of the step. */
typedef struct mla_batch {
    int32_t num_reqs;          /* R >= 0; R == 0 makes every call a no-op */
    int32_t page_size;         /* P: tokens per page, power of two in [1, 1024] */
    int32_t num_pages;         /* pages in the pool (for guards) */
    int32_t max_pages_per_req; /* block-table row stride, >= ceil((p_r + c_r) / P) */
    const int32_t *q_lens;     /* HOST [R]: c_r >= 1; read during the call only */
    const int32_t *prefix_lens;/* HOST [R]: p_r >= 0; read during the call only */
    const int32_t *cu_q_dev;        /* DEVICE [R + 1]: row offsets (prefix sums of q_lens) */
    const int32_t *prefix_lens_dev; /* DEVICE [R]: same values as prefix_lens */
    const int32_t *block_table_dev; /* DEVICE [R][max_pages_per_req]: logical page -> pool page */
} mla_batch;

/* ABI version of the loaded library (MLA_ABI_VERSION it was built with). */
int mla_abi_version(void);

/* Device-side error flags (sticky, per device, raised by any call of this
 * library on the current device since they were last cleared). */
#define MLA_FLAG_BAD_PAGE 1     /* a block-table entry outside [0, num_pages) was met */
#define MLA_FLAG_WAIT_EXPIRED 2 /* a bounded wait inside a kernel gave up: that call's results are undefined */

/* Synchronises `stream`, then stores the current device's flags in *flags
 * and clears them if `clear` is non-zero.  Errors: MLA_ERR_INVALID_ARG (flags
 * NULL), MLA_ERR_HIP. */
int mla_device_flags(int32_t clear, int32_t *flags, void *stream);

/* Debug settings, process-wide:
 *   MLA_DEBUG_CHECK       0 / 1: check mode (see Conventions); the first value
 *                         comes from the environment variable MLASTEP_CHECK;
 *   MLA_DEBUG_SPIN_LIMIT  sleeps a bounded wait inside a kernel takes before
 *                         it gives up (-1: the default, 65536); for tests of
 *                         the flag only: a small limit gives wrong results;
 *   MLA_DEBUG_CHUNK_KEYS  force the work plan's chunk key split (each block of
 *                         8 query tokens is cut into ceil((p + c) / value) key
 *                         ranges; a multiple of 64, capped by what one work
 *                         item may hold); 0 or -1: the planner's choice.  For
 *                         tuning and tests: results stay within rounding;
 *   MLA_DEBUG_WARM_PLAN   1 (the default; -1 restores it): a batch with as
 *                         many chunk requests as the last fully planned one
 *                         (same page size, table width and device), and
 *                         within 1/16 of its decode requests, decode tiles,
 *                         chunk query-key pairs and longest chunk, keeps
 *                         that plan's key split and decode unit size when
 *                         the unit still fits the kernel's limits (counts and
 *                         offsets are recomputed, O(requests)); 0: every new
 *                         batch is planned in full;
 *   MLA_DEBUG_DEC_UNIT    force the decode unit size, in 32-key tiles (made
 *                         smaller until a unit fits the kernel's segment and
 *                         page-window limits); 0 or -1: the planner's choice.
 *                         For tuning and tests: results stay within rounding;
 *   MLA_DEBUG_DEC_FIRST   force the number of workgroups of the attention
 *                         launch that take decode work before chunk work
 *                         (capped by the launch's workgroups; the others
 *                         start on the chunk work, and every workgroup moves
 *                         to the other kind once its own is used up): 0 for
 *                         none (chunk work first everywhere); -1 (the
 *                         default): the planner's choice.  For tuning and
 *                         tests: the results do not change.
 * Errors: MLA_ERR_INVALID_ARG (unknown knob, bad value). */
typedef enum {
    MLA_DEBUG_CHECK = 0,
    MLA_DEBUG_SPIN_LIMIT = 1,
    MLA_DEBUG_CHUNK_KEYS = 2,
    MLA_DEBUG_WARM_PLAN = 3,
    MLA_DEBUG_DEC_UNIT = 4,
    MLA_DEBUG_DEC_FIRST = 5,
    MLA_DEBUG_COUNT = 6
} mla_debug_knob;
int mla_debug_set(int32_t knob, int32_t value);

/* Message of the last non-OK return on this thread ("" if none). */
const char *mla_last_error(void);

/* Device workspace (bytes) that mixed_step_attn / mixed_step need for this
 * batch, or 0 on invalid arguments (then mla_last_error says why; an empty
 * batch also needs 0 bytes).  Depends only on the host arrays, the
 * device's CU count and the debug knobs that force the plan (a workspace
 * sized under one setting of MLA_DEBUG_CHUNK_KEYS, MLA_DEBUG_DEC_UNIT or
 * MLA_DEBUG_DEC_FIRST may be too small under another: the call then fails
 * with MLA_ERR_WORKSPACE).  The first 256 bytes hold the work-queue counters of the
 * attention launch: they must be zero when a workspace is first used (e.g.
 * hipMemset once after allocating it), and every completed call leaves them
 * zero again.  The rest holds fp32 partial results of rows whose keys are
 * split across work items; its contents on entry are ignored. */
size_t mixed_step_workspace_bytes(const mla_batch *batch);

/* Scatter the step's new latents into the paged cache (the append above).
 *   new_latents  DEVICE bf16 [T][576], row order of the batch.
 *   kv_cache     DEVICE bf16 [num_pages][P][576], updated in place; only the
 *                T written slots change.
 * Errors: MLA_ERR_INVALID_ARG (null pointer with T > 0, a negative length,
 * p_r + c_r > max_pages_per_req * P), MLA_ERR_UNSUPPORTED, MLA_ERR_HIP. */
int append_latent_kv(const mla_batch *batch, const uint16_t *new_latents, uint16_t *kv_cache,
                     void *stream);

/* Attention of every row of the step (the attend above).
 *   q              DEVICE bf16 [T][16][576]: absorbed queries (after RoPE).
 *   kv_cache       DEVICE bf16 [num_pages][P][576], already holding the
 *                  step's new latents.
 *   softmax_scale  finite, > 0 (1/sqrt(192) for the served model); applied to
 *                  the fp32 dot product.
 *   out            DEVICE [T][16][512], fp32 (MLA_OUT_F32) or bf16 rounded to
 *                  nearest even (MLA_OUT_BF16).
 *   lse            DEVICE fp32 [T][16] natural-log sum of exp(s), or NULL.
 *   workspace      DEVICE scratch of at least mixed_step_workspace_bytes(batch)
 *                  bytes (may be NULL if that is 0), zeroed once before its
 *                  first use (see mixed_step_workspace_bytes); calls that
 *                  overlap in time need distinct workspaces.
 * Errors: MLA_ERR_INVALID_ARG, MLA_ERR_UNSUPPORTED, MLA_ERR_WORKSPACE,
 * MLA_ERR_HIP. */
int mixed_step_attn(const mla_batch *batch, const uint16_t *q, const uint16_t *kv_cache,
                    float softmax_scale, void *out, int32_t out_dtype, float *lse,
                    void *workspace, size_t workspace_bytes, void *stream);

/* The whole step: append_latent_kv followed by mixed_step_attn, in one
 * launch (plus the split merge when the batch needs one).  Results (out, lse
 * and the cache) are bit-identical to the two calls.  The step's new keys are
 * read from new_latents while they are written into the cache, so no
 * workgroup waits for the append.
 *   new_latents  DEVICE bf16 [T][576], row order of the batch.
 *   kv_cache     DEVICE bf16 [num_pages][P][576]: holds the cached prefixes on
 *                entry; on return also the T new latents (only their slots
 *                change).
 *   other arguments as for mixed_step_attn.
 * Errors: as mixed_step_attn, and MLA_ERR_INVALID_ARG for a NULL new_latents
 * with T > 0. */
int mixed_step(const mla_batch *batch, const uint16_t *q, const uint16_t *new_latents, uint16_t *kv_cache,
               float softmax_scale, void *out, int32_t out_dtype, float *lse, void *workspace,
               size_t workspace_bytes, void *stream);

/* mixed_step without a workspace argument, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation.  Same arguments, contract and results (bit for bit)
 * as mixed_step; it allocates nothing and calls no allocating routine.  Its
 * workspace is a library-owned device buffer of MLA_NOALLOC_SCRATCH_BYTES per
 * device, set up on the first call on each device (make that call outside
 * graph capture); it lives until the process ends.
 *   - Every call on one device shares that buffer: calls that overlap in time
 *     on one device (several streams or threads) race and give undefined
 *     results.  Serialise them, or use mixed_step with distinct workspaces.
 *   - A batch whose plan needs more scratch than MLA_NOALLOC_SCRATCH_BYTES
 *     (mixed_step_workspace_bytes tells) is rejected with MLA_ERR_WORKSPACE
 *     before anything is enqueued.
 * Errors: as mixed_step. */
#define MLA_NOALLOC_SCRATCH_BYTES (128u << 20)
int mixed_step_noalloc(const mla_batch *batch, const uint16_t *q, const uint16_t *new_latents, uint16_t *kv_cache,
                       float softmax_scale, void *out, int32_t out_dtype, float *lse, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* MLA_STEP_H */
