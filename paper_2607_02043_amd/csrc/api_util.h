// Error reporting and batch checks shared by the entry points of libmlastep.
#pragma once
#include "mla_step.h"
#include "chunk_route.h"

namespace mla {

// Sets the thread's mla_last_error message (printf format) and returns code.
int set_error(int code, const char *fmt, ...);

// Host checks of a batch (those of every entry point); *num_rows = T on success.
// Clears the thread's error message first.
int batch_rows(const mla_batch *batch, int *num_rows);

// Workspace bytes of the attention launch for this batch (mixed_step_workspace_bytes
// with the status of the checks and the planning), leaving out the chunk
// requests that `route` sends to the multi-head path.
int attn_workspace(const mla_batch *batch, size_t *bytes, ChunkRoute route = kAbsorbAll);

// mixed_step (no lse) over every row except those of the chunk requests that
// `route` sends to the multi-head path, which are left untouched: neither
// attended nor appended.  new_latents NULL: no append (mixed_step_attn).
int attend_rows(const mla_batch *batch, const uint16_t *q, const uint16_t *new_latents, uint16_t *kv_cache,
                float softmax_scale, void *out, int32_t out_dtype, void *workspace, size_t workspace_bytes, void *stream,
                ChunkRoute route);

}  // namespace mla
