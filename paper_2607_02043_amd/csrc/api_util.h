// Error reporting and batch checks shared by the entry points of libmlastep.
#pragma once
#include "mla_step.h"

namespace mla {

// Sets the thread's mla_last_error message (printf format) and returns code.
int set_error(int code, const char *fmt, ...);

// Host checks of a batch (those of every entry point); *num_rows = T on success.
// Clears the thread's error message first.
int batch_rows(const mla_batch *batch, int *num_rows);

// Workspace bytes of the attention launch for this batch (mixed_step_workspace_bytes
// with the status of the checks and the planning).
int attn_workspace(const mla_batch *batch, size_t *bytes);

}  // namespace mla
