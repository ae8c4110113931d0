// Which chunk requests of a layer step leave the absorbed attention kernel
// for the multi-head path.  Shared by the host planner, the attention kernel
// (which must leave out exactly those requests) and the layer's dispatch.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mla {

// A chunk request of c rows at prefix p takes the multi-head path when
// c >= min_rows and its query-key pairs per up-projected key,
// c (p + c / 2) / (p + c), reach pair_keys.  The multi-head form saves a
// fixed time per pair and pays a fixed time per key of the request for the
// up-projection, so the ratio decides.  min_rows = INT32_MAX routes nothing.
struct ChunkRoute {
    int32_t min_rows;
    int32_t pair_keys;
    __host__ __device__ bool multi_head(long long p, long long c) const {
        return c >= min_rows && c * (2 * p + c) >= 2LL * pair_keys * (p + c);
    }
};

constexpr ChunkRoute kAbsorbAll{0x7fffffff, 0};

}  // namespace mla
