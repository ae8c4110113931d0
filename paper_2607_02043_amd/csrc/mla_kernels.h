// Launch-side description of the kernels of libmlastep (host <-> device).
#pragma once
#include "chunk_route.h"
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mla {

constexpr int kHeads = 16;
constexpr int kDqk = 576;   // latent: 512 compressed + 64 rope dims
constexpr int kDv = 512;    // value: first 512 latent dims
constexpr int kRowBytes = kDqk * 2;
constexpr int kKeysPerTile = 32;
constexpr int kPageWindow = 256;   // page ids one work item may touch
constexpr int kThreads = 256;      // 4 wavefronts of 64 (merge, append; DMA rounds of the attention kernel)
constexpr int kAttnThreads = 512;  // attention kernel: 8 wavefronts, two per SIMD
constexpr int kChunkBlockTokens = 8;                        // tokens per chunk work item
constexpr int kPartialFloats = kHeads * kDv;                // one row's partial output
constexpr int kPartialStats = kHeads * 2;                   // one row's (max, sum) per head
constexpr int kMaxDecSegments = 64;                         // requests one decode workgroup may touch
constexpr int kFlagBadPage = 1;       // a block-table entry outside [0, num_pages) was met (MLA_FLAG_BAD_PAGE)
constexpr int kFlagWaitExpired = 2;   // a bounded wait inside a kernel gave up (MLA_FLAG_WAIT_EXPIRED)
constexpr int kSpinLimit = 1 << 16;   // sleeps of a bounded wait before it gives up
constexpr size_t kNoAllocScratchBytes = size_t(128) << 20;  // scratch of mixed_step_noalloc, per device
constexpr int kMaxDevices = 64;

struct AttnArgs {
    const uint16_t *q;
    const uint16_t *kv;
    // Fused append (both null otherwise): the step's new latents, read in place
    // of their cache slots, and the cache they are written into.
    const uint16_t *new_kv;
    uint16_t *kv_out;
    const int32_t *cu_q;
    const int32_t *prefix;
    const int32_t *bt;
    void *out;
    float *lse;
    float *ws_chunk_o;    // [n_chunk_items][block tokens][16][512]
    float *ws_chunk_ml;   // [n_chunk_items][block tokens][16][2]
    float *ws_dec_o;      // [2 units][16][512]: first / last segment of each decode unit
    float *ws_dec_ml;     // [2 units][16][2]
    int32_t *work;        // [3]: next chunk item, workgroups done, next decode item; zero between calls
    int32_t num_reqs;
    int32_t num_rows;
    int32_t page_size;
    int32_t log2_page;
    int32_t max_pages;
    int32_t num_pages;
    float scale_log2;     // softmax scale * log2(e)
    int32_t ks_chunk;          // chunk blocks are cut into ceil((p + c) / ks_chunk) key ranges (a multiple of 64)
    int32_t chunk_rev;         // chunk items numbered from the last request to the first
    int32_t n_chunk_items;     // work items 0 .. n_chunk_items - 1
    int32_t n_dec_units;       // then the decode items: pairs of units (slices of the flattened decode
                               // tile list), one unit per wave group
    int32_t dec_unit_tiles;    // 32-key decode tiles per unit
    int32_t dec_total_tiles;
    int32_t grid;              // persistent workgroups of the attention launch
    int32_t dec_first_wgs;     // workgroups 0 .. dec_first_wgs - 1 take decode items before chunk items
    int32_t merge_hsplit;      // merge workgroups per split decode row (1, 4 or 8: heads split among them)
    int32_t out_bf16;
    int32_t spin_limit;        // sleeps of a bounded wait before it gives up (kSpinLimit)
    ChunkRoute route;          // chunk requests it sends to the multi-head path are left out of this launch
};

struct AppendArgs {
    const uint16_t *src;
    uint16_t *kv;
    const int32_t *cu_q;
    const int32_t *prefix;
    const int32_t *bt;
    int32_t num_reqs;
    int32_t num_rows;
    int32_t page_size;
    int32_t log2_page;
    int32_t max_pages;
    int32_t num_pages;
};

hipError_t launch_append(const AppendArgs &a, hipStream_t s);
// Reads the device's sticky kernel error flags (kFlag*), and clears them if asked.
hipError_t read_flags(int *flags, bool clear);
// Device address of the current device's no-allocation scratch
// (kNoAllocScratchBytes bytes, counters zero on first use); set up once per device.
hipError_t noalloc_scratch(void **ptr);
hipError_t launch_attention(const AttnArgs &a, hipStream_t s);
hipError_t launch_combine(const AttnArgs &a, hipStream_t s);

}  // namespace mla
