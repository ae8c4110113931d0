// Launch-side description of the projection kernels of libmlastep (host <-> device).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace proj {

constexpr int kHidden = 2048;                 // model width
constexpr int kHeads = 16;
constexpr int kNope = 128;                    // per-head query dims without position
constexpr int kRope = 64;                     // rope dims (per head for queries, shared for keys)
constexpr int kQkHead = kNope + kRope;        // 192
constexpr int kQCols = kHeads * kQkHead;      // 3072
constexpr int kLatent = 512;                  // compressed latent
constexpr int kDqk = kLatent + kRope;         // 576
constexpr int kVHead = 128;                   // per-head value dims after the up-projection
constexpr int kOCols = kHeads * kVHead;       // 2048

constexpr int kBN = 64;   // output columns per workgroup of the fp32-activation GEMM
constexpr int kBK = 64;   // reduction depth per pipeline stage

enum Epilogue : int {
    kStoreBf16 = 0,  // C (bf16, row stride ldc)
    kStoreF32 = 1,   // C (fp32, row stride ldc)
    kQkvSplit = 2,   // first projection: nope -> qn bf16, rope -> qpe fp32, latent -> kvf fp32
    kStoreF16 = 3,   // C (fp16, row stride ldc)
};

struct RowArgs {
    const float *qpe;         // [T][16][64]
    const float *kvf;         // [T][576]
    const uint16_t *gamma;    // [512] bf16
    const int32_t *cu_q;      // [R + 1]
    const int32_t *prefix;    // [R]
    uint16_t *q_abs;          // [T][16][576]: writes dims 512..575 of every head
    uint16_t *latent;         // [T][576]
    int32_t num_reqs;
    int32_t num_rows;
    float eps;
    double log2_base;         // log2 of the rope base
};

// Key rows of one chunk request for the multi-head path, run by extra
// workgroups of its up-projection launch (8 keys each): the rope key of every
// key 0 .. nkeys - 1 into kpe as fp16, and the new latents (keys p ..) into
// their cache slots.
struct KeyRowsJob {
    uint16_t *cache;         // bf16 [pages][P][576]: keys < p are read here, keys >= p written
    const uint16_t *lat;     // bf16 [nkeys - p][576]: the request's new latents
    const int32_t *bt;       // block-table row of the request
    int log2p, npages;
    int p, nkeys;
    uint16_t *kpe;           // fp16 [nkeys][64]
};
constexpr int kKeyRowsPerWg = 8;

// C[z][m][n] = sum_k A[z][m][k] * B[z][n][k]: both operands K-contiguous.
// Element strides; z = blockIdx.z.  Columns n >= n_split take their B rows
// from b2 (row n - n_split), so two weight matrices act as one.
struct GemmArgs {
    const void *a;        // bf16 bits or fp32 (a_f32)
    long long lda, a_bstride;
    const uint16_t *b;
    const uint16_t *b2;
    long long ldb, b_bstride;
    int n_split;
    int M, N, K;
    // Gathered A (non-null a_bt): row m is token m of one request in the paged
    // cache, at a + (a_bt[m >> a_log2p] * 2^a_log2p + (m & (2^a_log2p - 1))) * lda;
    // page ids outside [0, a_npages) read page 0.  Rows m >= a_new_from come
    // from a_new + (m - a_new_from) * lda instead (the step's new latents).
    const int32_t *a_bt;
    int a_log2p, a_npages;
    const uint16_t *a_new;
    int a_new_from;
    void *c;
    long long ldc, c_bstride;
    // kQkvSplit outputs
    uint16_t *qn;         // [M][16][128] bf16
    float *qpe;           // [M][16][64]
    float *kvf;           // [M][576]
    // Optional rope / norm rows run by rope_wgs extra workgroups of the
    // launch (blockIdx.x past the tiles, z = 0): independent work that
    // overlaps the GEMM instead of taking a launch of its own.
    RowArgs rope;
    int rope_wgs;
    KeyRowsJob keys;          // or the key rows of a multi-head chunk request
    int keys_wgs;
};


// Causal attention of one chunk request in the multi-head form: per head,
// queries (128 dims without position + 64 rope dims) against up-projected
// keys (W_UK c, 128 dims) plus the shared rope key, values W_UV c (128 dims).
struct MhaArgs {
    const uint16_t *qn;      // bf16 [T][16][128]: query dims without position
    const uint16_t *q_abs;   // bf16 [T][16][576]: dims 512..575 hold the rotated query rope dims
    const uint16_t *kv;      // fp16 [p + c][4096]: k (h * 128 + d), then v (2048 + h * 128 + d)
    const uint16_t *kpe;     // fp16 [p + c][64]: the rotated rope key of every key
    uint16_t *o;             // bf16 [T][2048]: o[row][h * 128 + d]
    int row0, c, p;          // the request's rows row0 .. row0 + c - 1 sit at positions p .. p + c - 1
    float scale_log2;        // softmax scale * log2(e)
};
constexpr int kMhaWaves = 8;
constexpr int kMhaTokens = 16 * kMhaWaves;  // query tokens per workgroup (16 per wave)
hipError_t launch_mha_prefill(const MhaArgs &a, hipStream_t s);

// Tile shape of one GEMM launch: bm x bn outputs per workgroup; `depth` > 0
// picks the LDS ring fed by direct loads with that many stages, 0 the
// register-staged kernel.  Instantiated: ring, bn 64 with (bm, depth) (32, 6),
// (64, 4), (128, 3); ring, bn 128 with (32, 4), (64, 3), (128, 2), (128, 3);
// register-staged (bm, bn) (128, 256) and (256, 128) on eight waves, (32,
// 128), (64, 128), (128, 128) on four.  fp32 activations use bn = 64 and any
// bm of 32, 64, 128 (N a multiple of 64).
struct GemmShape {
    int bm, bn, depth, epi;
};

// The launch covers ceil(M / bm) * ceil(N / bn) tiles x batch, plus
// g.rope_wgs workgroups of rope / norm rows (four rows each) or g.keys_wgs of
// key rows (kKeyRowsPerWg each).
hipError_t launch_gemm(const GemmArgs &g, const GemmShape &t, bool a_f32, int batch, hipStream_t s);
inline int rope_norm_wgs(int num_rows) { return (num_rows + 3) / 4; }

}  // namespace proj
