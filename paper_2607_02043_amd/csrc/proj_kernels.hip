// Projection kernels of one absorbed multi-head latent attention layer for
// gfx950: the GEMMs before and after the mixed-step attention and the per-row
// RoPE / RMSNorm epilogue.  Host-side contracts are in include/mla_layer.h.
//
// GEMM: C = A . B^T with both operands K-contiguous (activations [M][K],
// weights [N][K] as the model stores them), bf16 MFMA 16x16x32 with fp32
// accumulation.  A workgroup of four waves computes a BM x 64 tile; each wave
// a (BM / 2) x 32 block.  K advances 64 at a time through a ring of D LDS
// stages that direct global -> LDS loads fill D - 1 stages ahead, so that a
// workgroup keeps several round trips to HBM in flight (one stage in flight
// leaves the loop waiting a full memory latency per 64 of K).  A variant for
// fp32 activations converts them to bf16 in registers on the way to LDS
// (two stages, register staged).
#include "proj_kernels.h"

namespace proj {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x4 mfma(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// float -> bf16 bits, round to nearest even
__device__ __forceinline__ uint32_t bf16_of(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }
__device__ __forceinline__ uint32_t pack2(float lo, float hi) { return bf16_of(lo) | (bf16_of(hi) << 16); }
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// 16-byte slot of (row, k-chunk) in one LDS stage: a row is 8 chunks (64
// bf16 of K); the chunk index is XOR-ed with (row / 2) % 8 so that the 16 rows
// an MFMA operand read touches, and the 2 rows x 8 chunks of 16 consecutive
// lanes of a store pass, land on 16 distinct bank groups.
__device__ __forceinline__ int slot(int row, int kc) { return row * 8 + (kc ^ ((row >> 1) & 7)); }

// One 16-byte global -> LDS load per lane: lane i writes LDS bytes
// [lds + 16 i, lds + 16 i + 16); `lds` must be wave-uniform.  Completion is
// tracked by hand with vmcnt (the compiler does not see these loads).
__device__ __forceinline__ void dma16(const void *gsrc, uint32_t lds) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %1, off" : : "{m0}"(lds), "v"(gsrc) : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

// Wait until at most r * NPW of this wave's loads are in flight (r <= R).
template <int NPW, int R>
__device__ __forceinline__ void wait_stages(int r) {
    if constexpr (R == 0) {
        wait_vm<0>();
    } else {
        if (r >= R) wait_vm<R * NPW>();
        else wait_stages<NPW, R - 1>(r);
    }
}

// Stores of one tile.  acc[mb][nb][i] = C[rbase + 16 mb + i][cbase + 16 nb];
// columns at or past N are not stored.
template <int EPI, int MB, int NB>
__device__ __forceinline__ void store_tile(const GemmArgs &g, const f32x4 (&acc)[MB][NB], int rbase, int cbase,
                                           int z) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = rbase + mb * 16 + i;
            if (row >= g.M) continue;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                const float v = acc[mb][nb][i];
                const int n = cbase + nb * 16;
                if (n >= g.N) continue;
                if constexpr (EPI == kStoreBf16) {
                    static_cast<uint16_t *>(g.c)[z * g.c_bstride + (long long)row * g.ldc + n] = (uint16_t)bf16_of(v);
                } else if constexpr (EPI == kStoreF32) {
                    static_cast<float *>(g.c)[z * g.c_bstride + (long long)row * g.ldc + n] = v;
                } else if constexpr (EPI == kStoreF16) {
                    static_cast<_Float16 *>(g.c)[z * g.c_bstride + (long long)row * g.ldc + n] = (_Float16)v;
                } else {
                    if (n < kQCols) {
                        const int h = n / kQkHead, j = n - h * kQkHead;
                        if (j < kNope)
                            g.qn[((long long)row * kHeads + h) * kNope + j] = (uint16_t)bf16_of(v);
                        else
                            g.qpe[((long long)row * kHeads + h) * kRope + j - kNope] = v;
                    } else {
                        g.kvf[(long long)row * kDqk + n - kQCols] = v;
                    }
                }
            }
        }
    }
}

// One wave per row.  Position of row t of request r: prefix_r + (t - cu_q[r]).
// Rope rotates pairs (2i, 2i + 1) by pos * base^(-2i / 64); the angle and its
// sine and cosine are taken in double, the rotation in fp32.  The latent's
// 512 compressed dims are RMS-normalised in fp32 and scaled by the gain.
//
// The request of a row is found by a wave-parallel search of cu_q: each
// level, 64 lanes test 64 evenly spaced entries of the remaining range, so a
// level costs one load per lane and the range shrinks 64-fold.
__device__ __forceinline__ int request_of(const int32_t *cu_q, int num_reqs, int row, int lane) {
    int lo = 0, n = num_reqs;  // answer in [lo, lo + n): the last r with cu_q[r] <= row
    while (n > 1) {
        const int step = (n + 63) >> 6;
        const int idx = lo + lane * step;
        const bool le = idx < lo + n && cu_q[idx] <= row;
        const int k = __popcll(__ballot(le)) - 1;  // cu_q is increasing: the true lanes are a prefix
        lo += k * step;
        n = min(step, n - k * step);
    }
    return lo;
}

__device__ __forceinline__ void rope_norm_rows(const RowArgs &r, int wg) {
    const int row = wg * 4 + (threadIdx.x >> 6);
    if (row >= r.num_rows) return;
    const int lane = threadIdx.x & 63;
    const int req = request_of(r.cu_q, r.num_reqs, row, lane);
    const int pos = r.prefix[req] + row - r.cu_q[req];

    const int i = lane & 31;
    const double ang = (double)pos * exp2(-(double)(2 * i) / (double)kRope * r.log2_base);
    double sd, cd;
    sincos(ang, &sd, &cd);
    const float sn = (float)sd, cs = (float)cd;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const int h = (lane >> 5) + 2 * k;
        const float2 x = *reinterpret_cast<const float2 *>(r.qpe + ((long long)row * kHeads + h) * kRope + 2 * i);
        *reinterpret_cast<uint32_t *>(r.q_abs + ((long long)row * kHeads + h) * kDqk + kLatent + 2 * i) =
            pack2(x.x * cs - x.y * sn, x.x * sn + x.y * cs);
    }
    if (lane < 32) {
        const float2 x = *reinterpret_cast<const float2 *>(r.kvf + (long long)row * kDqk + kLatent + 2 * i);
        *reinterpret_cast<uint32_t *>(r.latent + (long long)row * kDqk + kLatent + 2 * i) =
            pack2(x.x * cs - x.y * sn, x.x * sn + x.y * cs);
    }

    const float *src = r.kvf + (long long)row * kDqk + lane * 8;
    const float4 a = *reinterpret_cast<const float4 *>(src), b = *reinterpret_cast<const float4 *>(src + 4);
    float ss = a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w + b.x * b.x + b.y * b.y + b.z * b.z + b.w * b.w;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
    const float inv = 1.0f / sqrtf(ss / (float)kLatent + r.eps);
    const u32x4 gw = *reinterpret_cast<const u32x4 *>(r.gamma + lane * 8);
    const u32x4 y = {pack2(a.x * inv * bf16_lo(gw[0]), a.y * inv * bf16_hi(gw[0])),
                     pack2(a.z * inv * bf16_lo(gw[1]), a.w * inv * bf16_hi(gw[1])),
                     pack2(b.x * inv * bf16_lo(gw[2]), b.y * inv * bf16_hi(gw[2])),
                     pack2(b.z * inv * bf16_lo(gw[3]), b.w * inv * bf16_hi(gw[3]))};
    *reinterpret_cast<u32x4 *>(r.latent + (long long)row * kDqk + lane * 8) = y;
}

// Tile of workgroup blockIdx.x.  Tiles are ordered in groups of kGroup row
// tiles: within a group the row tile varies fastest, then the column tile.
// Workgroups are dealt to the 8 XCDs round-robin, so the order is renumbered
// to give each XCD a contiguous run of it: the workgroups resident on one XCD
// then cover a block of about 8 x 8 tiles and share both operands in its L2.
constexpr int kGroup = 8;

__device__ __forceinline__ void tile_of(int M, int N, int BM, int BN, int *m0, int *n0) {
    const int mtiles = (M + BM - 1) / BM;
    const int ntiles = (N + BN - 1) / BN;
    const int tiles = mtiles * ntiles;
    int t = blockIdx.x;
    const int per = tiles >> 3;
    if (t < per * 8) t = (t & 7) * per + (t >> 3);
    const int g = t / (kGroup * ntiles);
    const int first = g * kGroup;
    const int gm = min(kGroup, mtiles - first);
    const int r = t - g * kGroup * ntiles;
    *m0 = (first + r % gm) * BM;
    *n0 = (r / gm) * BN;
}

__device__ __forceinline__ void key_rows(const KeyRowsJob &j, int wg) {
    // thread: key wg * 8 + tid / 32, 16-byte chunk tid % 32 of the 72 of a latent row
    const int key = wg * kKeyRowsPerWg + (threadIdx.x >> 5), lane = threadIdx.x & 31;
    if (key >= j.nkeys) return;
    // A page id outside the pool: a prefix key is read from page 0 instead
    // (wrong numbers, no fault); a new latent is not written anywhere, as in
    // the other append paths.
    const int pg_raw = j.bt[key >> j.log2p];
    const bool pg_ok = (unsigned)pg_raw < (unsigned)j.npages;
    const int pg = pg_ok ? pg_raw : 0;
    uint16_t *slot = j.cache + (((size_t)pg << j.log2p) + (key & ((1 << j.log2p) - 1))) * kDqk;
    const uint16_t *src = key < j.p ? slot : j.lat + (size_t)(key - j.p) * kDqk;
    const bool write = key >= j.p && pg_ok;
    for (int c = lane; c < kDqk / 8; c += 32) {
        const u32x4 v = *reinterpret_cast<const u32x4 *>(src + 8 * c);
        if (write) *reinterpret_cast<u32x4 *>(slot + 8 * c) = v;  // append of a new latent
        if (c >= kLatent / 8) {
            u32x4 h;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const auto f = __builtin_amdgcn_cvt_pkrtz(__uint_as_float(v[k] << 16), __uint_as_float(v[k] & 0xffff0000u));
                h[k] = __builtin_bit_cast(uint32_t, f);
            }
            *reinterpret_cast<u32x4 *>(j.kpe + (size_t)key * kRope + 8 * (c - kLatent / 8)) = h;
        }
    }
}

// Workgroups past the tiles run the launch's side job (z = 0) or nothing;
// true when this workgroup is one of them.
__device__ __forceinline__ bool is_rope_wg(const GemmArgs &g, int BM, int BN) {
    const int tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
    if ((int)blockIdx.x < tiles) return false;
    if (blockIdx.z == 0) {
        if (g.rope_wgs > 0) rope_norm_rows(g.rope, blockIdx.x - tiles);
        else key_rows(g.keys, blockIdx.x - tiles);
    }
    return true;
}

// bf16 activations.  D-stage LDS ring filled by direct loads; four waves in
// a 2 x 2 grid, each computing a (BM / 2) x (BN / 2) block.
template <int BM, int BN, int D, int EPI>
__global__ __launch_bounds__(256) void gemm_ring_kernel(const GemmArgs g) {
    constexpr int ROWS = BM + BN;            // A rows then B rows of a stage
    constexpr int STAGE = ROWS * 8;          // 16-byte slots per stage
    constexpr int NPW = STAGE / 64 / 4;      // loads per wave per stage
    constexpr int WM = BM / 2, MB = WM / 16;
    constexpr int WN = BN / 2, NB = WN / 16;
    static_assert(STAGE % 256 == 0, "a stage must split evenly over four waves");
    __shared__ __attribute__((aligned(1024))) u32x4 ring[D * STAGE];

    if (is_rope_wg(g, BM, BN)) return;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int m0, n0;
    tile_of(g.M, g.N, BM, BN, &m0, &n0);
    const int z = blockIdx.z;

    // Slot s = (wave * NPW + i) * 64 + lane of every stage is filled by this
    // lane's i-th load: chunk (row, kc) with slot(row, kc) = s.  Rows past M
    // or N repeat the last row; their results are never stored.
    const uint16_t *src[NPW];
    const uint16_t *bseg = n0 >= g.n_split ? g.b2 : g.b;
    const int nbase = n0 >= g.n_split ? g.n_split : 0;
#pragma unroll
    for (int i = 0; i < NPW; ++i) {
        const int s = (wave * NPW + i) * 64 + lane;
        const int row = s >> 3;
        const int kc = (s & 7) ^ ((row >> 1) & 7);
        if (row < BM) {
            const int r = min(m0 + row, g.M - 1);
            long long ar = r;
            const uint16_t *abase = static_cast<const uint16_t *>(g.a);
            if (g.a_bt != nullptr) {
                if (g.a_new != nullptr && r >= g.a_new_from) {
                    abase = g.a_new;
                    ar = r - g.a_new_from;
                } else {
                    int pg = g.a_bt[r >> g.a_log2p];
                    pg = (unsigned)pg < (unsigned)g.a_npages ? pg : 0;
                    ar = ((long long)pg << g.a_log2p) + (r & ((1 << g.a_log2p) - 1));
                }
            }
            src[i] = abase + z * g.a_bstride + ar * g.lda + kc * 8;
        } else {
            const int n = min(n0 + row - BM, g.N - 1) - nbase;
            src[i] = bseg + z * g.b_bstride + (long long)n * g.ldb + kc * 8;
        }
    }
    const uint32_t ring_lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(ring));
    auto issue = [&](int st) {
        const uint32_t dst = ring_lds + (uint32_t)((st % D) * STAGE * 16 + wave * NPW * 1024);
#pragma unroll
        for (int i = 0; i < NPW; ++i) dma16(src[i] + st * kBK, __builtin_amdgcn_readfirstlane(dst + i * 1024));
    };

    f32x4 acc[MB][NB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int wr = (wave >> 1) * WM;       // wave's first A row in the stage
    const int wc = BM + (wave & 1) * WN;   // wave's first B row in the stage
    const int nk = g.K / kBK;

#pragma unroll
    for (int st = 0; st < D - 1; ++st)
        if (st < nk) issue(st);
    for (int kt = 0; kt < nk; ++kt) {
        if (kt + D - 1 < nk) issue(kt + D - 1);
        // stage kt has landed once no more than the stages issued after it are in flight
        wait_stages<NPW, D - 1>(min(D - 1, nk - 1 - kt));
        __syncthreads();
        const u32x4 *cur = ring + (kt % D) * STAGE;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int kc = s * 4 + (lane >> 4);
            u32x4 fa[MB], fb[NB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) fa[mb] = cur[slot(wr + mb * 16 + (lane & 15), kc)];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) fb[nb] = cur[slot(wc + nb * 16 + (lane & 15), kc)];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = mfma(fa[mb], fb[nb], acc[mb][nb]);
        }
        __syncthreads();  // the slot of stage kt is refilled by the next iteration's load
    }
    store_tile<EPI, MB, NB>(g, acc, m0 + wr + 4 * (lane >> 4), n0 + (wave & 1) * WN + (lane & 15), z);
}

// bf16 activations, register-staged: each thread loads its share of the
// next two stages into registers (two register sets) while the current stage
// is consumed from LDS, then writes the older set to the other LDS buffer.
// Register loads stream from L2 well above the rate of direct global -> LDS
// loads, and the projection GEMMs re-read both operands from L2 many times.
// WR x WC waves, each computing a (BM / WR) x (BN / WC) block.
template <int BM, int BN, int WR, int WC, int EPI>
__global__ __launch_bounds__(64 * WR * WC) void gemm_reg_kernel(const GemmArgs g) {
    constexpr int NT = 64 * WR * WC;
    constexpr int ROWS = BM + BN;
    constexpr int STAGE = ROWS * 8;  // 16-byte slots per stage
    constexpr int LPT = STAGE / NT;  // loads per thread per stage
    static_assert(STAGE % NT == 0, "a stage must split evenly over the threads");
    constexpr int WM = BM / WR, MB = WM / 16;
    constexpr int WN = BN / WC, NB = WN / 16;
    __shared__ u32x4 sm[2 * STAGE];

    if (is_rope_wg(g, BM, BN)) return;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int m0, n0;
    tile_of(g.M, g.N, BM, BN, &m0, &n0);
    const int z = blockIdx.z;

    // Chunk c = tid + NT i: row c / 8, k-chunk c % 8 (eight threads read one
    // row's 128 bytes).  Rows past M or N repeat the last row; never stored.
    const uint16_t *src[LPT];
    int dst[LPT];
    const uint16_t *bseg = n0 >= g.n_split ? g.b2 : g.b;
    const int nbase = n0 >= g.n_split ? g.n_split : 0;
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
        const int c = tid + NT * i;
        const int row = c >> 3, kc = c & 7;
        dst[i] = slot(row, kc);
        if (row < BM) {
            const int r = min(m0 + row, g.M - 1);
            src[i] = static_cast<const uint16_t *>(g.a) + z * g.a_bstride + (long long)r * g.lda + kc * 8;
        } else {
            const int n = min(n0 + row - BM, g.N - 1) - nbase;
            src[i] = bseg + z * g.b_bstride + (long long)n * g.ldb + kc * 8;
        }
    }
    u32x4 r0[LPT], r1[LPT];
    auto load = [&](u32x4(&r)[LPT], int st) {
#pragma unroll
        for (int i = 0; i < LPT; ++i) r[i] = *reinterpret_cast<const u32x4 *>(src[i] + st * kBK);
    };
    auto store = [&](const u32x4(&r)[LPT], int buf) {
#pragma unroll
        for (int i = 0; i < LPT; ++i) sm[buf * STAGE + dst[i]] = r[i];
    };

    f32x4 acc[MB][NB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int wr = (wave / WC) * WM;
    const int wc = BM + (wave % WC) * WN;
    auto compute = [&](int buf) {
        const u32x4 *cur = sm + buf * STAGE;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int kc = s * 4 + (lane >> 4);
            u32x4 fa[MB], fb[NB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) fa[mb] = cur[slot(wr + mb * 16 + (lane & 15), kc)];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) fb[nb] = cur[slot(wc + nb * 16 + (lane & 15), kc)];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = mfma(fa[mb], fb[nb], acc[mb][nb]);
        }
    };

    // Loads past the last stage re-read the last stage (in bounds, never
    // stored): the loads stay unconditional, so the two register sets are not
    // merged at branch joins (a copy of a register still being loaded waits
    // for every load in flight).
    const int nk = g.K / kBK;
    load(r0, 0);
    load(r1, min(1, nk - 1));
    store(r0, 0);
    __syncthreads();
    for (int kt = 0; kt < nk; kt += 2) {
        // stage kt in buffer 0, stage kt + 1 in r1, stage kt + 2 loading into r0
        load(r0, min(kt + 2, nk - 1));
        compute(0);
        if (kt + 1 < nk) store(r1, 1);
        __syncthreads();
        if (kt + 1 >= nk) break;
        load(r1, min(kt + 3, nk - 1));
        compute(1);
        if (kt + 2 < nk) store(r0, 0);
        __syncthreads();
    }
    store_tile<EPI, MB, NB>(g, acc, m0 + wr + 4 * (lane >> 4), n0 + (wc - BM) + (lane & 15), z);
}

// fp32 activations, converted to bf16 (nearest even) in registers; two LDS
// stages, the next one held in registers while the current one is consumed.
template <int BM, int EPI>
__global__ __launch_bounds__(256) void gemm_f32a_kernel(const GemmArgs g) {
    constexpr int CA = BM / 32;  // A chunks (of 8 values) per thread per stage
    constexpr int WM = BM / 2;   // rows per wave
    constexpr int MB = WM / 16;  // 16-row MFMA blocks per wave
    constexpr int ROWS = BM + kBN;
    __shared__ u32x4 sm[2][ROWS * 8];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int m0, n0;
    tile_of(g.M, g.N, BM, kBN, &m0, &n0);
    const int z = blockIdx.z;

    // This thread moves chunk (row crow + 32 i, k-chunk ckc) of each operand.
    const int crow = tid >> 3, ckc = tid & 7;
    const uint16_t *bsrc = (n0 >= g.n_split ? g.b2 + (long long)(n0 - g.n_split) * g.ldb
                                            : g.b + (long long)n0 * g.ldb) +
                           z * g.b_bstride + (long long)crow * g.ldb + ckc * 8;
    long long aoff[CA];
#pragma unroll
    for (int i = 0; i < CA; ++i) {
        const int r = min(m0 + crow + 32 * i, g.M - 1);  // rows past M repeat the last row; never stored
        aoff[i] = z * g.a_bstride + (long long)r * g.lda + ckc * 8;
    }
    const float *af = static_cast<const float *>(g.a);

    u32x4 rb[2];
    float4 rf[CA][2];
    auto load = [&](int k0) {
#pragma unroll
        for (int i = 0; i < CA; ++i) {
            rf[i][0] = *reinterpret_cast<const float4 *>(af + aoff[i] + k0);
            rf[i][1] = *reinterpret_cast<const float4 *>(af + aoff[i] + k0 + 4);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) rb[i] = *reinterpret_cast<const u32x4 *>(bsrc + i * 32 * g.ldb + k0);
    };
    auto store = [&](u32x4 *s) {
#pragma unroll
        for (int i = 0; i < CA; ++i) {
            const float4 x = rf[i][0], y = rf[i][1];
            s[slot(crow + 32 * i, ckc)] = u32x4{pack2(x.x, x.y), pack2(x.z, x.w), pack2(y.x, y.y), pack2(y.z, y.w)};
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) s[slot(BM + crow + 32 * i, ckc)] = rb[i];
    };

    f32x4 acc[MB][2];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb][0] = acc[mb][1] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int wr = (wave >> 1) * WM;
    const int wc = BM + (wave & 1) * 32;
    const int nk = g.K / kBK;
    load(0);
    store(sm[0]);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const u32x4 *cur = sm[kt & 1];
        if (kt + 1 < nk) load((kt + 1) * kBK);
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int kc = s * 4 + (lane >> 4);
            u32x4 fa[MB], fb[2];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) fa[mb] = cur[slot(wr + mb * 16 + (lane & 15), kc)];
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) fb[nb] = cur[slot(wc + nb * 16 + (lane & 15), kc)];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int nb = 0; nb < 2; ++nb) acc[mb][nb] = mfma(fa[mb], fb[nb], acc[mb][nb]);
        }
        if (kt + 1 < nk) store(sm[(kt + 1) & 1]);
        __syncthreads();
    }
    store_tile<EPI, MB, 2>(g, acc, m0 + wr + 4 * (lane >> 4), n0 + (wave & 1) * 32 + (lane & 15), z);
}

// ------------------------------------------------------------------------
// Multi-head causal attention of one chunk request (see MhaArgs).  Grid
// (ceil(c / 128), 16 heads), eight waves; wave w owns tokens i0 + 16 w .. +
// 15.  Keys stream in tiles of 64 through three LDS stages (120 KB, one
// workgroup a CU), register staged one tile ahead; the second half of the
// waves runs its P V one tile behind its scores, so on each SIMD one wave's
// softmax overlaps the other wave's MFMAs.  The K tile holds 64 keys x
// 192 fp16 dims (384 bytes a key, 16-byte chunk c at position
// c ^ ((key >> 1) & 7) inside its group of 8), the V tile 64 keys x 128 fp16
// dims (chunk c at c ^ (2 (key & 7))); both keep the operand reads below free
// of bank conflicts.
//  * S^T = K Q^T (f16 MFMA 16x16x32): lane (g, t) holds the scores of token t
//    against keys 16 kb + 4 g + i of the tile, kb, i = 0..3.
//  * Online softmax per token (running max and sum, accumulators rescaled);
//    the probabilities stay in registers, already in the operand order of
//  * O^T += V^T P^T: slot 8 g + j of a 32-key step is key 4 g + j (j < 4) or
//    16 + 4 g + j - 4; V^T comes from transposing LDS reads in that order.
namespace mha {
constexpr int kKeys = 64;
constexpr int kKRowBytes = 192 * 2;
constexpr int kKTile = kKeys * kKRowBytes;  // 24576
constexpr int kVTile = kKeys * 256;         // 16384
constexpr int kStage = kKTile + kVTile;     // 40960

__device__ __forceinline__ int k_off(int key, int c) { return key * kKRowBytes + ((c ^ ((key >> 1) & 7)) << 4); }
__device__ __forceinline__ int v_off(int key, int c) { return key * 256 + ((c ^ ((key & 7) << 1)) << 4); }

// 8 bf16 -> 8 fp16 (exact inside the fp16 normal range)
__device__ __forceinline__ u32x4 bf16x8_to_f16x8(u32x4 w) {
    u32x4 r;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const auto h = __builtin_amdgcn_cvt_pkrtz(__uint_as_float(w[k] << 16), __uint_as_float(w[k] & 0xffff0000u));
        r[k] = __builtin_bit_cast(uint32_t, h);
    }
    return r;
}

__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
    typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                  0, 0);
}

__device__ __forceinline__ u32x2 read_tr16(const char *p) {
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(p));
    return __builtin_bit_cast(u32x2, v);
}

// max / sum over lanes l, l ^ 16, l ^ 32, l ^ 48 (the four key groups of a token)
__device__ __forceinline__ float max4(float v) {
    v = fmaxf(v, __shfl_xor(v, 16));
    return fmaxf(v, __shfl_xor(v, 32));
}
__device__ __forceinline__ float sum4(float v) {
    v += __shfl_xor(v, 16);
    return v + __shfl_xor(v, 32);
}

__device__ __forceinline__ uint32_t f16x2(float a, float b) {
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    const h2 v = {(_Float16)a, (_Float16)b};
    return __builtin_bit_cast(uint32_t, v);
}
}  // namespace mha

__global__ __launch_bounds__(64 * kMhaWaves) void mha_prefill_kernel(const MhaArgs a) {
    using namespace mha;
    __shared__ __attribute__((aligned(16))) char sm[3 * kStage];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, tl = lane & 15;
    // Workgroups are dealt to the 8 XCDs round-robin: XCD x gets heads 2 x and
    // 2 x + 1 (the keys and values of two heads stay in its L2), token blocks
    // with the most keys first.
    const int nblk = gridDim.x;
    const int lin = blockIdx.x + nblk * blockIdx.y;
    const int sl = lin >> 3;
    const int h = 2 * (lin & 7) + sl / nblk;
    const int i0 = (nblk - 1 - sl % nblk) * kMhaTokens;
    const int tok = i0 + wave * 16 + tl;  // this lane's token
    const int tokc = min(tok, a.c - 1);   // tokens past the chunk repeat its last one; never stored
    const int lim = a.p + tokc;           // last key this token sees
    const int nkeys = a.p + a.c;
    const int ntiles = (a.p + min(i0 + kMhaTokens, a.c) - 1) / kKeys + 1;
    // tiles wholly below the first key some token of this wave cannot see need no mask
    const int wave_lim = a.p + min(i0 + wave * 16, a.c - 1);

    // Q^T operands: lane (g, t) holds dims 32 s + 8 g .. + 7 of token t (s < 4: without position, s = 4, 5: rope)
    u32x4 qf[6];
    {
        const uint16_t *qn = a.qn + ((size_t)(a.row0 + tokc) * 16 + h) * 128 + 8 * g;
        const uint16_t *qr = a.q_abs + ((size_t)(a.row0 + tokc) * 16 + h) * 576 + 512 + 8 * g;
#pragma unroll
        for (int s = 0; s < 4; ++s) qf[s] = bf16x8_to_f16x8(*reinterpret_cast<const u32x4 *>(qn + 32 * s));
#pragma unroll
        for (int s = 0; s < 2; ++s) qf[4 + s] = bf16x8_to_f16x8(*reinterpret_cast<const u32x4 *>(qr + 32 * s));
    }

    // staging per thread and tile: kKLd of the 64 x 24 K chunks (16 from the
    // up-projected keys, 8 rope), kVLd of the 64 x 16 V chunks
    constexpr int kThreads = 64 * kMhaWaves, kKLd = 64 * 24 / kThreads, kVLd = 64 * 16 / kThreads;
    auto load = [&](u32x4(&r)[kKLd + kVLd], int t) {
        const int kb = t * kKeys;
#pragma unroll
        for (int j = 0; j < kKLd; ++j) {
            const int q = tid + kThreads * j, key = min(kb + q / 24, nkeys - 1), cc = q % 24;
            const uint16_t *src = cc < 16 ? a.kv + (size_t)key * 4096 + h * 128 + cc * 8
                                          : a.kpe + (size_t)key * 64 + (cc - 16) * 8;
            r[j] = *reinterpret_cast<const u32x4 *>(src);
        }
#pragma unroll
        for (int j = 0; j < kVLd; ++j) {
            const int q = tid + kThreads * j, key = min(kb + (q >> 4), nkeys - 1), cc = q & 15;
            r[kKLd + j] = *reinterpret_cast<const u32x4 *>(a.kv + (size_t)key * 4096 + 2048 + h * 128 + cc * 8);
        }
    };
    auto store = [&](const u32x4(&r)[kKLd + kVLd], int buf) {
        char *ks = sm + buf * kStage, *vs = ks + kKTile;
#pragma unroll
        for (int j = 0; j < kKLd; ++j) {
            const int q = tid + kThreads * j;
            *reinterpret_cast<u32x4 *>(ks + k_off(q / 24, q % 24)) = r[j];
        }
#pragma unroll
        for (int j = 0; j < kVLd; ++j) {
            const int q = tid + kThreads * j;
            *reinterpret_cast<u32x4 *>(vs + v_off(q >> 4, q & 15)) = r[kKLd + j];
        }
    };

    f32x4 acc[8];
#pragma unroll
    for (int db = 0; db < 8; ++db) acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;

    // V^T operand addresses (lane (g, t): dim 16 db + t of keys 32 m + 4 g + j and 32 m + 16 + 4 g + j)
    const int tr_key = 4 * g + (tl >> 2);
    const int tr_c = (tl & 3) >> 1, tr_b = 8 * (tl & 1);

    u32x4 pb[2];  // probabilities of the last scored tile, operand order of P V
    float alpha;  // and the factor that rescales the accumulators before it
    auto score = [&](int t, int buf) {
        const char *ks = sm + buf * kStage;
        f32x4 st[4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) st[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 6; ++s) {
            u32x4 ka[4];
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) ka[kb] = *reinterpret_cast<const u32x4 *>(ks + k_off(16 * kb + tl, 4 * s + g));
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) st[kb] = mfma16(ka[kb], qf[s], st[kb]);
        }
        // scaled, masked scores; running max
        const int kbase = t * kKeys + 4 * g;
        const bool need_mask = t * kKeys + kKeys - 1 > wave_lim;
        float x[16];
        float mx = -INFINITY;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            float v = st[e >> 2][e & 3] * a.scale_log2;
            if (need_mask && kbase + 16 * (e >> 2) + (e & 3) > lim) v = -INFINITY;
            x[e] = v;
            mx = fmaxf(mx, v);
        }
        mx = max4(mx);
        const float m_new = fmaxf(m_run, mx);
        alpha = __builtin_amdgcn_exp2f(m_run - m_new);  // 0 on the first tile (m_run = -inf)
        m_run = m_new;
        float ps = 0.f;
        float pe[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            pe[e] = __builtin_amdgcn_exp2f(x[e] - m_new);
            ps += pe[e];
        }
        l_run = l_run * alpha + ps;
#pragma unroll
        for (int m = 0; m < 2; ++m)
            pb[m] = u32x4{f16x2(pe[8 * m + 0], pe[8 * m + 1]), f16x2(pe[8 * m + 2], pe[8 * m + 3]),
                          f16x2(pe[8 * m + 4], pe[8 * m + 5]), f16x2(pe[8 * m + 6], pe[8 * m + 7])};
    };
    auto pv = [&](int buf) {
        const char *vs = sm + buf * kStage + kKTile;
#pragma unroll
        for (int db = 0; db < 8; ++db) acc[db] = acc[db] * alpha;
#pragma unroll
        for (int m = 0; m < 2; ++m) {
#pragma unroll
            for (int db = 0; db < 8; ++db) {
                const int k1 = 32 * m + tr_key, k2 = k1 + 16;
                const u32x2 lo = read_tr16(vs + v_off(k1, 2 * db + tr_c) + tr_b);
                const u32x2 hi = read_tr16(vs + v_off(k2, 2 * db + tr_c) + tr_b);
                acc[db] = mfma16(u32x4{lo[0], lo[1], hi[0], hi[1]}, pb[m], acc[db]);
            }
        }
    };

    // Tile t + 1 loads into registers while tile t is processed; the load of
    // the tile past the last one re-reads it (in bounds, never stored), so the
    // loads stay unconditional and the register set is never merged at a
    // branch join (a copy of a register still being loaded waits for every
    // load in flight).  The second half of the waves runs P V one tile
    // behind its scores: each SIMD holds one wave of each half, so one
    // wave's softmax overlaps the other's MFMAs instead of both waiting at
    // the same point between barriers.  Three LDS stages: tile t - 1 stays
    // readable while tile t + 1 is stored.
    const bool lag = wave >= kMhaWaves / 2;
    u32x4 r[kKLd + kVLd];
    load(r, 0);
    store(r, 0);
    __syncthreads();
    int b_prev = 2, b_cur = 0;
    for (int t = 0; t < ntiles; ++t) {
        const int b_next = b_cur == 2 ? 0 : b_cur + 1;
        load(r, min(t + 1, ntiles - 1));
        if (!lag) {
            score(t, b_cur);
            pv(b_cur);
        } else {
            if (t > 0) pv(b_prev);
            score(t, b_cur);
        }
        if (t + 1 < ntiles) store(r, b_next);
        __syncthreads();
        b_prev = b_cur;
        b_cur = b_next;
    }
    if (lag) pv(b_prev);
    const float l = sum4(l_run);
    if (tok < a.c) {
        const float inv = 1.f / l;
        uint16_t *dst = a.o + (size_t)(a.row0 + tok) * 2048 + h * 128 + 4 * g;
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const f32x4 v = acc[db] * inv;
            *reinterpret_cast<u32x2 *>(dst + 16 * db) = u32x2{pack2(v[0], v[1]), pack2(v[2], v[3])};
        }
    }
}

template <int BM, int BN, int D>
hipError_t launch_ring(const GemmArgs &g, int epi, dim3 grid, hipStream_t s) {
    if (epi == kStoreF16) gemm_ring_kernel<BM, BN, D, kStoreF16><<<grid, 256, 0, s>>>(g);
    else if (epi == kStoreBf16) gemm_ring_kernel<BM, BN, D, kStoreBf16><<<grid, 256, 0, s>>>(g);
    else if (epi == kStoreF32) gemm_ring_kernel<BM, BN, D, kStoreF32><<<grid, 256, 0, s>>>(g);
    else if (epi == kQkvSplit) gemm_ring_kernel<BM, BN, D, kQkvSplit><<<grid, 256, 0, s>>>(g);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

template <int BM, int BN, int WR, int WC>
hipError_t launch_reg(const GemmArgs &g, int epi, dim3 grid, hipStream_t s) {
    constexpr int NT = 64 * WR * WC;
    if (epi == kStoreBf16) gemm_reg_kernel<BM, BN, WR, WC, kStoreBf16><<<grid, NT, 0, s>>>(g);
    else if (epi == kStoreF32) gemm_reg_kernel<BM, BN, WR, WC, kStoreF32><<<grid, NT, 0, s>>>(g);
    else if (epi == kQkvSplit) gemm_reg_kernel<BM, BN, WR, WC, kQkvSplit><<<grid, NT, 0, s>>>(g);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

template <int BM>
hipError_t launch_f32a(const GemmArgs &g, int epi, dim3 grid, hipStream_t s) {
    if (epi == kStoreBf16) gemm_f32a_kernel<BM, kStoreBf16><<<grid, 256, 0, s>>>(g);
    else if (epi == kStoreF32) gemm_f32a_kernel<BM, kStoreF32><<<grid, 256, 0, s>>>(g);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace

hipError_t launch_mha_prefill(const MhaArgs &a, hipStream_t s) {
    if (a.c <= 0) return hipSuccess;
    if (a.p < 0) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((a.c + kMhaTokens - 1) / kMhaTokens), 16);
    mha_prefill_kernel<<<grid, 64 * kMhaWaves, 0, s>>>(a);
    return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs &g, const GemmShape &t, bool a_f32, int batch, hipStream_t s) {
    if (g.M <= 0 || batch <= 0) return hipSuccess;
    if (g.K % kBK != 0 || g.K <= 0 || g.N <= 0) return hipErrorInvalidValue;
    const int bn = a_f32 ? kBN : t.bn;
    const long long tiles = (long long)((g.M + t.bm - 1) / t.bm) * ((g.N + bn - 1) / bn) + g.rope_wgs + g.keys_wgs;
    if (tiles > 0x7FFFFFFF || g.rope_wgs < 0 || g.keys_wgs < 0 || (g.rope_wgs > 0 && g.keys_wgs > 0))
        return hipErrorInvalidValue;
    const dim3 grid((unsigned)tiles, 1, (unsigned)batch);
    if (a_f32 || t.depth == 0) {
        // gathered rows and fp16 output exist in the LDS-ring kernel only
        if (g.a_bt != nullptr || t.epi == kStoreF16) return hipErrorInvalidValue;
    }
    if (a_f32) {
        if (g.rope_wgs != 0 || g.keys_wgs != 0) return hipErrorInvalidValue;
        if (g.N % kBN != 0) return hipErrorInvalidValue;
        switch (t.bm) {
            case 32: return launch_f32a<32>(g, t.epi, grid, s);
            case 64: return launch_f32a<64>(g, t.epi, grid, s);
            case 128: return launch_f32a<128>(g, t.epi, grid, s);
            default: return hipErrorInvalidValue;
        }
    }
    // BN = 64 tiles must not straddle a head (the split epilogue handles any column, the others any N)
    const int key = t.bm * 1000 + t.bn * 10 + t.depth;
    switch (key) {
        case 128 * 1000 + 256 * 10 + 0: return launch_reg<128, 256, 2, 4>(g, t.epi, grid, s);
        case 256 * 1000 + 128 * 10 + 0: return launch_reg<256, 128, 4, 2>(g, t.epi, grid, s);
        case 128 * 1000 + 128 * 10 + 0: return launch_reg<128, 128, 2, 2>(g, t.epi, grid, s);
        case 64 * 1000 + 128 * 10 + 0: return launch_reg<64, 128, 2, 2>(g, t.epi, grid, s);
        case 32 * 1000 + 128 * 10 + 0: return launch_reg<32, 128, 2, 2>(g, t.epi, grid, s);
        case 32 * 1000 + 64 * 10 + 6: return launch_ring<32, 64, 6>(g, t.epi, grid, s);
        case 64 * 1000 + 64 * 10 + 4: return launch_ring<64, 64, 4>(g, t.epi, grid, s);
        case 128 * 1000 + 64 * 10 + 3: return launch_ring<128, 64, 3>(g, t.epi, grid, s);
        case 32 * 1000 + 128 * 10 + 4: return launch_ring<32, 128, 4>(g, t.epi, grid, s);
        case 64 * 1000 + 128 * 10 + 3: return launch_ring<64, 128, 3>(g, t.epi, grid, s);
        case 128 * 1000 + 128 * 10 + 2: return launch_ring<128, 128, 2>(g, t.epi, grid, s);
        case 128 * 1000 + 128 * 10 + 3: return launch_ring<128, 128, 3>(g, t.epi, grid, s);
        default: return hipErrorInvalidValue;
    }
}


}  // namespace proj
