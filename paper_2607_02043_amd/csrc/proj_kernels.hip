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

// Workgroups past the tiles run the launch's rope / norm rows (z = 0) or
// nothing; true when this workgroup is one of them.
__device__ __forceinline__ bool is_rope_wg(const GemmArgs &g, int BM, int BN) {
    const int tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
    if ((int)blockIdx.x < tiles) return false;
    if (blockIdx.z == 0) rope_norm_rows(g.rope, blockIdx.x - tiles);
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
            src[i] = static_cast<const uint16_t *>(g.a) + z * g.a_bstride + (long long)r * g.lda + kc * 8;
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

template <int BM, int BN, int D>
hipError_t launch_ring(const GemmArgs &g, int epi, dim3 grid, hipStream_t s) {
    if (epi == kStoreBf16) gemm_ring_kernel<BM, BN, D, kStoreBf16><<<grid, 256, 0, s>>>(g);
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

hipError_t launch_gemm(const GemmArgs &g, const GemmShape &t, bool a_f32, int batch, hipStream_t s) {
    if (g.M <= 0 || batch <= 0) return hipSuccess;
    if (g.K % kBK != 0 || g.K <= 0 || g.N <= 0) return hipErrorInvalidValue;
    const int bn = a_f32 ? kBN : t.bn;
    const long long tiles = (long long)((g.M + t.bm - 1) / t.bm) * ((g.N + bn - 1) / bn) + g.rope_wgs;
    if (tiles > 0x7FFFFFFF || g.rope_wgs < 0) return hipErrorInvalidValue;
    const dim3 grid((unsigned)tiles, 1, (unsigned)batch);
    if (a_f32) {
        if (g.rope_wgs != 0) return hipErrorInvalidValue;
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
