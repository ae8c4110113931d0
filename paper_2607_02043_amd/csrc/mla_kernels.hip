// gfx950 kernels of libmlastep: latent append, mixed-step latent attention
// (decode rows and chunked-prefill rows of one step), split merge.
//
// The step is the one a decode node runs when it serves deflected prefill
// chunks next to its in-flight decodes (section 2.3; section 4.3.1, Eq. 4 of
// the paper); the head shapes are those of the served model's absorbed latent
// attention (DeepSeek-V2-Lite, section 6).
//
// Work decomposition.  Every request is cut into work items:
//   * decode request (c = 1): key ranges of ks_dec keys (split-KV).  A
//     workgroup streams its range through a 4-deep ring of 32-key tiles that
//     the wavefronts fill asynchronously (global -> LDS DMA); all four waves
//     score the tile (16 heads = the MFMA's 16 columns) and each wave
//     accumulates one 128-wide slice of the 512 value dims.
//   * chunk request (c > 1): blocks of 4 query tokens (one per wave, 16 head
//     rows each) times key ranges of ks_chunk keys.  Tiles go through a
//     3-deep DMA ring; each tile's value part is converted once to fp16 and
//     transposed in LDS so that P*V runs on fp16 MFMA.
// Items of one request that split the key range write fp32 partials
// (unnormalised sum, running max and sum in log2 units); the merge kernel
// combines them in a fixed order, so results are run-to-run deterministic and
// do not depend on the physical page order.
#include "mla_kernels.h"

#include <math.h>

namespace mla {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kTileBytes = kKeysPerTile * kRowBytes;          // 36864
constexpr int kChunksPerRow = kRowBytes / 16;                 // 72 16-byte chunks
constexpr int kDmaPerTile = kTileBytes / (kThreads * 16);     // 9 per thread
constexpr int kDecRing = 4;
constexpr int kChunkRing = 3;
constexpr int kVtStride = 80;                                 // bytes per dv row of V^T (32 fp16 + pad)
constexpr int kVtBytes = kDv * kVtStride;                     // 40960
constexpr int kDecLds = kDecRing * kTileBytes;                // 147456
constexpr int kChunkLds = kChunkRing * kTileBytes + kVtBytes; // 151552
constexpr int kMainLds = kDecLds > kChunkLds ? kDecLds : kChunkLds;
constexpr float kNegInf = -INFINITY;
constexpr float kLn2 = 0.69314718055994530942f;

static_assert(kTileBytes % (kThreads * 16) == 0, "tile must split into whole DMA rounds");

// ---------------------------------------------------------------- helpers
__device__ __forceinline__ float bf16_bits_to_float(uint32_t b) { return __uint_as_float(b << 16); }

__device__ __forceinline__ uint32_t lds_addr(const void *p) {
    return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
}

// One 16-byte global -> LDS DMA per lane: lane i writes LDS bytes
// [base + 16 i, base + 16 i + 16).  `base` must be wave-uniform.  Issued with
// inline assembly so that the compiler does not drain the whole ring before
// every barrier; completion is tracked by hand with wait_vm below.
__device__ __forceinline__ void lds_dma16(const void *gsrc, uint32_t lds_base) {
    asm volatile(
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off\n\t"
        :
        : "{m0}"(lds_base), "v"(gsrc)
        : "memory");
}

// Wait until at most `newer_tiles` tiles of DMA issued after the awaited one
// are still in flight (9 DMA instructions per tile and wave).
__device__ __forceinline__ void wait_dma_tiles(int newer_tiles) {
    if (newer_tiles <= 0)
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    else if (newer_tiles == 1)
        asm volatile("s_waitcnt vmcnt(9)" ::: "memory");
    else
        asm volatile("s_waitcnt vmcnt(18)" ::: "memory");
}

__device__ __forceinline__ f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_f16(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ float wave_max16(float v) {  // reduce over lanes l, l^16, l^32, l^48
    v = fmaxf(v, __shfl_xor(v, 16, 64));
    v = fmaxf(v, __shfl_xor(v, 32, 64));
    return v;
}
__device__ __forceinline__ float wave_sum16(float v) {
    v += __shfl_xor(v, 16, 64);
    v += __shfl_xor(v, 32, 64);
    return v;
}

// LDS byte offset of 16-byte chunk c of key k inside a tile.  Chunk
// positions are xor-swizzled with the key's low 3 bits so that 8 lanes that
// read the same chunk of 8 consecutive keys hit 8 different bank groups.
__device__ __forceinline__ int tile_off(int k, int c) { return (k * kChunksPerRow + (c ^ (k & 7))) * 16; }

// ------------------------------------------------------ work-item lookup
// Items of one kind are numbered request by request; request r owns
// count(r) consecutive items.  The workgroup scans the per-request counts
// (256 requests per round) and finds the request owning item `target`.
struct ReqLens {
    const int32_t *cu_q;
    const int32_t *prefix;
};

template <typename CountFn>
__device__ bool locate_item(int target, int num_reqs, const ReqLens &rl, CountFn count, int *s_tmp,
                            int &req, int &local) {
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    if (tid == 0) s_tmp[4] = -1;
    int running = 0;
    for (int base = 0; base < num_reqs; base += kThreads) {
        const int r = base + tid;
        int cnt = 0;
        if (r < num_reqs) {
            const int c = rl.cu_q[r + 1] - rl.cu_q[r];
            cnt = count(rl.prefix[r], c);
        }
        int inc = cnt;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int v = __shfl_up(inc, d, 64);
            if (lane >= d) inc += v;
        }
        if (lane == 63) s_tmp[wv] = inc;
        __syncthreads();
        int off = 0, total = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int t = s_tmp[k];
            off += (k < wv) ? t : 0;
            total += t;
        }
        inc += off;
        const int exc = inc - cnt;
        if (cnt > 0 && target >= running + exc && target < running + inc) {
            s_tmp[4] = r;
            s_tmp[5] = target - running - exc;
        }
        __syncthreads();
        if (s_tmp[4] >= 0) {
            req = s_tmp[4];
            local = s_tmp[5];
            return true;
        }
        running += total;
    }
    return false;
}

__device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

struct ChunkCount {
    int ks;
    __device__ int operator()(int p, int c) const {
        return c > 1 ? ceil_div(c, kChunkBlockTokens) * ceil_div(p + c, ks) : 0;
    }
};
struct DecCount {
    int ks;
    __device__ int operator()(int p, int c) const { return c == 1 ? ceil_div(p + 1, ks) : 0; }
};

struct ChunkItem {
    int r, p, c, row0, i0, i1, k0, k1, nks_eff;
};

__device__ __forceinline__ ChunkItem decode_chunk_item(const AttnArgs &a, int r, int local) {
    ChunkItem it;
    it.r = r;
    it.p = a.prefix[r];
    it.row0 = a.cu_q[r];
    it.c = a.cu_q[r + 1] - it.row0;
    const int nrb = ceil_div(it.c, kChunkBlockTokens);
    const int nks = ceil_div(it.p + it.c, a.ks_chunk);
    const int rb = nrb - 1 - local / nks;  // longest rows first
    const int ks = local % nks;
    it.i0 = rb * kChunkBlockTokens;
    it.i1 = min(it.i0 + kChunkBlockTokens, it.c);
    const int klim = it.p + it.i1;
    it.nks_eff = ceil_div(klim, a.ks_chunk);
    it.k0 = ks * a.ks_chunk;
    it.k1 = min(klim, it.k0 + a.ks_chunk);
    return it;
}

// Page ids of logical pages [lp0, lp0 + n) of a request into LDS; an id
// outside the pool is replaced by page 0 so no access leaves the pool.
__device__ __forceinline__ void load_page_window(const AttnArgs &a, int r, int lp0, int n, int *s_pages) {
    const int32_t *row = a.bt + (size_t)r * a.max_pages;
    n = min(n, kPageWindow);
    for (int i = threadIdx.x; i < n; i += kThreads) {
        const int lp = lp0 + i;
        int pg = lp < a.max_pages ? row[lp] : 0;
        s_pages[i] = ((unsigned)pg < (unsigned)a.num_pages) ? pg : 0;
    }
}

// Issue the DMA of one 32-key tile (keys kbase .. kbase+31, clamped to the
// last valid key k1-1 so every byte read is a finite cached latent).
__device__ __forceinline__ void issue_tile(const AttnArgs &a, const int *s_pages, int lp0, int kbase, int k1,
                                           uint32_t lds_tile, int wv, int lane) {
    const char *kv = reinterpret_cast<const char *>(a.kv);
#pragma unroll
    for (int i = 0; i < kDmaPerTile; ++i) {
        const int seg = i * 4 + wv;
        const int u = seg * 64 + lane;
        const int kk = u / kChunksPerRow;
        const int c = (u - kk * kChunksPerRow) ^ (kk & 7);
        int key = kbase + kk;
        key = key < k1 ? key : k1 - 1;
        const int page = s_pages[min((key >> a.log2_page) - lp0, kPageWindow - 1)];
        const size_t slot = (size_t)page * a.page_size + (key & (a.page_size - 1));
        lds_dma16(kv + slot * kRowBytes + c * 16, __builtin_amdgcn_readfirstlane(lds_tile + seg * 1024));
    }
}

// S^T (32 keys x 16 heads) of one tile against the query operand of one
// token: lane l gets s[kt][i] = score of key 16 kt + 4 (l/16) + i, head l%16.
__device__ __forceinline__ void score_tile(const char *tile, const u32x4 *qreg, int lane, f32x4 s[2]) {
    const int g = lane >> 4;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
        const int key = kt * 16 + (lane & 15);
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < 18; ++st) {
            const u32x4 av = *reinterpret_cast<const u32x4 *>(tile + tile_off(key, st * 4 + g));
            acc = mfma_bf16(av, qreg[st], acc);
        }
        s[kt] = acc;
    }
}

// ------------------------------------------------------------ decode path
__device__ void decode_item(const AttnArgs &a, int item, char *smem, int *s_tmp, int *s_pages) {
    int r, ks;
    if (!locate_item(item, a.num_reqs, ReqLens{a.cu_q, a.prefix}, DecCount{a.ks_dec}, s_tmp, r, ks)) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, h = lane & 15;
    const int p = a.prefix[r];
    const int row = a.cu_q[r];
    if (p < 0 || row < 0 || row >= a.num_rows) return;  // device lengths disagree with the host's
    const int n_keys = p + 1;
    const int nks = ceil_div(n_keys, a.ks_dec);
    const int k0 = ks * a.ks_dec;
    const int k1 = min(n_keys, k0 + a.ks_dec);
    const int ntiles = ceil_div(k1 - k0, kKeysPerTile);
    if (nks > 1 && a.ws_dec_o == nullptr) return;
    const int lp0 = k0 >> a.log2_page;
    load_page_window(a, r, lp0, ((k1 - 1) >> a.log2_page) - lp0 + 1, s_pages);
    __syncthreads();

    const uint32_t ring = lds_addr(smem);
    for (int t = 0; t < kDecRing - 1 && t < ntiles; ++t)
        issue_tile(a, s_pages, lp0, k0 + t * kKeysPerTile, k1, ring + t * kTileBytes, wv, lane);

    u32x4 qreg[18];
    {
        const uint16_t *qp = a.q + ((size_t)row * kHeads + h) * kDqk + g * 8;
#pragma unroll
        for (int st = 0; st < 18; ++st) qreg[st] = *reinterpret_cast<const u32x4 *>(qp + st * 32);
    }
    // Drain the query loads with the ring prologue: the compiler would otherwise
    // wait for its own loads with vmcnt(0) inside the pipelined loop.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

    f32x4 acc[8];
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = kNegInf, l_run = 0.f;

    for (int t = 0; t < ntiles; ++t) {
        wait_dma_tiles(min(kDecRing - 2, ntiles - 1 - t));
        __syncthreads();
        if (t + kDecRing - 1 < ntiles)
            issue_tile(a, s_pages, lp0, k0 + (t + kDecRing - 1) * kKeysPerTile, k1,
                       ring + ((t + kDecRing - 1) % kDecRing) * kTileBytes, wv, lane);
        const char *tile = smem + (t % kDecRing) * kTileBytes;
        const int kbase = k0 + t * kKeysPerTile;

        f32x4 s[2];
        score_tile(tile, qreg, lane, s);
        float x[8];
        float mt = kNegInf;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int key = kbase + 16 * (j >> 2) + 4 * g + (j & 3);
            const float v = s[j >> 2][j & 3] * a.scale_log2;
            x[j] = key < k1 ? v : kNegInf;
            mt = fmaxf(mt, x[j]);
        }
        mt = wave_max16(mt);
        const float m_new = fmaxf(m_run, mt);
        const float alpha = exp2f(m_run - m_new);
        m_run = m_new;
        float ps = 0.f;
        uint32_t ph[4], pl[4];
#pragma unroll
        for (int j = 0; j < 8; j += 2) {
            const float p0 = exp2f(x[j] - m_new), p1 = exp2f(x[j + 1] - m_new);
            ps += p0 + p1;
            const __bf16 h0 = (__bf16)p0, h1 = (__bf16)p1;
            const __bf16 l0 = (__bf16)(p0 - (float)h0), l1 = (__bf16)(p1 - (float)h1);
            ph[j >> 1] = (uint32_t)__builtin_bit_cast(uint16_t, h0) | ((uint32_t)__builtin_bit_cast(uint16_t, h1) << 16);
            pl[j >> 1] = (uint32_t)__builtin_bit_cast(uint16_t, l0) | ((uint32_t)__builtin_bit_cast(uint16_t, l1) << 16);
        }
        l_run = l_run * alpha + ps;
        const u32x4 bh = {ph[0], ph[1], ph[2], ph[3]};
        const u32x4 bl = {pl[0], pl[1], pl[2], pl[3]};
#pragma unroll
        for (int mt2 = 0; mt2 < 8; ++mt2) {
            const int dv = wv * 128 + mt2 * 16 + (lane & 15);
            const int c = dv >> 3, e = dv & 7;
            uint32_t w[4];
#pragma unroll
            for (int j = 0; j < 8; j += 2) {
                const int k0j = 16 * (j >> 2) + 4 * g + (j & 3);
                const int k1j = k0j + 1;
                const uint32_t v0 = *reinterpret_cast<const uint16_t *>(tile + tile_off(k0j, c) + e * 2);
                const uint32_t v1 = *reinterpret_cast<const uint16_t *>(tile + tile_off(k1j, c) + e * 2);
                w[j >> 1] = v0 | (v1 << 16);
            }
            const u32x4 av = {w[0], w[1], w[2], w[3]};
            acc[mt2] = acc[mt2] * alpha;
            acc[mt2] = mfma_bf16(av, bh, acc[mt2]);
            acc[mt2] = mfma_bf16(av, bl, acc[mt2]);
        }
    }

    const float l_tot = wave_sum16(l_run);
    if (nks == 1) {
        const float inv = 1.f / l_tot;
        if (a.out_bf16) {
            uint16_t *o = reinterpret_cast<uint16_t *>(a.out) + ((size_t)row * kHeads + h) * kDv;
#pragma unroll
            for (int mt2 = 0; mt2 < 8; ++mt2) {
                const int dv = wv * 128 + mt2 * 16 + 4 * g;
                uint32_t w0 = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[mt2][0] * inv)) |
                              ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[mt2][1] * inv)) << 16);
                uint32_t w1 = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[mt2][2] * inv)) |
                              ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[mt2][3] * inv)) << 16);
                *reinterpret_cast<u32x2 *>(o + dv) = u32x2{w0, w1};
            }
        } else {
            float *o = reinterpret_cast<float *>(a.out) + ((size_t)row * kHeads + h) * kDv;
#pragma unroll
            for (int mt2 = 0; mt2 < 8; ++mt2) {
                const int dv = wv * 128 + mt2 * 16 + 4 * g;
                *reinterpret_cast<f32x4 *>(o + dv) = acc[mt2] * inv;
            }
        }
        if (a.lse && wv == 0 && g == 0) a.lse[(size_t)row * kHeads + h] = (m_run + log2f(l_tot)) * kLn2;
    } else {
        float *po = a.ws_dec_o + ((size_t)item * kHeads + h) * kDv;
#pragma unroll
        for (int mt2 = 0; mt2 < 8; ++mt2) {
            const int dv = wv * 128 + mt2 * 16 + 4 * g;
            *reinterpret_cast<f32x4 *>(po + dv) = acc[mt2];
        }
        if (wv == 0 && g == 0) {
            a.ws_dec_ml[((size_t)item * kHeads + h) * 2 + 0] = m_run;
            a.ws_dec_ml[((size_t)item * kHeads + h) * 2 + 1] = l_tot;
        }
    }
}

// ------------------------------------------------------------- chunk path
// Convert the value part of a tile (keys 0..31, dims 0..511, bf16) into a
// transposed fp16 copy vt[dv][slot] (row stride 80 bytes, four 16-byte slot
// groups per row, group q of row dv stored at position q ^ ((dv / 8) % 4) so
// that lanes writing rows 8 apart spread over the banks).  Slot order matches
// the score layout: slot 8 g + 4 kt + i holds key 16 kt + 4 g + i, so the
// probabilities a lane already holds are the MFMA's B operand as they are.
__device__ __forceinline__ int vt_off(int dv, int slot) {
    return dv * kVtStride + ((((slot >> 3) ^ (dv >> 3)) & 3) << 4) + (slot & 7) * 2;
}

__device__ __forceinline__ void convert_values(const char *tile, char *vt, int tid) {
#pragma unroll
    for (int rep = 0; rep < 2; ++rep) {
        const int pr = tid + rep * kThreads;
        const int c = pr & 63;   // value chunk: dims 8c .. 8c+7
        const int qd = pr >> 6;  // key quad: keys 4 qd .. 4 qd + 3
        u32x4 kq[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
            kq[kk] = *reinterpret_cast<const u32x4 *>(tile + tile_off(qd * 4 + kk, c));
        const int slot = 8 * (qd & 3) + 4 * (qd >> 2);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            f16x4 hv;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const uint32_t word = kq[kk][e >> 1];
                const uint32_t bits = (e & 1) ? (word >> 16) : (word & 0xffffu);
                hv[kk] = (_Float16)bf16_bits_to_float(bits);
            }
            *reinterpret_cast<u32x2 *>(vt + vt_off(8 * c + e, slot)) = __builtin_bit_cast(u32x2, hv);
        }
    }
}

__device__ void chunk_item(const AttnArgs &a, int item, char *smem, int *s_tmp, int *s_pages) {
    int r, local;
    if (!locate_item(item, a.num_reqs, ReqLens{a.cu_q, a.prefix}, ChunkCount{a.ks_chunk}, s_tmp, r, local)) return;
    const ChunkItem it = decode_chunk_item(a, r, local);
    if (it.k0 >= it.k1) return;  // key range past this block's causal limit
    if (it.p < 0 || it.row0 < 0 || it.row0 + it.i1 > a.num_rows) return;
    if (it.nks_eff > 1 && a.ws_chunk_o == nullptr) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, h = lane & 15;
    const int my_i = it.i0 + wv;            // this wave's token within the request
    const bool active = my_i < it.i1;
    const int my_lim = it.p + my_i;         // last key this token may see
    const int ntiles = ceil_div(it.k1 - it.k0, kKeysPerTile);
    const int lp0 = it.k0 >> a.log2_page;
    load_page_window(a, r, lp0, ((it.k1 - 1) >> a.log2_page) - lp0 + 1, s_pages);
    __syncthreads();

    const uint32_t ring = lds_addr(smem);
    char *vt = smem + kChunkRing * kTileBytes;
    for (int t = 0; t < kChunkRing - 1 && t < ntiles; ++t)
        issue_tile(a, s_pages, lp0, it.k0 + t * kKeysPerTile, it.k1, ring + t * kTileBytes, wv, lane);

    u32x4 qreg[18];
    const int qrow = it.row0 + (active ? my_i : it.i0);
    {
        const uint16_t *qp = a.q + ((size_t)qrow * kHeads + h) * kDqk + g * 8;
#pragma unroll
        for (int st = 0; st < 18; ++st) qreg[st] = *reinterpret_cast<const u32x4 *>(qp + st * 32);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    f32x4 acc[32];
#pragma unroll
    for (int mt = 0; mt < 32; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_ref = kNegInf, l_run = 0.f;

    for (int t = 0; t < ntiles; ++t) {
        wait_dma_tiles(min(kChunkRing - 2, ntiles - 1 - t));
        __syncthreads();
        if (t + kChunkRing - 1 < ntiles)
            issue_tile(a, s_pages, lp0, it.k0 + (t + kChunkRing - 1) * kKeysPerTile, it.k1,
                       ring + ((t + kChunkRing - 1) % kChunkRing) * kTileBytes, wv, lane);
        const char *tile = smem + (t % kChunkRing) * kTileBytes;
        convert_values(tile, vt, tid);
        __syncthreads();
        if (!active) continue;
        const int kbase = it.k0 + t * kKeysPerTile;
        f32x4 s[2];
        score_tile(tile, qreg, lane, s);
        float x[8];
        float mt = kNegInf;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int key = kbase + 16 * (j >> 2) + 4 * g + (j & 3);
            const float v = s[j >> 2][j & 3] * a.scale_log2;
            x[j] = (key < it.k1 && key <= my_lim) ? v : kNegInf;
            mt = fmaxf(mt, x[j]);
        }
        mt = wave_max16(mt);
        // Lazy rescale: keep the reference max unless the tile max exceeds it
        // by more than 2^8 (probabilities then stay <= 256, exact range for fp16).
        const bool grow = mt > m_ref + 8.f;
        if (__builtin_amdgcn_ballot_w64(grow) != 0) {
            const float m_new = fmaxf(m_ref, mt);
            const float alpha = (m_ref == kNegInf) ? 0.f : exp2f(m_ref - m_new);
#pragma unroll
            for (int mt2 = 0; mt2 < 32; ++mt2) acc[mt2] = acc[mt2] * alpha;
            l_run *= alpha;
            m_ref = m_new;
        }
        float ps = 0.f;
        f16x8 pv;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float pj = (x[j] == kNegInf) ? 0.f : exp2f(x[j] - m_ref);
            const _Float16 hj = (_Float16)pj;
            ps += (float)hj;  // the normaliser sums exactly the weights the MFMA uses
            pv[j] = hj;
        }
        l_run += ps;
        const u32x4 bop = __builtin_bit_cast(u32x4, pv);
#pragma unroll
        for (int mt2 = 0; mt2 < 32; ++mt2) {
            const int dv = mt2 * 16 + (lane & 15);
            const u32x4 av = *reinterpret_cast<const u32x4 *>(vt + vt_off(dv, 8 * g));
            acc[mt2] = mfma_f16(av, bop, acc[mt2]);
        }
    }
    if (!active) return;

    const float l_tot = wave_sum16(l_run);
    const int row = it.row0 + my_i;
    if (it.nks_eff == 1) {
        const float inv = 1.f / l_tot;
        if (a.out_bf16) {
            uint16_t *o = reinterpret_cast<uint16_t *>(a.out) + ((size_t)row * kHeads + h) * kDv;
#pragma unroll
            for (int mt2 = 0; mt2 < 32; ++mt2) {
                const int dv = mt2 * 16 + 4 * g;
                uint32_t w0 = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[mt2][0] * inv)) |
                              ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[mt2][1] * inv)) << 16);
                uint32_t w1 = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[mt2][2] * inv)) |
                              ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[mt2][3] * inv)) << 16);
                *reinterpret_cast<u32x2 *>(o + dv) = u32x2{w0, w1};
            }
        } else {
            float *o = reinterpret_cast<float *>(a.out) + ((size_t)row * kHeads + h) * kDv;
#pragma unroll
            for (int mt2 = 0; mt2 < 32; ++mt2) {
                const int dv = mt2 * 16 + 4 * g;
                *reinterpret_cast<f32x4 *>(o + dv) = acc[mt2] * inv;
            }
        }
        if (a.lse && g == 0) a.lse[(size_t)row * kHeads + h] = (m_ref + log2f(l_tot)) * kLn2;
    } else {
        const size_t prow = (size_t)item * kChunkBlockTokens + wv;
        float *po = a.ws_chunk_o + (prow * kHeads + h) * kDv;
#pragma unroll
        for (int mt2 = 0; mt2 < 32; ++mt2) {
            const int dv = mt2 * 16 + 4 * g;
            *reinterpret_cast<f32x4 *>(po + dv) = acc[mt2];
        }
        if (g == 0) {
            a.ws_chunk_ml[(prow * kHeads + h) * 2 + 0] = m_ref;
            a.ws_chunk_ml[(prow * kHeads + h) * 2 + 1] = l_tot;
        }
    }
}

__global__ __launch_bounds__(kThreads, 1) void attention_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) char smem[kMainLds];
    __shared__ int s_tmp[8];
    __shared__ int s_pages[kPageWindow];
    const int b = blockIdx.x;
    if (b < a.n_chunk_items)
        chunk_item(a, b, smem, s_tmp, s_pages);
    else
        decode_item(a, b - a.n_chunk_items, smem, s_tmp, s_pages);
}

// ------------------------------------------------------------------ merge
// Combine the key-split partials of one row: m_s, l_s in log2 units, o_s
// unnormalised.  256 threads: head = tid / 16, dims (tid % 16) * 32 .. +32.
__device__ void merge_row(const float *po, const float *pml, size_t stride_o, size_t stride_ml, int nsplit,
                          void *out, int out_bf16, float *lse, int row) {
    const int tid = threadIdx.x;
    const int hh = tid >> 4, d0 = (tid & 15) * 32;
    float mmax = kNegInf;
    for (int s = 0; s < nsplit; ++s) mmax = fmaxf(mmax, pml[s * stride_ml + hh * 2]);
    float denom = 0.f;
    f32x4 o[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) o[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < nsplit; ++s) {
        const float ms = pml[s * stride_ml + hh * 2];
        const float w = (ms == kNegInf) ? 0.f : exp2f(ms - mmax);
        denom += w * pml[s * stride_ml + hh * 2 + 1];
        const f32x4 *src = reinterpret_cast<const f32x4 *>(po + s * stride_o + hh * kDv + d0);
#pragma unroll
        for (int k = 0; k < 8; ++k) o[k] += w * src[k];
    }
    const float inv = 1.f / denom;
    if (out_bf16) {
        uint16_t *dst = reinterpret_cast<uint16_t *>(out) + ((size_t)row * kHeads + hh) * kDv + d0;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const f32x4 v = o[k] * inv;
            uint32_t w0 = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[0]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[1]) << 16);
            uint32_t w1 = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[2]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[3]) << 16);
            *reinterpret_cast<u32x2 *>(dst + 4 * k) = u32x2{w0, w1};
        }
    } else {
        f32x4 *dst = reinterpret_cast<f32x4 *>(reinterpret_cast<float *>(out) + ((size_t)row * kHeads + hh) * kDv + d0);
#pragma unroll
        for (int k = 0; k < 8; ++k) dst[k] = o[k] * inv;
    }
    if (lse && (tid & 15) == 0) lse[(size_t)row * kHeads + hh] = (mmax + log2f(denom)) * kLn2;
}

__global__ __launch_bounds__(kThreads) void combine_kernel(AttnArgs a) {
    __shared__ int s_tmp[8];
    const int b = blockIdx.x;
    int r, local;
    if (b < a.n_chunk_items) {
        if (!locate_item(b, a.num_reqs, ReqLens{a.cu_q, a.prefix}, ChunkCount{a.ks_chunk}, s_tmp, r, local)) return;
        const ChunkItem it = decode_chunk_item(a, r, local);
        if (it.k0 != 0 || it.nks_eff <= 1 || a.ws_chunk_o == nullptr) return;
        if (it.row0 < 0 || it.row0 + it.i1 > a.num_rows) return;
        const size_t so = (size_t)kChunkBlockTokens * kPartialFloats;
        const size_t sm = (size_t)kChunkBlockTokens * kPartialStats;
        for (int i = it.i0; i < it.i1; ++i) {
            const size_t prow = (size_t)b * kChunkBlockTokens + (i - it.i0);
            merge_row(a.ws_chunk_o + prow * kPartialFloats, a.ws_chunk_ml + prow * kPartialStats, so, sm, it.nks_eff,
                      a.out, a.out_bf16, a.lse, it.row0 + i);
        }
    } else {
        const int item = b - a.n_chunk_items;
        if (!locate_item(item, a.num_reqs, ReqLens{a.cu_q, a.prefix}, DecCount{a.ks_dec}, s_tmp, r, local)) return;
        const int nks = ceil_div(a.prefix[r] + 1, a.ks_dec);
        if (local != 0 || nks <= 1 || a.ws_dec_o == nullptr) return;
        if (a.cu_q[r] < 0 || a.cu_q[r] >= a.num_rows) return;
        merge_row(a.ws_dec_o + (size_t)item * kPartialFloats, a.ws_dec_ml + (size_t)item * kPartialStats,
                  kPartialFloats, kPartialStats, nks, a.out, a.out_bf16, a.lse, a.cu_q[r]);
    }
}

// ----------------------------------------------------------------- append
// Request of a global row: wave-parallel 64-ary search of cu_q.
__device__ __forceinline__ int find_request(const int32_t *cu_q, int num_reqs, int row, int lane) {
    int lo = 0, hi = num_reqs;  // cu_q[lo] <= row < cu_q[hi]
    while (hi - lo > 1) {
        const int step = ceil_div(hi - lo, 64);
        const int idx = lo + lane * step;
        const bool le = idx < hi && cu_q[idx] <= row;
        const uint64_t m = __builtin_amdgcn_ballot_w64(le);
        if (m == 0) break;
        const int last = 63 - __builtin_clzll(m);
        lo = lo + last * step;
        hi = min(hi, lo + step);
    }
    return lo;
}

constexpr int kAppendRowsPerWave = 4;

__global__ __launch_bounds__(kThreads) void append_kernel(AppendArgs a) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int row_base = (blockIdx.x * 4 + wv) * kAppendRowsPerWave;
#pragma unroll
    for (int k = 0; k < kAppendRowsPerWave; ++k) {
        const int row = row_base + k;
        if (row >= a.num_rows) return;
        const int r = find_request(a.cu_q, a.num_reqs, row, lane);
        const int t = a.prefix[r] + (row - a.cu_q[r]);
        const int lp = t >> a.log2_page;
        const int page = (t >= 0 && lp < a.max_pages) ? a.bt[(size_t)r * a.max_pages + lp] : -1;
        if ((unsigned)page >= (unsigned)a.num_pages) continue;
        const size_t slot = (size_t)page * a.page_size + (t & (a.page_size - 1));
        const u32x4 *src = reinterpret_cast<const u32x4 *>(a.src + (size_t)row * kDqk);
        u32x4 *dst = reinterpret_cast<u32x4 *>(a.kv + slot * kDqk);
        dst[lane] = src[lane];
        if (lane < kChunksPerRow - 64) dst[64 + lane] = src[64 + lane];
    }
}

}  // namespace

hipError_t launch_append(const AppendArgs &a, hipStream_t s) {
    const int rows_per_block = 4 * kAppendRowsPerWave;
    const int grid = (a.num_rows + rows_per_block - 1) / rows_per_block;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL(append_kernel, dim3(grid), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs &a, hipStream_t s) {
    const int grid = a.n_chunk_items + a.n_dec_items;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL(attention_kernel, dim3(grid), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_combine(const AttnArgs &a, hipStream_t s) {
    const int grid = a.n_chunk_items + a.n_dec_items;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL(combine_kernel, dim3(grid), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace mla
