// gfx950 kernels of libmlastep: latent append and mixed-step latent attention
// (decode rows and chunked-prefill rows of one step in one launch).
//
// The step is the one a decode node runs when it serves deflected prefill
// chunks next to its in-flight decodes (section 2.3; section 4.3.1, Eq. 4 of
// the paper); the head shapes are those of the served model's absorbed latent
// attention (DeepSeek-V2-Lite, section 6).
//
// Work decomposition (one launch for all rows of a step):
//   * decode rows (c = 1): persistent workgroups own equal shares of the list
//     of all decode tiles (32 keys each); see the decode section below.
//   * chunk rows (c > 1): one workgroup (4 wavefronts) per block of 4 query
//     tokens (one per wave, 16 head rows each) times a key range of ks_chunk
//     keys.  32-key tiles go through a 3-deep global -> LDS DMA ring; each
//     tile's value part is converted once to fp16 and transposed in LDS so
//     that P*V runs on fp16 MFMA.
// Rows whose keys are split across workgroups leave fp32 partials (the
// unnormalised sum, the running max and sum in log2 units); a second, small
// merge kernel combines them in a fixed order.  Results are therefore
// run-to-run deterministic and do not depend on the physical page order.
#include "mla_kernels.h"

#include <limits.h>
#include <math.h>

namespace mla {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int kChunksPerRow = kRowBytes / 16;  // 72 16-byte chunks per latent
// decode path
constexpr int kDecKeys = kKeysPerTile;  // 32
constexpr int kDecTileBytes = kDecKeys * kRowBytes;  // 36864
constexpr int kDecRing = 4;
constexpr int kDecLds = kDecRing * kDecTileBytes + 4 * kHeads * 20 * 4;  // ring + partial score blocks
// chunk path
constexpr int kChunkKeys = kKeysPerTile;  // 32
constexpr int kChunkTileBytes = kChunkKeys * kRowBytes;  // 36864

constexpr float kNegInf = -INFINITY;

// Optional per-workgroup timeline for profiling builds (-DMLA_TRACE): slot k
// of workgroup b records the 100 MHz real-time counter at point k.
#ifdef MLA_TRACE
// Trace builds only: per work item, 16 stamps (slot = the item's queue index).
__device__ unsigned long long g_trace[1 << 20];
__shared__ int s_trace_item;
#define TRACE_ITEM(item)                                                                  \
    do {                                                                                  \
        if (threadIdx.x == 0) {                                                           \
            s_trace_item = (item);                                                        \
            unsigned xcc, hw;                                                             \
            asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));           \
            asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));             \
            if ((item) < (1 << 16)) {                                                     \
                g_trace[(size_t)(item) * 16 + 0] = __builtin_amdgcn_s_memrealtime();      \
                g_trace[(size_t)(item) * 16 + 9] = ((unsigned long long)xcc << 32) | hw;  \
            }                                                                             \
        }                                                                                 \
    } while (0)
#define TRACE(k)                                                                          \
    do {                                                                                  \
        if (threadIdx.x == 0 && s_trace_item < (1 << 16))                                 \
            g_trace[(size_t)s_trace_item * 16 + (k)] = __builtin_amdgcn_s_memrealtime();  \
    } while (0)
#define TRACE_VAL(k, v)                                                                   \
    do {                                                                                  \
        if (threadIdx.x == 0 && s_trace_item < (1 << 16)) g_trace[(size_t)s_trace_item * 16 + (k)] = (v); \
    } while (0)
// shader-clock stamps inside the third tile of an item (slots 10..15)
#define TRACE_TILE(t, k)                                                                  \
    do {                                                                                  \
        if ((t) == 2 && threadIdx.x == 0 && s_trace_item < (1 << 16))                     \
            g_trace[(size_t)s_trace_item * 16 + (k)] = __builtin_amdgcn_s_memtime();      \
    } while (0)
#else
#define TRACE_ITEM(item) \
    do {                 \
    } while (0)
#define TRACE_TILE(t, k) \
    do {                 \
    } while (0)
#define TRACE(k) \
    do {         \
    } while (0)
#define TRACE_VAL(k, v) \
    do {                \
    } while (0)
#endif

constexpr float kLn2 = 0.69314718055994530942f;

// ---------------------------------------------------------------- helpers
__device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

__device__ __forceinline__ float bf16_bits_to_float(uint32_t b) { return __uint_as_float(b << 16); }

__device__ __forceinline__ uint32_t bf16_bits(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }

__device__ __forceinline__ uint32_t lds_addr(const void *p) {
    return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
}

// One 16-byte global -> LDS DMA per lane: lane i writes LDS bytes
// [base + 16 i, base + 16 i + 16).  `base` must be wave-uniform.  Issued with
// inline assembly so that the compiler does not drain the whole ring before
// every barrier; completion is tracked by hand (vmcnt).
__device__ __forceinline__ void lds_dma16(const void *gsrc, uint32_t lds_base) {
    asm volatile(
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off\n\t"
        :
        : "{m0}"(lds_base), "v"(gsrc)
        : "memory");
}

__device__ __forceinline__ void wait_dma_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void wait_dma_keep9() { asm volatile("s_waitcnt vmcnt(9)" ::: "memory"); }

// vmcnt(0) with expcnt / lgkmcnt left alone (gfx9 s_waitcnt encoding),
// issued through the builtin so the compiler's scoreboard accounts for it
// and inserts no vmcnt wait of its own inside the pipelined loops.
__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

__device__ __forceinline__ f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_f16(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// Reductions over lanes l, l^16, l^32, l^48 (the four row groups of a
// 16-column MFMA tile) with the gfx950 cross-row swaps: permlane32_swap pairs
// lane l with l +- 32, permlane16_swap pairs row groups 0-1 and 2-3.
__device__ __forceinline__ float wave_max16(float v) {
    const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float wave_sum16(float v) {
    const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// LDS byte offset of 16-byte chunk c of key k inside a tile.  Chunk
// positions are xor-swizzled with the key's low 3 bits so that 8 lanes that
// read the same chunk of 8 consecutive keys hit 8 different bank groups.
__device__ __forceinline__ int tile_off(int k, int c) { return (k * kChunksPerRow + (c ^ (k & 7))) * 16; }

// Transposing LDS read (gfx950): inside each 16-lane group, lane i receives
// element (i & 3) of the 8 bytes read by lane 4 j + (i >> 2), j = 0..3.
__device__ __forceinline__ u32x2 lds_read_tr16(const char *p) {
    const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(p));
    return __builtin_bit_cast(u32x2, v);
}

// ------------------------------------------------------ work-item lookup
// Items of one kind are numbered request by request; request r owns
// count(r) consecutive items.  The workgroup scans the per-request counts
// (256 requests per round) and finds the request owning item `target`.
struct ReqLens {
    const int32_t *cu_q;
    const int32_t *prefix;
};

struct Located {
    int r, local, p, row0, c;
};

template <typename CountFn>
__device__ bool locate_item(int target, int num_reqs, const ReqLens &rl, CountFn count, int *s_tmp,
                            Located &loc) {
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    if (tid == 0) s_tmp[4] = -1;
    int running = 0;
    for (int base = 0; base < num_reqs; base += kThreads) {
        const int r = base + tid;
        int cnt = 0, p = 0, row0 = 0, c = 0;
        if (r < num_reqs) {
            row0 = rl.cu_q[r];
            c = rl.cu_q[r + 1] - row0;
            p = rl.prefix[r];
            cnt = count(p, c);
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
            s_tmp[6] = p;
            s_tmp[7] = row0;
            s_tmp[8] = c;
        }
        __syncthreads();
        if (s_tmp[4] >= 0) {
            loc = Located{s_tmp[4], s_tmp[5], s_tmp[6], s_tmp[7], s_tmp[8]};
            return true;
        }
        running += total;
    }
    return false;
}

struct ChunkCount {
    int ks;
    __device__ int operator()(int p, int c) const {
        return c > 1 ? ceil_div(c, kChunkBlockTokens) * ceil_div(p + c, ks) : 0;
    }
};

struct ChunkItem {
    int r, p, c, row0, i0, i1, k0, k1, ks, nks_eff;
};

__device__ __forceinline__ ChunkItem decode_chunk_item(const AttnArgs &a, const Located &lc) {
    ChunkItem it;
    it.r = lc.r;
    it.p = lc.p;
    it.row0 = lc.row0;
    it.c = lc.c;
    const int nrb = ceil_div(it.c, kChunkBlockTokens);
    const int nks = ceil_div(it.p + it.c, a.ks_chunk);
    const int rb = nrb - 1 - lc.local / nks;  // longest rows first
    it.ks = lc.local % nks;
    it.i0 = rb * kChunkBlockTokens;
    it.i1 = min(it.i0 + kChunkBlockTokens, it.c);
    const int klim = it.p + it.i1;
    it.nks_eff = ceil_div(klim, a.ks_chunk);
    it.k0 = it.ks * a.ks_chunk;
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

// Issue the DMA of one tile of KEYS keys (kbase .. kbase + KEYS - 1, clamped
// to the last valid key k1 - 1 so every byte read is a finite cached latent).
// Instruction i of wave wv fills 1 KB segment i * 4 + wv of the tile.
// With a fused append, keys p_new .. are the step's new latents: key k comes
// from row new_row0 + k - p_new of a.new_kv instead of its cache slot.
template <int KEYS>
__device__ __forceinline__ void issue_tile(const AttnArgs &a, const int *s_pages, int lp0, int kbase, int k1,
                                           uint32_t lds_tile, int wv, int lane, int p_new, int new_row0) {
    constexpr int kDma = KEYS * kRowBytes / (kThreads * 16);
    const char *kv = reinterpret_cast<const char *>(a.kv);
    const char *nkv = reinterpret_cast<const char *>(a.new_kv);
    const char *src[kDma];
#pragma unroll
    for (int i = 0; i < kDma; ++i) {  // all page-id reads first, then the DMA burst
        const int seg = i * 4 + wv;
        const int u = seg * 64 + lane;
        const int kk = u / kChunksPerRow;
        const int c = (u - kk * kChunksPerRow) ^ (kk & 7);
        int key = kbase + kk;
        key = key < k1 ? key : k1 - 1;
        const int page = s_pages[min((key >> a.log2_page) - lp0, kPageWindow - 1)];
        const size_t slot = (size_t)page * a.page_size + (key & (a.page_size - 1));
        src[i] = (nkv != nullptr && key >= p_new) ? nkv + (size_t)(new_row0 + key - p_new) * kRowBytes + c * 16
                                                  : kv + slot * kRowBytes + c * 16;
    }
#pragma unroll
    for (int i = 0; i < kDma; ++i)
        lds_dma16(src[i], __builtin_amdgcn_readfirstlane(lds_tile + (i * 4 + wv) * 1024));
}

// DMA of a 32-key tile that lies inside one page: a uniform source base (the
// tile's first key) in SGPRs plus per-lane offsets fixed for all tiles.
// Round i of wave wv fills LDS chunk u = 256 i + 64 wv + lane of the tile,
// which holds source chunk (u % 72) ^ (key & 7) of key u / 72.
constexpr int kTileDma = kKeysPerTile * kRowBytes / (kThreads * 16);  // 9 rounds per tile
// Offsets (< 2^16) packed two per register: round i in the half i & 1 of word i / 2.
__device__ __forceinline__ void tile_dma_offsets(int wv, int lane, uint32_t (&off)[(kTileDma + 1) / 2]) {
#pragma unroll
    for (int w = 0; w < (kTileDma + 1) / 2; ++w) off[w] = 0;
#pragma unroll
    for (int i = 0; i < kTileDma; ++i) {
        const int u = (i * 4 + wv) * 64 + lane;
        const int kk = u / kChunksPerRow;
        const int c = (u - kk * kChunksPerRow) ^ (kk & 7);
        off[i / 2] |= (uint32_t)(kk * kRowBytes + c * 16) << (16 * (i & 1));
    }
}

__device__ __forceinline__ void lds_dma16_sbase(const void *sbase, uint32_t voff, uint32_t lds_base) {
    asm volatile(
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %0, %1\n\t"
        :
        : "v"(voff), "s"(sbase), "{m0}"(lds_base)
        : "memory");
}

// Fused append: copy n new latents (rows row0 .. of a.new_kv, keys key0 .. of
// request r) into their cache slots; the whole workgroup takes part.  Slots
// with a page id outside the pool are skipped.
__device__ __forceinline__ void append_rows(const AttnArgs &a, int r, int key0, int row0, int n) {
    const int32_t *btr = a.bt + (size_t)r * a.max_pages;
    for (int x = threadIdx.x; x < n * kChunksPerRow; x += kThreads) {
        const int i = x / kChunksPerRow, c = x - i * kChunksPerRow;
        const int key = key0 + i;
        const int lp = key >> a.log2_page;
        const int page = lp < a.max_pages ? btr[lp] : -1;
        if ((unsigned)page >= (unsigned)a.num_pages) continue;
        const u32x4 v = *reinterpret_cast<const u32x4 *>(a.new_kv + (size_t)(row0 + i) * kDqk + c * 8);
        *reinterpret_cast<u32x4 *>(a.kv_out + ((size_t)page * a.page_size + (key & (a.page_size - 1))) * kDqk +
                                   c * 8) = v;
    }
}

// Scores of 16 keys (tile rows key_base .. key_base + 15) against one token's
// query operand: lane l gets S[key_base + 4 (l/16) + i][head l%16], i = 0..3.
// Reads are staged 6 steps at a time; two accumulation chains.
__device__ __forceinline__ f32x4 score16(const char *tile, int key_base, const u32x4 *qreg, int lane) {
    const int g = lane >> 4, key = key_base + (lane & 15);
    f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    constexpr int G = 6;
#pragma unroll
    for (int grp = 0; grp < 18 / G; ++grp) {
        u32x4 av[G];
#pragma unroll
        for (int j = 0; j < G; ++j)
            av[j] = *reinterpret_cast<const u32x4 *>(tile + tile_off(key, (grp * G + j) * 4 + g));
#pragma unroll
        for (int j = 0; j < G; j += 2) {
            acc0 = mfma_bf16(av[j], qreg[grp * G + j], acc0);
            acc1 = mfma_bf16(av[j + 1], qreg[grp * G + j + 1], acc1);
        }
        __builtin_amdgcn_sched_group_barrier(0x100, G, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, G, 0);
    }
    return acc0 + acc1;
}

__device__ __forceinline__ void load_query(const AttnArgs &a, int row, int lane, u32x4 *qreg) {
    const uint16_t *qp = a.q + ((size_t)row * kHeads + (lane & 15)) * kDqk + (lane >> 4) * 8;
#pragma unroll
    for (int st = 0; st < 18; ++st) qreg[st] = *reinterpret_cast<const u32x4 *>(qp + st * 32);
}

// Store 4 consecutive dims of one (row, head) output, fp32 or bf16.
__device__ __forceinline__ void store_out4(const AttnArgs &a, int row, int head, int dv, f32x4 v) {
    const size_t off = ((size_t)row * kHeads + head) * kDv + dv;
    if (a.out_bf16) {
        const uint32_t w0 = bf16_bits(v[0]) | (bf16_bits(v[1]) << 16);
        const uint32_t w1 = bf16_bits(v[2]) | (bf16_bits(v[3]) << 16);
        *reinterpret_cast<u32x2 *>(reinterpret_cast<uint16_t *>(a.out) + off) = u32x2{w0, w1};
    } else {
        *reinterpret_cast<f32x4 *>(reinterpret_cast<float *>(a.out) + off) = v;
    }
}

// ------------------------------------------------------------------ merge
// Merge the key-split partials of one output row in split order.  Split s
// holds an unnormalised output o_s (16 heads x 512 dims) with its max m_s
// and sum l_s in log2 units; slot(s) gives pointers to both.  256 threads:
// head tid / 16, dims (tid % 16) * 32 .. + 32.  The loads of up to four splits
// go out together; the running result is rescaled whenever the max grows.
struct SplitRef {
    const float *o, *ml;
};

template <int NH, typename Slot>
__device__ void merge_heads(const AttnArgs &a, int row, int hh0, int nsplit, Slot slot) {
    // NH heads per workgroup: head hh0 + tid / (256 / NH), DPT value dims per thread
    constexpr int TPH = kThreads / NH, DPT = kDv / TPH, NV = DPT / 4;
    constexpr int B = NH >= 16 ? 4 : 8;  // splits whose loads go out together
    const int tid = threadIdx.x;
    const int hh = hh0 + tid / TPH, d0 = (tid % TPH) * DPT;
    float M = kNegInf, den = 0.f;
    f32x4 o[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) o[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < nsplit; s0 += B) {
        float ms[B], ls[B];
        f32x4 v[B][NV];
#pragma unroll
        for (int q = 0; q < B; ++q) {
            ms[q] = kNegInf;
            ls[q] = 0.f;
            if (s0 + q < nsplit) {
                const SplitRef sr = slot(s0 + q);
                ms[q] = sr.ml[hh * 2];
                ls[q] = sr.ml[hh * 2 + 1];
                const f32x4 *src = reinterpret_cast<const f32x4 *>(sr.o + hh * kDv + d0);
#pragma unroll
                for (int k = 0; k < NV; ++k) v[q][k] = src[k];
            } else {
#pragma unroll
                for (int k = 0; k < NV; ++k) v[q][k] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
        }
#pragma unroll
        for (int q = 0; q < B; ++q) {
            if (ms[q] == kNegInf) continue;  // a split that saw no key of this row
            const float m_new = fmaxf(M, ms[q]);
            const float c_old = (M == kNegInf) ? 0.f : exp2f(M - m_new);
            const float c_new = exp2f(ms[q] - m_new);
            den = den * c_old + ls[q] * c_new;
#pragma unroll
            for (int k = 0; k < NV; ++k) o[k] = o[k] * c_old + v[q][k] * c_new;
            M = m_new;
        }
    }
    const float inv = 1.f / den;
#pragma unroll
    for (int k = 0; k < NV; ++k) store_out4(a, row, hh, d0 + 4 * k, o[k] * inv);
    if (a.lse && tid % TPH == 0) a.lse[(size_t)row * kHeads + hh] = (M + log2f(den)) * kLn2;
}

template <typename Slot>
__device__ void merge_row(const AttnArgs &a, int row, int nsplit, Slot slot) {
    merge_heads<kHeads>(a, row, 0, nsplit, slot);
}

// ------------------------------------------------------------ decode path
// Decode rows run on persistent workgroups.  The 32-key tiles of all decode
// requests, request after request, form one list; workgroup w owns tiles
// [w S, (w + 1) S).  Its share splits into segments, one per request it
// touches.  A segment streams its query block and then its tiles through a
// 4-slot global -> LDS DMA ring, so prefetch runs on across request
// boundaries and the start-up latency is paid once per workgroup.  Per tile,
// wave w scores 16 keys over half of the 576 latent dims (the four partial
// 16 x 16 score blocks meet in LDS), then accumulates its 128-wide slice of
// the value dims over all 32 keys.  A request spread over several workgroups
// leaves fp32 partials (slot 2 w for a workgroup's first segment, 2 w + 1 for
// its last) that the merge kernel combines.
constexpr int kMaxSeg = kMaxDecSegments;
constexpr int kXStride = 20;  // floats per head row of a partial score block (16 + pad)

struct DecSeg {
    int r, p, row, t0, t1, pw, lp0;  // tiles t0 .. t1-1 of request r; page window offset / first page
};

__device__ __forceinline__ int dec_tiles(int p, int c) { return c == 1 ? ceil_div(p + 1, kDecKeys) : 0; }

// Exclusive prefix sum over the 256 threads of the workgroup (uses s_w[0..3]).
__device__ __forceinline__ int block_scan_excl(int v, int *s_w, int &total) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    int inc = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int t = __shfl_up(inc, d, 64);
        if (lane >= d) inc += t;
    }
    if (lane == 63) s_w[wv] = inc;
    __syncthreads();
    int off = 0;
    total = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int t = s_w[k];
        off += (k < wv) ? t : 0;
        total += t;
    }
    __syncthreads();
    return inc - v + off;
}

// Segments (request order) of the decode tile range [R0, R1); returns their count.
__device__ int find_segments(const AttnArgs &a, int R0, int R1, DecSeg *s_seg, int *s_tmp) {
    const int tid = threadIdx.x;
    int running = 0, nseg = 0;
    for (int base = 0; base < a.num_reqs && running < R1; base += kThreads) {
        const int r = base + tid;
        int nt = 0, p = 0, row0 = 0;
        if (r < a.num_reqs) {
            row0 = a.cu_q[r];
            p = a.prefix[r];
            // rows outside [0, T) only arise from device lengths that disagree with the host's
            nt = (p >= 0 && row0 >= 0 && row0 < a.num_rows) ? dec_tiles(p, a.cu_q[r + 1] - row0) : 0;
        }
        int tot_t, tot_s;
        const int T = running + block_scan_excl(nt, s_tmp, tot_t);
        const bool ov = nt > 0 && T < R1 && T + nt > R0;
        const int j = nseg + block_scan_excl(ov ? 1 : 0, s_tmp, tot_s);
        if (ov && j < kMaxSeg) s_seg[j] = DecSeg{r, p, row0, max(R0 - T, 0), min(R1 - T, nt), 0, 0};
        nseg += tot_s;
        running += tot_t;
    }
    __syncthreads();
    return min(nseg, kMaxSeg);
}

// Unit cursor of a workgroup's stream: segment j, tile t (t < 0: the query block).
struct Cursor {
    int j, t;
};
__device__ __forceinline__ void advance(Cursor &c, const DecSeg *s_seg) {
    if (c.t < 0)
        c.t = s_seg[c.j].t0;
    else
        ++c.t;
    if (c.t >= s_seg[c.j].t1) {
        ++c.j;
        c.t = -1;
    }
}

// DMA of one stream unit into a 36 KB ring slot.  A query block (16 heads x
// 576 dims, 18 KB) is copied twice over so every unit takes 9 DMA rounds.  A
// full tile inside one page uses the uniform-base form (offsets `dma_off`).
__device__ __forceinline__ void issue_unit(const AttnArgs &a, const DecSeg &sg, int t, const int *s_pages,
                                           uint32_t slot, int wv, int lane,
                                           const uint32_t (&dma_off)[(kTileDma + 1) / 2]) {
    constexpr int kDma = kDecTileBytes / (kThreads * 16);  // 9
    const int kbase = t * kDecKeys;
    const int last_cached = a.new_kv != nullptr ? sg.p - 1 : sg.p;  // key p is the new latent when fused
    if (t >= 0 && a.page_size >= kDecKeys && kbase + kDecKeys - 1 <= last_cached) {
        const int page = s_pages[min(sg.pw + (kbase >> a.log2_page) - sg.lp0, kPageWindow - 1)];
        const char *src = reinterpret_cast<const char *>(a.kv) +
                          ((size_t)__builtin_amdgcn_readfirstlane(page) * a.page_size + (kbase & (a.page_size - 1))) *
                              kRowBytes;
#pragma unroll
        for (int i = 0; i < kDma; ++i)
            lds_dma16_sbase(src, (dma_off[i / 2] >> (16 * (i & 1))) & 0xffffu,
                            __builtin_amdgcn_readfirstlane(slot + (i * 4 + wv) * 1024));
        return;
    }
    const char *src[kDma];
    if (t < 0) {
        const char *qb = reinterpret_cast<const char *>(a.q + (size_t)sg.row * kHeads * kDqk);
#pragma unroll
        for (int i = 0; i < kDma; ++i) {
            const int u = (i * 4 + wv) * 64 + lane;
            src[i] = qb + (u % (kHeads * kChunksPerRow)) * 16;
        }
    } else {
        const char *kv = reinterpret_cast<const char *>(a.kv);
        const int klast = sg.p;
#pragma unroll
        for (int i = 0; i < kDma; ++i) {
            const int u = (i * 4 + wv) * 64 + lane;
            const int kk = u / kChunksPerRow;
            const int c = (u - kk * kChunksPerRow) ^ (kk & 7);
            const int key = min(kbase + kk, klast);
            const int page = s_pages[min(sg.pw + (key >> a.log2_page) - sg.lp0, kPageWindow - 1)];
            src[i] = (a.new_kv != nullptr && key == klast)
                         ? reinterpret_cast<const char *>(a.new_kv) + (size_t)sg.row * kRowBytes + c * 16
                         : kv + ((size_t)page * a.page_size + (key & (a.page_size - 1))) * kRowBytes + c * 16;
        }
    }
#pragma unroll
    for (int i = 0; i < kDma; ++i) lds_dma16(src[i], __builtin_amdgcn_readfirstlane(slot + (i * 4 + wv) * 1024));
}

__device__ __forceinline__ void wait_units_newer(int n) {  // n of the later units may stay in flight
    if (n <= 0)
        wait_dma_all();
    else if (n == 1)
        wait_dma_keep9();
    else
        asm volatile("s_waitcnt vmcnt(18)" ::: "memory");
}

__device__ void decode_wg(const AttnArgs &a, int w, char *smem, int *s_tmp, int *s_pages, DecSeg *s_seg) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, h = lane & 15;
    const int R0 = w * a.dec_unit_tiles;
    const int R1 = min(R0 + a.dec_unit_tiles, a.dec_total_tiles);
    if (R0 >= R1) return;
    const int nseg = find_segments(a, R0, R1, s_seg, s_tmp);
    TRACE(1);
    if (nseg == 0) return;
    if (tid == 0) {  // page-window offsets of the segments
        int pw = 0;
        for (int j = 0; j < nseg; ++j) {
            const DecSeg sg = s_seg[j];
            const int lp0 = (sg.t0 * kDecKeys) >> a.log2_page;
            const int klast = min(sg.t1 * kDecKeys, sg.p + 1) - 1;
            s_seg[j].pw = pw;
            s_seg[j].lp0 = lp0;
            pw += (klast >> a.log2_page) - lp0 + 1;
        }
    }
    __syncthreads();
    for (int j = 0; j < nseg; ++j) {
        const DecSeg sg = s_seg[j];
        const int klast = min(sg.t1 * kDecKeys, sg.p + 1) - 1;
        const int n = (klast >> a.log2_page) - sg.lp0 + 1;
        const int32_t *btr = a.bt + (size_t)sg.r * a.max_pages;
        for (int i = tid; i < n && sg.pw + i < kPageWindow; i += kThreads) {
            const int lp = sg.lp0 + i;
            const int pg = lp < a.max_pages ? btr[lp] : 0;
            s_pages[sg.pw + i] = ((unsigned)pg < (unsigned)a.num_pages) ? pg : 0;
        }
    }
    if (a.new_kv != nullptr) {  // fused append: the workgroup holding a request's last tile writes its latent
        for (int j = 0; j < nseg; ++j) {
            const DecSeg sg = s_seg[j];
            if (sg.t1 == dec_tiles(sg.p, 1)) append_rows(a, sg.r, sg.p, sg.row, 1);
        }
    }
    __syncthreads();
    TRACE(2);

    const int n_units = nseg + (R1 - R0);
    TRACE_VAL(8, 1000000ull * 2 + n_units);
    uint32_t dma_off[(kTileDma + 1) / 2];
    tile_dma_offsets(wv, lane, dma_off);
    const uint32_t ring = lds_addr(smem);
    float *s_X = reinterpret_cast<float *>(smem + kDecRing * kDecTileBytes);
    Cursor prod{0, -1}, cons{0, -1};
    for (int u = 0; u < kDecRing - 1 && u < n_units; ++u) {
        issue_unit(a, s_seg[prod.j], prod.t, s_pages, ring + u * kDecTileBytes, wv, lane, dma_off);
        advance(prod, s_seg);
    }

    u32x4 qreg[9];  // this wave's half of the query operand: steps 9 (wv >> 1) .. + 9
    f32x4 acc[8];
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_ref = kNegInf, l_run = 0.f;
    const int hf = wv >> 1;
    const int kq = 16 * (wv & 1) + (lane & 15);             // key this lane scores
    const int tr_key = 4 * g + ((lane & 15) >> 2);          // transposing-read source row
    const int tr_dv = wv * 128 + 4 * (lane & 3);            // and its first value dim

    TRACE(3);
    for (int u = 0; u < n_units; ++u) {
        TRACE_TILE(u, 10);
        wait_units_newer(min(kDecRing - 2, n_units - 1 - u));
        __syncthreads();
        if (prod.j < nseg) {
            issue_unit(a, s_seg[prod.j], prod.t, s_pages, ring + ((u + kDecRing - 1) % kDecRing) * kDecTileBytes, wv,
                       lane, dma_off);
            advance(prod, s_seg);
        }
        const char *slot = smem + (u % kDecRing) * kDecTileBytes;
        const DecSeg sg = s_seg[cons.j];
        if (cons.t < 0) {  // a new request: its query block
#pragma unroll
            for (int s2 = 0; s2 < 9; ++s2)
                qreg[s2] = *reinterpret_cast<const u32x4 *>(slot + (h * kChunksPerRow + (9 * hf + s2) * 4 + g) * 16);
            advance(cons, s_seg);
            continue;
        }
        TRACE_TILE(u, 11);
        const int kbase = cons.t * kDecKeys;
        // partial scores: keys 16 (wv & 1) .. + 16, dims of steps 9 hf .. 9 hf + 8
        f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
        {
            u32x4 av[9];
#pragma unroll
            for (int s2 = 0; s2 < 9; ++s2)
                av[s2] = *reinterpret_cast<const u32x4 *>(slot + tile_off(kq, (9 * hf + s2) * 4 + g));
#pragma unroll
            for (int s2 = 0; s2 < 9; s2 += 2) {
                sa = mfma_bf16(av[s2], qreg[s2], sa);
                if (s2 + 1 < 9) sb = mfma_bf16(av[s2 + 1], qreg[s2 + 1], sb);
            }
        }
        *reinterpret_cast<f32x4 *>(s_X + (wv * kHeads + h) * kXStride + 4 * g) = sa + sb;
        __syncthreads();
        TRACE_TILE(u, 12);
        // full scores of this lane's head: x[kt][i] = key 16 kt + 4 g + i (kt = 0, 1)
        f32x4 x[2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            const f32x4 lo = *reinterpret_cast<const f32x4 *>(s_X + (kt * kHeads + h) * kXStride + 4 * g);
            const f32x4 hi = *reinterpret_cast<const f32x4 *>(s_X + ((kt + 2) * kHeads + h) * kXStride + 4 * g);
            x[kt] = lo + hi;
        }
        float mt = kNegInf;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                x[kt][i] = (kbase + 16 * kt + 4 * g + i <= sg.p) ? x[kt][i] * a.scale_log2 : kNegInf;
                mt = fmaxf(mt, x[kt][i]);
            }
        }
        mt = wave_max16(mt);
        // Lazy rescale (the same decision in every wave): keep the reference max
        // unless the tile max exceeds it by more than 2^8.
        if (__builtin_amdgcn_ballot_w64(mt > m_ref + 8.f) != 0) {
            const float m_new = fmaxf(m_ref, mt);
            const float alpha = (m_ref == kNegInf) ? 0.f : exp2f(m_ref - m_new);
#pragma unroll
            for (int mt2 = 0; mt2 < 8; ++mt2) acc[mt2] = acc[mt2] * alpha;
            l_run *= alpha;
            m_ref = m_new;
        }
        // probabilities, split into bf16 hi + lo so that P*V keeps ~16 bits;
        // slot 8 g + 4 kt + i of the B operand holds key 16 kt + 4 g + i
        uint32_t bh[4], bl[4];
        float ps = 0.f;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int i = 0; i < 4; i += 2) {
                const float p0 = (x[kt][i] == kNegInf) ? 0.f : exp2f(x[kt][i] - m_ref);
                const float p1 = (x[kt][i + 1] == kNegInf) ? 0.f : exp2f(x[kt][i + 1] - m_ref);
                ps += p0 + p1;
                const uint32_t h0 = bf16_bits(p0), h1 = bf16_bits(p1);
                bh[kt * 2 + (i >> 1)] = h0 | (h1 << 16);
                bl[kt * 2 + (i >> 1)] = bf16_bits(p0 - bf16_bits_to_float(h0)) |
                                        (bf16_bits(p1 - bf16_bits_to_float(h1)) << 16);
            }
        }
        l_run += ps;
        TRACE_TILE(u, 13);
        u32x4 vop[8];
#pragma unroll
        for (int mt2 = 0; mt2 < 8; ++mt2) {
            const int dv = tr_dv + mt2 * 16;
            const int byte = ((dv >> 2) & 1) * 8;
            const u32x2 lo = lds_read_tr16(slot + tile_off(tr_key, dv >> 3) + byte);
            const u32x2 hi = lds_read_tr16(slot + tile_off(tr_key + 16, dv >> 3) + byte);
            vop[mt2] = u32x4{lo[0], lo[1], hi[0], hi[1]};
        }
        const u32x4 opb_h = {bh[0], bh[1], bh[2], bh[3]};
        const u32x4 opb_l = {bl[0], bl[1], bl[2], bl[3]};
#pragma unroll
        for (int mt2 = 0; mt2 < 8; ++mt2) acc[mt2] = mfma_bf16(vop[mt2], opb_h, acc[mt2]);
#pragma unroll
        for (int mt2 = 0; mt2 < 8; ++mt2) acc[mt2] = mfma_bf16(vop[mt2], opb_l, acc[mt2]);

        TRACE_TILE(u, 14);
        const int jseg = cons.j;
        advance(cons, s_seg);
        if (cons.j != jseg) {  // the segment's last tile: finish it
            const float l_tot = wave_sum16(l_run);
            if (sg.t0 == 0 && sg.t1 == dec_tiles(sg.p, 1)) {
                const float inv = 1.f / l_tot;
#pragma unroll
                for (int mt2 = 0; mt2 < 8; ++mt2)
                    store_out4(a, sg.row, h, wv * 128 + mt2 * 16 + 4 * g, acc[mt2] * inv);
                if (a.lse && wv == 0 && g == 0) a.lse[(size_t)sg.row * kHeads + h] = (m_ref + log2f(l_tot)) * kLn2;
            } else if (a.ws_dec_o != nullptr) {
                const size_t slot_id = 2 * (size_t)w + (jseg == 0 ? 0 : 1);
                float *po = a.ws_dec_o + (slot_id * kHeads + h) * kDv;
#pragma unroll
                for (int mt2 = 0; mt2 < 8; ++mt2)
                    *reinterpret_cast<f32x4 *>(po + wv * 128 + mt2 * 16 + 4 * g) = acc[mt2];
                if (wv == 0 && g == 0) {
                    a.ws_dec_ml[(slot_id * kHeads + h) * 2 + 0] = m_ref;
                    a.ws_dec_ml[(slot_id * kHeads + h) * 2 + 1] = l_tot;
                }
            }
#pragma unroll
            for (int mt2 = 0; mt2 < 8; ++mt2) acc[mt2] = f32x4{0.f, 0.f, 0.f, 0.f};
            m_ref = kNegInf;
            l_run = 0.f;
        }
    }
    TRACE(4);
}

// Merge kernel side: workgroup (r, part) merges heads part * 16 / hsplit ..
// of decode request r when its tiles span several decode units.  Unit v
// keeps its first segment in slot 2 v and its last one in slot 2 v + 1.
__device__ void decode_merge(const AttnArgs &a, int r, int part, int *s_tmp) {
    if (a.ws_dec_o == nullptr || r >= a.num_reqs) return;
    const int tid = threadIdx.x;
    // T = decode tiles of the requests before r (one block-wide sum per 256 requests)
    int T = 0;
    for (int base = 0; base < r; base += kThreads) {
        const int q = base + tid;
        int nt = 0;
        if (q < r) {
            const int row0 = a.cu_q[q], p = a.prefix[q];
            nt = (p >= 0 && row0 >= 0 && row0 < a.num_rows) ? dec_tiles(p, a.cu_q[q + 1] - row0) : 0;
        }
        int total;
        block_scan_excl(nt, s_tmp, total);
        T += total;
    }
    const int row = a.cu_q[r], p = a.prefix[r];
    if (p < 0 || row < 0 || row >= a.num_rows || a.cu_q[r + 1] - row != 1) return;
    const int S = a.dec_unit_tiles, nt = dec_tiles(p, 1);
    const int w0 = T / S, w1 = (T + nt - 1) / S;
    if (w0 == w1) return;  // one unit wrote the row itself
    auto slot = [&](int s) {
        const int v = w0 + s;
        const size_t sl = 2 * (size_t)v + ((v == w0 && T != w0 * S) ? 1 : 0);
        return SplitRef{a.ws_dec_o + sl * kHeads * kDv, a.ws_dec_ml + sl * kHeads * 2};
    };
    const int n = w1 - w0 + 1;
    if (a.merge_hsplit == 8)
        merge_heads<2>(a, row, 2 * part, n, slot);
    else if (a.merge_hsplit == 4)
        merge_heads<4>(a, row, 4 * part, n, slot);
    else
        merge_heads<16>(a, row, 0, n, slot);
}

// ------------------------------------------------------------- chunk path
// Chunk rows: one workgroup per block of 6 query tokens and a key range of
// ks_chunk keys; 32-key tiles stream through a 3-slot DMA ring.
//  * Scores.  Waves 2p and 2p+1 hold the queries of tokens 3p .. 3p+2, wave 2p
//    over latent dims 0..287 and wave 2p+1 over dims 288..575, so every K
//    operand read from LDS feeds three MFMAs per key block.  The pair then
//    swaps partial scores through LDS so that wave 2p+h holds the full scores
//    of keys 16h .. 16h+15 of the tile for its three tokens.
//  * Softmax.  Probabilities against a fixed reference max (no rescaling; see
//    the passes below), published in LDS as fp16 in MFMA B-operand order.
//  * P*V.  Every wave accumulates its 128-wide slice of the value dims for all
//    6 tokens: each transposed V^T operand read is converted to fp16 once and
//    feeds 6 MFMAs.  fp16 holds every bf16 value in [2^-14, 65504] exactly.
// The loop is software-pipelined: the softmax of tile t runs in the same
// stretch of code as the P*V products of tile t - 1, so VALU work issues
// while the matrix cores are busy; two barriers per tile.
__device__ __forceinline__ void score_bases(int key, int g, int base[2]) {
    // chunk 4 st + g of `key` sits at base[st & 1] + 128 (st >> 1): the xor
    // swizzle only touches the chunk index's low 3 bits
#pragma unroll
    for (int e = 0; e < 2; ++e) base[e] = (key * kChunksPerRow + ((4 * e + g) ^ (key & 7))) * 16;
}

constexpr int kPairTokens = kChunkBlockTokens / 2;  // 3 tokens per wave pair

// Partial scores of one 32-key tile over k-steps 9 HALF .. 9 HALF + 8 (288
// latent dims) for the wave's 3 tokens, element i of key block kt = key
// 16 kt + 4 g + i, head l%16.  keep[j] is key block HALF (this wave finishes
// it), give[j] the other block (handed to the partner).  K operands are read
// two steps ahead.
template <int HALF>
__device__ __forceinline__ void score_half(const char *tile, const u32x4 (&qreg)[kPairTokens][9], int lane,
                                           f32x4 (&keep)[kPairTokens], f32x4 (&give)[kPairTokens]) {
    f32x4 s[kPairTokens][2];
    const int g = lane >> 4;
    int b0[2], b1[2];
    score_bases(lane & 15, g, b0);
    score_bases(16 + (lane & 15), g, b1);
#pragma unroll
    for (int j = 0; j < kPairTokens; ++j) s[j][0] = s[j][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    u32x4 a0[3], a1[3];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
        const int gs = 9 * HALF + st;
        a0[st] = *reinterpret_cast<const u32x4 *>(tile + b0[gs & 1] + 128 * (gs >> 1));
        a1[st] = *reinterpret_cast<const u32x4 *>(tile + b1[gs & 1] + 128 * (gs >> 1));
    }
#pragma unroll
    for (int st = 0; st < 9; ++st) {
        if (st + 2 < 9) {  // operands two steps ahead
            const int gs = 9 * HALF + st + 2;
            a0[(st + 2) % 3] = *reinterpret_cast<const u32x4 *>(tile + b0[gs & 1] + 128 * (gs >> 1));
            a1[(st + 2) % 3] = *reinterpret_cast<const u32x4 *>(tile + b1[gs & 1] + 128 * (gs >> 1));
        }
#pragma unroll
        for (int j = 0; j < kPairTokens; ++j) {
            s[j][0] = mfma_bf16(a0[st % 3], qreg[j][st], s[j][0]);
            s[j][1] = mfma_bf16(a1[st % 3], qreg[j][st], s[j][1]);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int j = 0; j < kPairTokens; ++j) {
        keep[j] = s[j][HALF];
        give[j] = s[j][1 - HALF];
    }
}

// bf16 pairs -> fp16 pairs (exact for |v| in [2^-14, 65504]; larger values
// clamp to +-65504, smaller ones round toward zero).
__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t w) {
    const auto h = __builtin_amdgcn_cvt_pkrtz(__uint_as_float(w << 16), __uint_as_float(w & 0xffff0000u));
    return __builtin_bit_cast(uint32_t, h);
}

__device__ __forceinline__ uint32_t f16x2_bits(float a, float b) {
    typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
    const f16x2 v = {(_Float16)a, (_Float16)b};  // round to nearest even
    return __builtin_bit_cast(uint32_t, v);
}

// V^T operand of 16 value dims x 32 keys (transposing reads of keys k and
// k + 16, see tr_base) converted to fp16.
__device__ __forceinline__ u32x4 load_vt_f16(const char *vb) {
    const u32x2 lo = lds_read_tr16(vb);
    const u32x2 hi = lds_read_tr16(vb + 16 * kRowBytes);
    return u32x4{bf16x2_to_f16x2(lo[0]), bf16x2_to_f16x2(lo[1]), bf16x2_to_f16x2(hi[0]), bf16x2_to_f16x2(hi[1])};
}

constexpr int kChunkRing = 3;
constexpr int kXBytes = 4 * kPairTokens * 64 * 16;         // score swap: [wave][token][lane] f32x4
constexpr int kPBytes = 2 * kChunkBlockTokens * 64 * 16;  // fp16 P, two buffers: [buf][token][lane] u32x4
constexpr int kHsBytes = 4 * kPairTokens * kHeads * 4;     // per-wave half maxima / sums: [wave][token][head]
constexpr int kChunkLds = kChunkRing * kChunkTileBytes + kXBytes + kPBytes + kHsBytes + 16;
// Largest exponent (log2 units) a probability may take against the reference
// max: 2^15 stays inside fp16.
constexpr float kMaxPExp = 15.f;

// Passes of a chunk item.  The reference max of each (token, head) is fixed
// for the whole key range, so the accumulators are never rescaled:
//   kPassMain   reference = max of the first tile.  Each lane also tracks the
//               max of every score it sees.  If a later score exceeds the
//               reference by more than 2^15, the pass still runs to the end
//               (an exit from the middle of the loop costs the accumulators
//               their registers) and its products are discarded;
//   kPassExact  then redoes the item against the exact max.
enum { kPassMain = 0, kPassExact = 1 };

__device__ void chunk_item(const AttnArgs &a, int item, char *smem, int *s_tmp, int *s_pages) {
    Located lc;
    if (!locate_item(item, a.num_reqs, ReqLens{a.cu_q, a.prefix}, ChunkCount{a.ks_chunk}, s_tmp, lc)) return;
    const ChunkItem it = decode_chunk_item(a, lc);
    TRACE(1);
    const int r = it.r;
    if (it.k0 >= it.k1) return;  // key range past this block's causal limit
    if (it.p < 0 || it.row0 < 0 || it.row0 + it.i1 > a.num_rows) return;
    if (it.nks_eff > 1 && a.ws_chunk_o == nullptr) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, h = lane & 15;
    const int pair = wv >> 1, half = wv & 1, partner = wv ^ 1;
    const int nt = it.i1 - it.i0;  // tokens of this block (1 .. 6)
    const int ntiles = ceil_div(it.k1 - it.k0, kChunkKeys);
    const int lp0 = it.k0 >> a.log2_page;
    // queries of tokens 3 pair + j over this wave's half of the latent dims
    // (issued first: their latency overlaps the page-window load)
    u32x4 qreg[kPairTokens][9];
#pragma unroll
    for (int j = 0; j < kPairTokens; ++j) {
        const int row = it.row0 + it.i0 + min(kPairTokens * pair + j, nt - 1);  // an idle token re-reads a row
        const uint16_t *qp = a.q + ((size_t)row * kHeads + h) * kDqk + 9 * half * 32 + g * 8;
#pragma unroll
        for (int st = 0; st < 9; ++st) qreg[j][st] = *reinterpret_cast<const u32x4 *>(qp + st * 32);
    }
    load_page_window(a, r, lp0, ((it.k1 - 1) >> a.log2_page) - lp0 + 1, s_pages);
    TRACE(2);
    TRACE_VAL(8, 1000000ull * 1 + ntiles);

    const uint32_t ring = lds_addr(smem);
    char *const lds_x = smem + kChunkRing * kChunkTileBytes;
    f32x4 *s_X = reinterpret_cast<f32x4 *>(lds_x);                                  // [wave][token][lane]
    uint32_t *s_P = reinterpret_cast<uint32_t *>(lds_x + kXBytes);                  // [buf][token][lane][4]
    float *s_hs = reinterpret_cast<float *>(lds_x + kXBytes + kPBytes);             // [wave][token][head]
    int *s_abort = reinterpret_cast<int *>(lds_x + kXBytes + kPBytes + kHsBytes);

    // Key of score i (0..3) of this lane within a tile: 16 half + 4 g + i.
    // A score counts if its key <= elim[j] (the token's causal limit, clipped
    // to the item's key range; -1 for an idle token).
    int elim[kPairTokens];
#pragma unroll
    for (int j = 0; j < kPairTokens; ++j) {
        const int tb = kPairTokens * pair + j;
        elim[j] = tb < nt ? min(it.p + it.i0 + tb, it.k1 - 1) - (16 * half + 4 * g) : -1 - (it.k1 + 64);
    }
    // V^T reads: value dims wv*128 + 16 mt + 4 (l & 3) .. + 3 of keys tr_key and
    // tr_key + 16.  Their 16-byte chunk is wv*16 + 8 (mt >> 2) + (2 (mt & 3) +
    // ((l & 3) >> 1)); the xor swizzle touches only the low three bits, so four
    // bases plus immediate offsets cover all mt.
    const int tr_key = 4 * g + ((lane & 15) >> 2);
    int tr_base[4];
#pragma unroll
    for (int m4 = 0; m4 < 4; ++m4)
        tr_base[m4] = (tr_key * kChunksPerRow + wv * 16 + ((2 * m4 + ((lane & 3) >> 1)) ^ (tr_key & 7))) * 16 +
                      (lane & 1) * 8;

    uint32_t dma_off[(kTileDma + 1) / 2];
    tile_dma_offsets(wv, lane, dma_off);
    // DMA of tile t into its ring slot: a full tile inside one page takes the
    // uniform-base form, any other tile (small pages, the last partial tile)
    // the general one.  page_of(t) may be read well before the issue.
    const bool in_page = a.page_size >= kChunkKeys;
    // with a fused append, keys p .. come from the new latents (general path)
    const int cached_end = a.new_kv != nullptr ? min(it.k1, it.p) : it.k1;
    auto page_of = [&](int t) {
        return s_pages[min(((it.k0 + t * kChunkKeys) >> a.log2_page) - lp0, kPageWindow - 1)];
    };
    auto issue = [&](int t, int page) {
        const int kbase = it.k0 + t * kChunkKeys;
        const uint32_t dst = ring + (t % kChunkRing) * kChunkTileBytes;
        if (in_page && kbase + kChunkKeys <= cached_end) {
            const char *src = reinterpret_cast<const char *>(a.kv) +
                              ((size_t)__builtin_amdgcn_readfirstlane(page) * a.page_size +
                               (kbase & (a.page_size - 1))) * kRowBytes;
#pragma unroll
            for (int i = 0; i < kTileDma; ++i)
                lds_dma16_sbase(src, (dma_off[i / 2] >> (16 * (i & 1))) & 0xffffu,
                                __builtin_amdgcn_readfirstlane(dst + (i * 4 + wv) * 1024));
        } else {
            issue_tile<kChunkKeys>(a, s_pages, lp0, kbase, it.k1, dst, wv, lane, it.p, it.row0);
        }
    };

    float m_ref[kPairTokens], m_lane[kPairTokens], l_run[kPairTokens];
#pragma unroll
    for (int j = 0; j < kPairTokens; ++j) m_ref[j] = m_lane[j] = kNegInf;
    f32x4 acc[kChunkBlockTokens][8];  // [token][value-dim tile of this wave's 128-wide slice]
    f32x4 keep[kPairTokens];
    bool bad = false;

    auto scores = [&](int t) {
        const char *tile = smem + (t % kChunkRing) * kChunkTileBytes;
        f32x4 give[kPairTokens];
        if (half)
            score_half<1>(tile, qreg, lane, keep, give);
        else
            score_half<0>(tile, qreg, lane, keep, give);
        // hand the other key half over to the partner
#pragma unroll
        for (int j = 0; j < kPairTokens; ++j) s_X[(wv * kPairTokens + j) * 64 + lane] = give[j];
    };
    // full scores of this lane's 4 keys of token j (masked), raw dot products
    auto tile_scores = [&](int t, int j, float raw[4]) {
        const f32x4 f = keep[j] + s_X[(partner * kPairTokens + j) * 64 + lane];
        const int rel = elim[j] - (it.k0 + t * kChunkKeys);
#pragma unroll
        for (int i = 0; i < 4; ++i) raw[i] = i <= rel ? f[i] : kNegInf;
    };
    auto softmax = [&](int t, bool main_pass, int j) {
        float raw[4];
        tile_scores(t, j, raw);
        const float xm = fmaxf(fmaxf(raw[0], raw[1]), fmaxf(raw[2], raw[3])) * a.scale_log2;
        m_lane[j] = fmaxf(m_lane[j], xm);
        // also true for a first visible key after the first tile
        bad |= main_pass && xm - m_ref[j] > kMaxPExp;
        // the scaled score is rounded before the max is subtracted, so the max
        // key gets p = 1 exactly; masked scores give p = 0
        const float mref = m_ref[j] == kNegInf ? 0.f : m_ref[j];
        float p[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma clang fp contract(off)
            p[i] = __builtin_amdgcn_exp2f(raw[i] * a.scale_log2 - mref);
        }
        l_run[j] += (p[0] + p[1]) + (p[2] + p[3]);
        const int tb = kPairTokens * pair + j;
        *reinterpret_cast<u32x2 *>(s_P + (((t & 1) * kChunkBlockTokens + tb) * 64 + lane) * 4 + 2 * half) =
            u32x2{f16x2_bits(p[0], p[1]), f16x2_bits(p[2], p[3])};
    };
    auto pv = [&](int t, bool with_softmax, bool main_pass) {  // P*V of tile t (and softmax of t + 1)
        const char *tile = smem + (t % kChunkRing) * kChunkTileBytes;
        u32x4 bp[kChunkBlockTokens];
#pragma unroll
        for (int j = 0; j < kChunkBlockTokens; ++j)
            bp[j] = *reinterpret_cast<const u32x4 *>(s_P + (((t & 1) * kChunkBlockTokens + j) * 64 + lane) * 4);
        u32x4 av[2];
        av[0] = load_vt_f16(tile + tr_base[0]);
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) {
            if (mt + 1 < 8) av[(mt + 1) & 1] = load_vt_f16(tile + tr_base[(mt + 1) & 3] + 128 * ((mt + 1) >> 2));
#pragma unroll
            for (int j = 0; j < kChunkBlockTokens; ++j) acc[j][mt] = mfma_f16(av[mt & 1], bp[j], acc[j][mt]);
            if (with_softmax && (mt & 1) && mt < 2 * kPairTokens) softmax(t + 1, main_pass, mt >> 1);
        }
    };

    TRACE(3);
    for (int pass = kPassMain; pass <= kPassExact; ++pass) {
        const bool main_pass = pass == kPassMain;
        if (tid == 0) *s_abort = 0;
        __syncthreads();  // page window and abort flag ready; the ring is idle
        for (int t = 0; t < 2 && t < ntiles; ++t) issue(t, page_of(t));
        wait_units_newer(min(1, ntiles - 1));  // queries and tile 0 landed
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kChunkBlockTokens; ++j)
#pragma unroll
            for (int mt = 0; mt < 8; ++mt) acc[j][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < kPairTokens; ++j) l_run[j] = 0.f;
        bad = false;

        // tile 0: scores, the reference max (both key halves), probabilities
        TRACE_TILE(0, 11);
        scores(0);
        __syncthreads();
        if (main_pass) {
#pragma unroll
            for (int j = 0; j < kPairTokens; ++j) {
                float raw[4];
                tile_scores(0, j, raw);
                const float hm = wave_max16(fmaxf(fmaxf(raw[0], raw[1]), fmaxf(raw[2], raw[3])) * a.scale_log2);
                if (g == 0) s_hs[(wv * kPairTokens + j) * kHeads + h] = hm;
                m_ref[j] = hm;
            }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kPairTokens; ++j)
                m_ref[j] = fmaxf(m_ref[j], s_hs[(partner * kPairTokens + j) * kHeads + h]);
        }
#pragma unroll
        for (int j = 0; j < kPairTokens; ++j) softmax(0, main_pass, j);
        if (ntiles > 1) wait_dma_all();  // tile 1
        if (__builtin_amdgcn_ballot_w64(bad) != 0 && lane == 0) *s_abort = 1;
        __syncthreads();
        if (2 < ntiles) issue(2, page_of(2));
        // steady state: scores of tile t, then P*V of t - 1 with the softmax of t
        for (int t = 1; t < ntiles; ++t) {
            TRACE_TILE(t, 11);
            const int next_page = page_of(min(t + 2, ntiles - 1));  // consumed after the second barrier
            scores(t);
            __syncthreads();
            TRACE_TILE(t, 12);
            pv(t - 1, true, main_pass);
            TRACE_TILE(t, 15);
            if (t + 1 < ntiles) wait_dma_all();  // tile t + 1
            if (__builtin_amdgcn_ballot_w64(bad) != 0 && lane == 0) *s_abort = 1;
            __syncthreads();
            TRACE_TILE(t, 13);
            if (t + 2 < ntiles) issue(t + 2, next_page);
            TRACE_TILE(t, 14);
        }
        pv(ntiles - 1, false, main_pass);
        // the last barrier passed after every wave's last flag write
        if (!main_pass || __builtin_amdgcn_readfirstlane(*s_abort) == 0) break;
        // abandoned: the exact max of both key halves, then the exact pass
#pragma unroll
        for (int j = 0; j < kPairTokens; ++j) {
            const float hm = wave_max16(m_lane[j]);
            if (g == 0) s_hs[(wv * kPairTokens + j) * kHeads + h] = hm;
            m_ref[j] = hm;
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kPairTokens; ++j) m_ref[j] = fmaxf(m_ref[j], s_hs[(partner * kPairTokens + j) * kHeads + h]);
        __syncthreads();  // every wave read the flag and the maxima
    }

    TRACE(4);
    // per-head sums of each key half, then each wave stores its value-dim slice
#pragma unroll
    for (int j = 0; j < kPairTokens; ++j) {
        const float lh = wave_sum16(l_run[j]);
        if (g == 0) s_hs[(wv * kPairTokens + j) * kHeads + h] = lh;
    }
    __syncthreads();
    TRACE(6);
    auto row_sum = [&](int tb) {  // key half 0 + key half 1, in that order
        const int w0 = 2 * (tb / kPairTokens), jj = tb % kPairTokens;
        return s_hs[(w0 * kPairTokens + jj) * kHeads + h] + s_hs[((w0 + 1) * kPairTokens + jj) * kHeads + h];
    };
#pragma unroll
    for (int j = 0; j < kChunkBlockTokens; ++j) {
        if (j >= nt) break;
        const int row = it.row0 + it.i0 + j;
        if (it.nks_eff == 1) {
            const float inv = 1.f / row_sum(j);
#pragma unroll
            for (int mt = 0; mt < 8; ++mt) store_out4(a, row, h, wv * 128 + mt * 16 + 4 * g, acc[j][mt] * inv);
        } else {
            const size_t prow = (size_t)item * kChunkBlockTokens + j;
            float *po = a.ws_chunk_o + (prow * kHeads + h) * kDv;
#pragma unroll
            for (int mt = 0; mt < 8; ++mt) *reinterpret_cast<f32x4 *>(po + wv * 128 + mt * 16 + 4 * g) = acc[j][mt];
        }
    }
    if (half == 0 && g == 0) {
#pragma unroll
        for (int j = 0; j < kPairTokens; ++j) {
            const int tb = kPairTokens * pair + j;
            if (tb >= nt) break;
            const int row = it.row0 + it.i0 + tb;
            const float l = row_sum(tb);
            if (it.nks_eff == 1) {
                if (a.lse) a.lse[(size_t)row * kHeads + h] = (m_ref[j] + log2f(l)) * kLn2;
            } else {
                const size_t prow = (size_t)item * kChunkBlockTokens + tb;
                a.ws_chunk_ml[(prow * kHeads + h) * 2 + 0] = m_ref[j];
                a.ws_chunk_ml[(prow * kHeads + h) * 2 + 1] = l;
            }
        }
    }
    // fused append: split 0 of a block writes the block's own new latents
    // (nothing in this launch reads those slots, so it can come last)
    if (a.new_kv != nullptr && it.ks == 0) append_rows(a, r, it.p + it.i0, it.row0 + it.i0, it.i1 - it.i0);
    TRACE(5);
}

constexpr int kMainLds = kDecLds > kChunkLds ? kDecLds : kChunkLds;

// Persistent workgroups (one per CU) take work items from a counter in the
// workspace: the chunk items first (largest blocks first), then the decode
// units, whose small size fills the tail.  An item's results and partial
// slots depend only on its index, so the schedule never changes the output
// bits.  The last workgroup to finish zeroes the counters for the next call.
__global__ __launch_bounds__(kThreads, 1) void attention_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) char smem[kMainLds];
    __shared__ int s_tmp[12];
    __shared__ int s_pages[kPageWindow];
    __shared__ DecSeg s_seg[kMaxSeg];
    __shared__ int s_item;
    const int n_items = a.n_chunk_items + a.n_dec_units;
    for (;;) {
        if (threadIdx.x == 0) s_item = __hip_atomic_fetch_add(a.work, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __syncthreads();
        const int item = s_item;
        if (item >= n_items) break;
        TRACE_ITEM(item);
        if (item < a.n_chunk_items)
            chunk_item(a, item, smem, s_tmp, s_pages);
        else
            decode_wg(a, item - a.n_chunk_items, smem, s_tmp, s_pages, s_seg);
        TRACE(7);
        __syncthreads();  // LDS (and s_item) free for the next item
    }
    if (threadIdx.x == 0) {
        const int done = __hip_atomic_fetch_add(a.work + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (done == (int)gridDim.x - 1) {  // every workgroup has taken its last item
            __hip_atomic_store(a.work, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(a.work + 1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// Split merges, after the attention kernel (the kernel boundary makes every
// partial visible): first merge_hsplit workgroups per request (decode rows
// split across units), then one per (chunk item, block row).
__global__ __launch_bounds__(kThreads) void combine_kernel(AttnArgs a) {
    __shared__ int s_tmp[12];
    __shared__ DecSeg s_seg[kMaxSeg];
    const int b = blockIdx.x;
    const int n_dec = a.num_reqs * a.merge_hsplit;
    if (b < n_dec) {
        decode_merge(a, b / a.merge_hsplit, b % a.merge_hsplit, s_tmp);
        return;
    }
    // one workgroup per (chunk item, row of its block): the item with key split
    // 0 merges that row over the block's splits
    const int item = (b - n_dec) / kChunkBlockTokens, j = (b - n_dec) % kChunkBlockTokens;
    Located lc;
    if (!locate_item(item, a.num_reqs, ReqLens{a.cu_q, a.prefix}, ChunkCount{a.ks_chunk}, s_tmp, lc)) return;
    const ChunkItem it = decode_chunk_item(a, lc);
    if (it.ks != 0 || it.nks_eff <= 1 || a.ws_chunk_o == nullptr || j >= it.i1 - it.i0) return;
    if (it.p < 0 || it.row0 < 0 || it.row0 + it.i1 > a.num_rows) return;
    // split ks of this block is item + ks
    merge_row(a, it.row0 + it.i0 + j, it.nks_eff, [&](int ks) {
        const size_t prow = (size_t)(item + ks) * kChunkBlockTokens + j;
        return SplitRef{a.ws_chunk_o + prow * kPartialFloats, a.ws_chunk_ml + prow * kPartialStats};
    });
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

constexpr int kAppendRowsPerWave = 8;

// Each wave copies 8 consecutive rows.  Source rows are loaded first (they do
// not depend on the lookup); the owning requests come from one window of 64
// consecutive cu_q / prefix entries, so a wave needs one dependent round for
// the lengths and one for the page ids.
__global__ __launch_bounds__(kThreads) void append_kernel(AppendArgs a) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int row0 = (blockIdx.x * 4 + wv) * kAppendRowsPerWave;
    if (row0 >= a.num_rows) return;
    const int nrows = min(kAppendRowsPerWave, a.num_rows - row0);
    u32x4 va[kAppendRowsPerWave], vb[kAppendRowsPerWave];
#pragma unroll
    for (int k = 0; k < kAppendRowsPerWave; ++k) {
        va[k] = u32x4{0u, 0u, 0u, 0u};
        vb[k] = u32x4{0u, 0u, 0u, 0u};
        if (k < nrows) {
            const u32x4 *src = reinterpret_cast<const u32x4 *>(a.src + (size_t)(row0 + k) * kDqk);
            va[k] = src[lane];
            if (lane < kChunksPerRow - 64) vb[k] = src[64 + lane];
        }
    }
    const int r0 = a.num_reqs <= 64 ? 0 : find_request(a.cu_q, a.num_reqs, row0, lane);
    const int wi = r0 + lane;
    const int cw = wi <= a.num_reqs ? a.cu_q[wi] : INT_MAX;
    const int pw = wi < a.num_reqs ? a.prefix[wi] : 0;
    int page[kAppendRowsPerWave], slot_in_page[kAppendRowsPerWave];
#pragma unroll
    for (int k = 0; k < kAppendRowsPerWave; ++k) {
        page[k] = -1;
        slot_in_page[k] = 0;
        if (k >= nrows) continue;
        const int row = row0 + k;
        const uint64_t m = __builtin_amdgcn_ballot_w64(cw <= row);
        const int cnt = __builtin_popcountll(m);
        int r, start, pr;
        if (cnt >= 1 && (cnt < 64 || r0 + 64 > a.num_reqs)) {
            r = r0 + cnt - 1;
            start = __shfl(cw, cnt - 1, 64);
            pr = __shfl(pw, cnt - 1, 64);
        } else {  // beyond the window (or inconsistent cu_q): search again
            r = find_request(a.cu_q, a.num_reqs, row, lane);
            start = a.cu_q[r];
            pr = a.prefix[r];
        }
        const int t = pr + (row - start);
        const int lp = t >> a.log2_page;
        if (t >= 0 && lp < a.max_pages && r < a.num_reqs) page[k] = a.bt[(size_t)r * a.max_pages + lp];
        slot_in_page[k] = t & (a.page_size - 1);
    }
#pragma unroll
    for (int k = 0; k < kAppendRowsPerWave; ++k) {
        if (k >= nrows || (unsigned)page[k] >= (unsigned)a.num_pages) continue;
        u32x4 *dst = reinterpret_cast<u32x4 *>(a.kv + ((size_t)page[k] * a.page_size + slot_in_page[k]) * kDqk);
        dst[lane] = va[k];
        if (lane < kChunksPerRow - 64) dst[64 + lane] = vb[k];
    }
}

}  // namespace

#ifdef MLA_TRACE
extern "C" int mla_trace_read(void *dst, size_t bytes) {
    return (int)hipMemcpyFromSymbol(dst, HIP_SYMBOL(g_trace), bytes, 0, hipMemcpyDeviceToHost);
}
#endif

hipError_t launch_append(const AppendArgs &a, hipStream_t s) {
    const int rows_per_block = 4 * kAppendRowsPerWave;
    const int grid = (a.num_rows + rows_per_block - 1) / rows_per_block;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL(append_kernel, dim3(grid), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs &a, hipStream_t s) {
    const int grid = a.grid;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL(attention_kernel, dim3(grid), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_combine(const AttnArgs &a, hipStream_t s) {
    const long long grid_ll = (long long)a.num_reqs * a.merge_hsplit + (long long)a.n_chunk_items * kChunkBlockTokens;
    if (grid_ll > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const int grid = (int)grid_ll;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL(combine_kernel, dim3(grid), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace mla
