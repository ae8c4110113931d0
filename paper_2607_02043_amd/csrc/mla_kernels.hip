// gfx950 kernels of libmlastep: latent append and mixed-step latent attention
// (decode rows and chunked-prefill rows of one step in one launch).
//
// The step is the one a decode node runs when it serves deflected prefill
// chunks next to its in-flight decodes (section 2.3; section 4.3.1, Eq. 4 of
// the paper); the head shapes are those of the served model's absorbed latent
// attention (DeepSeek-V2-Lite, section 6).
//
// Work decomposition (one persistent launch for all rows of a step: one
// 8-wavefront workgroup per CU takes work items from two atomic counters,
// one per kind; the workgroups the host plans as decode-first start on the
// decode items, the others on the chunk items, and each moves to the other
// kind when its own runs out):
//   * chunk rows (c > 1): an item is a block of 8 query tokens (one per
//     wave, 16 head rows each) times a range of its causal keys.  32-key
//     tiles stream through a 3-slot global -> LDS DMA ring; scores on bf16
//     MFMA against a fixed reference max, probabilities to LDS as fp16, and
//     each wave accumulates P*V for its 64 value dims of all 8 tokens on fp16
//     MFMA, V read with transposing LDS reads and converted in registers.
//   * decode rows (c = 1): the decode tiles (32 keys each) of all decode
//     requests form one list cut into equal units; an item is a pair of
//     units, one per 4-wave group of the workgroup, each streaming its tiles
//     through its own 2-slot ring.
// Rows whose keys are split across items leave fp32 partials (the
// unnormalised sum, the max and sum in log2 units); a second, small merge
// kernel combines them in a fixed order.  Results are therefore run-to-run
// deterministic and do not depend on the physical page order.
#include "mla_kernels.h"

#include <limits.h>
#include <math.h>

#include <mutex>

// Scratch of the no-allocation entry point (mixed_step_noalloc): the
// attention workspace (work-queue counters, then split partials) for callers
// that cannot allocate.  Each device holds its own copy until the process
// ends; host code reaches it only through the address that
// hipGetSymbolAddress returns on that device (noalloc_scratch below).
static __device__ __align__(256) unsigned char scratch[mla::kNoAllocScratchBytes];


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
constexpr int kDecRing = 2;                                   // ring slots of each decode wave group
constexpr int kDecGroupBytes = kDecRing * kDecTileBytes;
constexpr int kDecXBytes = 4 * kHeads * 20 * 4;               // partial score blocks of a group
constexpr int kDecLds = 2 * kDecGroupBytes + 2 * kDecXBytes;  // two groups: rings, then score blocks
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

// Sticky error flags of the kernels on this device (MLA_FLAG_* of
// mla_step.h): raised on the rare error paths only, read and cleared by the
// host (mla_device_flags).
__device__ int g_flags;

__device__ __forceinline__ void raise_flag(int f) {
    __hip_atomic_fetch_or(&g_flags, f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

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

// LDS byte offset of 16-byte chunk c of key k inside a decode tile (keys
// row-major, 72 chunks each).  Chunk positions are xor-swizzled inside
// aligned groups of 8 chunks with the key's low 3 bits, so 8 lanes that read
// the same chunk of 8 consecutive keys hit 8 different bank groups.  Chunk
// tiles use their own octet layout (see the chunk section).
__device__ __forceinline__ int tile_swz(int k) { return k & 7; }
__device__ __forceinline__ int tile_off(int k, int c) { return (k * kChunksPerRow + (c ^ tile_swz(k))) * 16; }

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
    bool rev;  // number the items from the last request to the first
};

struct Located {
    int r, local, p, row0, c;
};

template <typename CountFn>
__device__ bool locate_item(int target, int num_reqs, const ReqLens &rl, CountFn count, int *s_tmp,
                            Located &loc) {
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int nthr = blockDim.x, nw = nthr >> 6;
    if (tid == 0) s_tmp[8] = -1;
    int running = 0;
    for (int base = 0; base < num_reqs; base += nthr) {
        const int r = rl.rev ? num_reqs - 1 - (base + tid) : base + tid;
        int cnt = 0, p = 0, row0 = 0, c = 0;
        if (base + tid < num_reqs) {
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
        for (int k = 0; k < nw; ++k) {
            const int t = s_tmp[k];
            off += (k < wv) ? t : 0;
            total += t;
        }
        inc += off;
        const int exc = inc - cnt;
        if (cnt > 0 && target >= running + exc && target < running + inc) {
            s_tmp[8] = r;
            s_tmp[9] = target - running - exc;
            s_tmp[10] = p;
            s_tmp[11] = row0;
            s_tmp[12] = c;
        }
        __syncthreads();
        if (s_tmp[8] >= 0) {  // the same values in every lane: keep them in scalar registers
            loc = Located{__builtin_amdgcn_readfirstlane(s_tmp[8]), __builtin_amdgcn_readfirstlane(s_tmp[9]),
                          __builtin_amdgcn_readfirstlane(s_tmp[10]), __builtin_amdgcn_readfirstlane(s_tmp[11]),
                          __builtin_amdgcn_readfirstlane(s_tmp[12])};
            return true;
        }
        running += total;
    }
    return false;
}

struct ChunkCount {
    int ks;
    ChunkRoute route;
    __device__ int operator()(int p, int c) const {
        return c > 1 && !route.multi_head(p, c) ? ceil_div(c, kChunkBlockTokens) * ceil_div(p + c, ks) : 0;
    }
};

struct ChunkItem {
    int r, p, c, row0, i0, i1, k0, k1, ks, nks_eff;
};

// Item `local` of a chunk request: every block of 8 query tokens (the
// longest rows first) takes nks = ceil((p + c) / ks_chunk) queue slots.  The
// block's keys (0 .. p + i1 - 1, its causal limit klim) are cut into
// ceil(klim / ks_chunk) ranges of equal length, rounded up to a multiple of
// 64 keys (at most ks_chunk); the remaining slots are empty items.  A block
// whose keys fit one range writes its rows directly.
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
    const int kp = ceil_div(ceil_div(klim, ceil_div(klim, a.ks_chunk)), 64) * 64;  // keys per range (<= ks_chunk)
    it.nks_eff = ceil_div(klim, kp);
    it.k0 = it.ks * kp;
    it.k1 = min(klim, it.k0 + kp);
    return it;
}

// Page ids of logical pages [lp0, lp0 + n) of a request into LDS; an id
// outside the pool is replaced by page 0 so no access leaves the pool.
__device__ __forceinline__ void load_page_window(const AttnArgs &a, int r, int lp0, int n, int *s_pages) {
    const int32_t *row = a.bt + (size_t)r * a.max_pages;
    n = min(n, kPageWindow);
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
        const int lp = lp0 + i;
        int pg = lp < a.max_pages ? row[lp] : 0;
        const bool ok = (unsigned)pg < (unsigned)a.num_pages;
        if (!ok) raise_flag(kFlagBadPage);
        s_pages[i] = ok ? pg : 0;
    }
}

// DMA of a 32-key tile that lies inside one page: a uniform source base (the
// tile's first key) in SGPRs plus per-lane offsets fixed for all tiles.
// Round i of wave wv fills LDS chunk u = 256 i + 64 wv + lane of the tile,
// which holds source chunk (u % 72) ^ swz(key) of key u / 72.
constexpr int kTileDma = kKeysPerTile * kRowBytes / (kThreads * 16);  // 9 rounds per tile
// Offsets (< 2^16) packed two per register: round i in the half i & 1 of word i / 2.
__device__ __forceinline__ void tile_dma_offsets(int wv, int lane, uint32_t (&off)[(kTileDma + 1) / 2]) {
#pragma unroll
    for (int w = 0; w < (kTileDma + 1) / 2; ++w) off[w] = 0;
#pragma unroll
    for (int i = 0; i < kTileDma; ++i) {
        const int u = (i * 4 + wv) * 64 + lane;
        const int kk = u / kChunksPerRow;
        const int c = (u - kk * kChunksPerRow) ^ tile_swz(kk);
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
    for (int x = threadIdx.x; x < n * kChunksPerRow; x += blockDim.x) {
        const int i = x / kChunksPerRow, c = x - i * kChunksPerRow;
        const int key = key0 + i;
        const int lp = key >> a.log2_page;
        const int page = lp < a.max_pages ? btr[lp] : -1;
        if ((unsigned)page >= (unsigned)a.num_pages) {
            raise_flag(kFlagBadPage);
            continue;
        }
        const u32x4 v = *reinterpret_cast<const u32x4 *>(a.new_kv + (size_t)(row0 + i) * kDqk + c * 8);
        *reinterpret_cast<u32x4 *>(a.kv_out + ((size_t)page * a.page_size + (key & (a.page_size - 1))) * kDqk +
                                   c * 8) = v;
    }
}

// The same for one 256-thread group of a larger workgroup (gtid = thread index in it).
__device__ __forceinline__ void append_rows_group(const AttnArgs &a, int r, int key0, int row0, int n, int gtid) {
    const int32_t *btr = a.bt + (size_t)r * a.max_pages;
    for (int x = gtid; x < n * kChunksPerRow; x += kThreads) {
        const int i = x / kChunksPerRow, c = x - i * kChunksPerRow;
        const int key = key0 + i;
        const int lp = key >> a.log2_page;
        const int page = lp < a.max_pages ? btr[lp] : -1;
        if ((unsigned)page >= (unsigned)a.num_pages) {
            raise_flag(kFlagBadPage);
            continue;
        }
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
    constexpr int B = NH >= 16 ? 2 : NH >= 4 ? 8 : 16;  // splits whose loads go out together
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
// The 32-key tiles of all decode requests, request after request, form one
// list cut into units of S tiles; unit v owns tiles [v S, (v + 1) S), and a
// decode item is a pair of units, one per 4-wave group of the workgroup
// (the groups run independently, synchronised by LDS arrival counters).  A
// unit's share splits into segments, one per request it touches.  A segment
// streams its query block and then its tiles through the group's 2-slot
// global -> LDS DMA ring, so prefetch runs on across request boundaries and
// the start-up latency is paid once per unit.  Per tile, wave w scores 16
// keys over half of the 576 latent dims (the four partial 16 x 16 score
// blocks meet in LDS), then accumulates its 128-wide slice of the value dims
// over all 32 keys.  A request spread over several units leaves fp32
// partials (slot 2 v for unit v's first segment, 2 v + 1 for its last) that
// the merge kernel combines.
constexpr int kMaxSeg = kMaxDecSegments;
constexpr int kXStride = 20;  // floats per head row of a partial score block (16 + pad)

struct DecSeg {
    int r, p, row, t0, t1, pw, lp0;  // tiles t0 .. t1-1 of request r; page window offset / first page
};

__device__ __forceinline__ int dec_tiles(int p, int c) { return c == 1 ? ceil_div(p + 1, kDecKeys) : 0; }

// Exclusive prefix sum over the threads of the workgroup (uses s_w[0 .. waves - 1]).
__device__ __forceinline__ int block_scan_excl(int v, int *s_w, int &total) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
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
    for (int k = 0; k < nw; ++k) {
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
    for (int base = 0; base < a.num_reqs && running < R1; base += blockDim.x) {
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

// threadIdx.x behind an empty asm: values derived from it inside a work item
// are then computed per item instead of being hoisted out of the persistent
// loop, where they would stay live across both paths and spill to scratch (a
// scratch reload waits on vmcnt, i.e. on every DMA in flight).
__device__ __forceinline__ int item_tid() {
    int t = threadIdx.x;
    asm volatile("" : "+v"(t));
    return t;
}

// Barrier of the four wavefronts of one wave group, through an arrival
// counter in LDS; epoch (wave-uniform) counts the group's barriers so far.
// Each wave first waits for its own LDS accesses, so what it wrote before the
// barrier is visible to the group after it.  The wait is bounded (far beyond
// any real skew): a broken count cannot hang the kernel; an expired wait
// raises kFlagWaitExpired (that call's results are then undefined).
__device__ __forceinline__ void group_barrier(int *ctr, int &epoch, int spin_limit) {
    ++epoch;
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if ((threadIdx.x & 63) == 0) __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    const int target = 4 * epoch;
    int spin = 0;
    for (; spin < spin_limit; ++spin) {
        const int seen = __builtin_amdgcn_readfirstlane(__hip_atomic_load(ctr, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP));
        if (seen >= target) break;
        __builtin_amdgcn_s_sleep(1);
    }
    if (spin == spin_limit && (threadIdx.x & 63) == 0) raise_flag(kFlagWaitExpired);
    asm volatile("" ::: "memory");
}

__device__ void decode_wg(const AttnArgs &a, int w, char *smem, int *s_tmp, int (*s_pages_g)[kPageWindow],
                          DecSeg (*s_seg_g)[kMaxSeg], int *s_gbar) {
    const int tid = item_tid(), lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = wv >> 2, gw = wv & 3, gtid = tid & 255;  // wave group, wave and thread inside it
    const int g = lane >> 4, h = lane & 15;
    const int S = a.dec_unit_tiles;
    // Item w is the pair of decode units 2 w and 2 w + 1 (S tiles each), one per
    // wave group.  Both groups find their segments (block-wide scans).
    int nseg2[2], nunits2[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int R0 = (2 * w + q) * S;
        const int R1 = min(R0 + S, a.dec_total_tiles);
        nseg2[q] = R0 < R1 ? find_segments(a, R0, R1, s_seg_g[q], s_tmp) : 0;
        nunits2[q] = nseg2[q] > 0 ? nseg2[q] + (R1 - R0) : 0;
    }
    TRACE(1);
    const int n_iter = max(nunits2[0], nunits2[1]);
    if (n_iter == 0) return;  // both groups idle (uniform)
    const int v = 2 * w + grp;  // this group's unit
    const int R0 = v * S;
    const int nseg = nseg2[grp], n_units = nunits2[grp];
    DecSeg *const s_seg = s_seg_g[grp];
    int *const s_pages = s_pages_g[grp];
    if (gtid == 0) {  // page-window offsets of the segments
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
        for (int i = gtid; i < n && sg.pw + i < kPageWindow; i += kThreads) {
            const int lp = sg.lp0 + i;
            const int pg = lp < a.max_pages ? btr[lp] : 0;
            const bool ok = (unsigned)pg < (unsigned)a.num_pages;
            if (!ok) raise_flag(kFlagBadPage);
            s_pages[sg.pw + i] = ok ? pg : 0;
        }
    }
    if (a.new_kv != nullptr) {  // fused append: the group holding a request's last tile writes its latent
        for (int j = 0; j < nseg; ++j) {
            const DecSeg sg = s_seg[j];
            if (sg.t1 == dec_tiles(sg.p, 1)) append_rows_group(a, sg.r, sg.p, sg.row, 1, gtid);
        }
    }
    if (tid < 2) s_gbar[tid] = 0;
    __syncthreads();
    if (n_units == 0) return;  // this group has no unit (the other one may)
    int epoch = 0;
    int *const gbar = s_gbar + grp;
    TRACE(2);
    TRACE_VAL(8, 1000000ull * 2 + n_units);

    uint32_t dma_off[(kTileDma + 1) / 2];
    tile_dma_offsets(gw, lane, dma_off);
    const uint32_t ring = lds_addr(smem) + grp * kDecGroupBytes;
    float *s_X = reinterpret_cast<float *>(smem + 2 * kDecGroupBytes + grp * kDecXBytes);
    Cursor prod{0, -1}, cons{0, -1};
    issue_unit(a, s_seg[prod.j], prod.t, s_pages, ring, gw, lane, dma_off);
    advance(prod, s_seg);

    u32x4 qreg[9];  // this wave's half of the query operand: steps 9 (gw >> 1) .. + 9
    f32x4 acc[8];
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_ref = kNegInf, l_run = 0.f;
    const int hf = gw >> 1;
    const int kq = 16 * (gw & 1) + (lane & 15);             // key this lane scores
    const int tr_key = 4 * g + ((lane & 15) >> 2);          // transposing-read source row
    const int tr_dv = gw * 128 + 4 * (lane & 3);            // and its first value dim

    TRACE(3);
    // The two groups run independently, each with barriers of its own four
    // wavefronts (two per unit).
    for (int u = 0; u < n_units; ++u) {
        TRACE_TILE(u, 10);
        wait_dma_all();                // unit u (the only one in flight)
        group_barrier(gbar, epoch, a.spin_limit);    // unit u landed; slot (u + 1) % 2 is free
        bool tile_unit = false;
        DecSeg sg{};
        const char *slot = smem + grp * kDecGroupBytes + (u % kDecRing) * kDecTileBytes;
        {
            if (prod.j < nseg) {
                issue_unit(a, s_seg[prod.j], prod.t, s_pages, ring + ((u + 1) % kDecRing) * kDecTileBytes, gw, lane,
                           dma_off);
                advance(prod, s_seg);
            }
            sg = s_seg[cons.j];
            if (cons.t < 0) {  // a new request: its query block
#pragma unroll
                for (int s2 = 0; s2 < 9; ++s2)
                    qreg[s2] = *reinterpret_cast<const u32x4 *>(slot + (h * kChunksPerRow + (9 * hf + s2) * 4 + g) * 16);
                advance(cons, s_seg);
            } else {
                tile_unit = true;
                TRACE_TILE(u, 11);
                // partial scores: keys 16 (gw & 1) .. + 16, dims of steps 9 hf .. 9 hf + 8
                f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
                u32x4 av[9];
#pragma unroll
                for (int s2 = 0; s2 < 9; ++s2)
                    av[s2] = *reinterpret_cast<const u32x4 *>(slot + tile_off(kq, (9 * hf + s2) * 4 + g));
#pragma unroll
                for (int s2 = 0; s2 < 9; s2 += 2) {
                    sa = mfma_bf16(av[s2], qreg[s2], sa);
                    if (s2 + 1 < 9) sb = mfma_bf16(av[s2 + 1], qreg[s2 + 1], sb);
                }
                *reinterpret_cast<f32x4 *>(s_X + (gw * kHeads + h) * kXStride + 4 * g) = sa + sb;
            }
        }
        if (!tile_unit) continue;
        group_barrier(gbar, epoch, a.spin_limit);  // partial score blocks complete
        TRACE_TILE(u, 12);
        const int kbase = cons.t * kDecKeys;
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
        // Lazy rescale (the same decision in every wave of the group): keep the
        // reference max unless the tile max exceeds it by more than 2^8.
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
                    store_out4(a, sg.row, h, gw * 128 + mt2 * 16 + 4 * g, acc[mt2] * inv);
                if (a.lse && gw == 0 && g == 0) a.lse[(size_t)sg.row * kHeads + h] = (m_ref + log2f(l_tot)) * kLn2;
            } else if (a.ws_dec_o != nullptr) {
                const size_t slot_id = 2 * (size_t)v + (jseg == 0 ? 0 : 1);
                float *po = a.ws_dec_o + (slot_id * kHeads + h) * kDv;
#pragma unroll
                for (int mt2 = 0; mt2 < 8; ++mt2)
                    *reinterpret_cast<f32x4 *>(po + gw * 128 + mt2 * 16 + 4 * g) = acc[mt2];
                if (gw == 0 && g == 0) {
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
    (void)R0;
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
    for (int base = 0; base < r; base += blockDim.x) {
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
// Chunk rows: one workgroup of 8 wavefronts (two per SIMD) per block of 8
// query tokens (128 rows of 16 heads) and a key range of ks_chunk keys;
// 32-key tiles stream through a 3-slot global -> LDS DMA ring.  Two
// wavefronts per SIMD let one issue matrix work while the other waits on LDS
// or runs its softmax.
//  * Scores.  Wave w holds the query of token w (16 heads) over all 576
//    latent dims (18 operands of 32 dims) and forms S^T = K Q^T for two
//    16-key blocks with 16x16x32 MFMAs; nothing is exchanged between waves.
//  * Softmax.  Probabilities against a fixed reference max (no rescaling; see
//    the passes below), written to LDS as fp16 in the B-operand order of P*V:
//    slot 8 g + 4 kt + i of lane (g, head) holds key 16 kt + 4 g + i, which
//    is exactly what the lane's own scores hold, so each lane stores 16 bytes.
//  * P*V.  Wave w accumulates value dims 64 w .. 64 w + 63 of all 8 tokens
//    (4 dim blocks x 8 tokens of 16x16 accumulators); V^T comes from
//    transposing LDS reads with the same key order, converted bf16 -> fp16 in
//    registers (exact for |v| in [2^-14, 65504]).
// Per tile: one barrier.  After it, the P*V of tile t and the scores of tile
// t+1 run back to back (their operands come from different ring slots and P
// buffers), then the softmax of tile t+1 fills the other P buffer.

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

constexpr int kCT = kChunkBlockTokens;                 // 8 tokens per item, one per wave
constexpr int kQSteps = kDqk / 32;                     // 18 query operands of 32 dims
constexpr int kQRegSteps = 16;                         // the first 16 stay in registers, the rope ones in LDS
constexpr int kChunkRing = 3;
constexpr int kPTile = kCT * 64 * 16;                  // fp16 P of one tile: [token][lane] 16 bytes
constexpr int kQLdsBytes = (kQSteps - kQRegSteps) * kCT * 64 * 16;  // rope query operands: [step][token][lane]
constexpr int kChunkLds = kChunkRing * kChunkTileBytes + 2 * kPTile + kQLdsBytes + 2 * kCT * kHeads * 4 + 16;
// Largest exponent (log2 units) a probability may take against the reference
// max: 2^15 stays inside fp16.
constexpr float kMaxPExp = 15.f;

// Chunk tiles are laid out by octets of chunks: 16-byte chunk c (8 latent
// dims) of tile key k (0..31) sits at position 256 (c >> 3) + 8 k +
// ((c & 7) ^ (k & 7)), i.e. the eight chunks (128 bytes) of a key that share
// an octet stay together, xor-swizzled with the key's low three bits.  One
// DMA round (64 positions) then reads eight keys' 128-byte pieces, one cache
// line per key, and the 16-key operand reads keep the bank pattern of a
// row-major tile (conflict-free).  Round j fills octet j >> 2, keys
// 8 (j & 3) .. + 7: lane l loads chunk 8 (j >> 2) + ((l & 7) ^ ((l >> 3) & 7))
// of key 8 (j & 3) + (l >> 3).
// The instruction offset OFF moves the LDS destination as well as the
// global source, so M0 is set to lds_base - OFF.
template <int OFF>
__device__ __forceinline__ void lds_dma16_imm(const void *gsrc, uint32_t lds_base) {
    asm volatile(
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off offset:%2\n\t"
        :
        : "{m0}"(lds_base - OFF), "v"(gsrc), "i"(OFF)
        : "memory");
}
template <int OFF>
__device__ __forceinline__ void lds_dma16_sbase_imm(const void *sbase, uint32_t voff, uint32_t lds_base) {
    asm volatile(
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %0, %1 offset:%3\n\t"
        :
        : "v"(voff), "s"(sbase), "{m0}"(lds_base - OFF), "i"(OFF)
        : "memory");
}

// Passes of a chunk item.  The reference max of each row is fixed for the
// whole key range, so the accumulators are never rescaled:
//   main    reference = max of the first tile.  Each lane also tracks the max
//           of every score it sees.  If a later score exceeds the reference by
//           more than 2^15, the pass still runs to the end and its products
//           are discarded;
//   exact   then the item runs again against the exact max.

// Returns true when the main pass was abandoned: the caller then runs the
// item again with exact = true (the exact maxima wait in LDS).
__device__ bool chunk_item(const AttnArgs &a, int item, char *smem, int *s_tmp, int *s_pages, bool exact) {
    Located lc;
    if (!locate_item(item, a.num_reqs, ReqLens{a.cu_q, a.prefix, a.chunk_rev != 0}, ChunkCount{a.ks_chunk, a.route}, s_tmp, lc)) return false;
    const ChunkItem it = decode_chunk_item(a, lc);
    TRACE(1);
    const int r = it.r;
    if (it.k0 >= it.k1) return false;  // key range past this block's causal limit
    if (it.p < 0 || it.row0 < 0 || it.row0 + it.i1 > a.num_rows) return false;
    if (it.nks_eff > 1 && a.ws_chunk_o == nullptr) return false;
    const int tid = item_tid(), lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, hd = lane & 15;
    const int nt = it.i1 - it.i0;  // tokens of this block (1 .. 8)
    const int ntiles = ceil_div(it.k1 - it.k0, kChunkKeys);
    const int lp0 = it.k0 >> a.log2_page;
    // This wave's token (an idle token repeats the last one; its results are
    // not stored).  Query operands: lane l holds dims 32 s + 8 g .. + 7 of
    // head hd, s = 0..17 (issued first: their latency overlaps the page-window
    // load).
    const int tk = min(wv, nt - 1);
    u32x4 qreg[kQRegSteps];
    char *const s_q = smem + kChunkRing * kChunkTileBytes + 2 * kPTile;  // rope query operands
    {
        const uint16_t *qp = a.q + ((size_t)(it.row0 + it.i0 + tk) * kHeads + hd) * kDqk + 8 * g;
#pragma unroll
        for (int s = 0; s < kQRegSteps; ++s) qreg[s] = *reinterpret_cast<const u32x4 *>(qp + 32 * s);
        u32x4 qr[kQSteps - kQRegSteps];
#pragma unroll
        for (int s = kQRegSteps; s < kQSteps; ++s) qr[s - kQRegSteps] = *reinterpret_cast<const u32x4 *>(qp + 32 * s);
#pragma unroll
        for (int s = 0; s < kQSteps - kQRegSteps; ++s)
            *reinterpret_cast<u32x4 *>(s_q + ((s * kCT + wv) * 64 + lane) * 16) = qr[s];
    }
    load_page_window(a, r, lp0, ((it.k1 - 1) >> a.log2_page) - lp0 + 1, s_pages);
    // The query loads must count as complete before the tile DMAs go out: a
    // wait the compiler places later for them would also wait for those DMAs.
#pragma unroll
    for (int s = 0; s < kQRegSteps; ++s) asm volatile("" : "+v"(qreg[s]));
    TRACE(2);
    TRACE_VAL(8, 1000000ull * 1 + ntiles);

    const uint32_t ring = lds_addr(smem);
    char *const s_pbuf = smem + kChunkRing * kChunkTileBytes;           // [2][token][lane] 16 bytes
    float *const s_l = reinterpret_cast<float *>(s_q + kQLdsBytes);     // [token][head] row sums
    float *const s_mx = s_l + kCT * kHeads;                            // [token][head] exact maxima
    int *const s_abort = reinterpret_cast<int *>(s_mx + kCT * kHeads);

    // Causal limit of this wave's token (absolute key index, clipped to the
    // item's key range); wave-uniform.
    const int lim = __builtin_amdgcn_readfirstlane(min(it.p + it.i0 + tk, it.k1 - 1));

    // K operand of key block kb, step s (keys 16 kb + hd, dims 32 s + 8 g ..):
    // chunk 4 s + g, at kq_off[s & 1] + 2048 kb + 4096 (s >> 1).
    int kq_off[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) kq_off[e] = 128 * hd + 16 * ((4 * e + g) ^ (hd & 7));
    // V^T operand of value block db (dims 64 wv + 16 db + (lane & 15)): two
    // transposing reads of keys tr_key .. + 3 and tr_key + 16 .. + 3 at dims
    // 64 wv + 16 db + 4 (lane & 3) .. + 3, i.e. chunk 8 wv + 2 db + b with
    // b = (lane >> 1) & 1: vt_off[db] (+ 2048 for the second read).
    const int tr_key = 4 * g + ((lane & 15) >> 2);
    int vt_off[4];
#pragma unroll
    for (int db = 0; db < 4; ++db)
        vt_off[db] = 4096 * wv + 128 * tr_key + 16 * ((2 * db + ((lane >> 1) & 1)) ^ (tr_key & 7)) + 8 * (lane & 1);

    // DMA of tile t into its ring slot, issued by waves 4..7 only (nine rounds
    // each: round i = (wv - 4) + 4 j).  Issuing stalls a wave for a while; the
    // other wave of the same SIMD meanwhile runs ahead on its matrix work, so
    // the two wavefronts of a SIMD drift apart by about that much and the
    // softmax of one overlaps the products of the other.  A full tile inside
    // one page takes a uniform (scalar) base; any other tile (small pages, the
    // last partial tile, new latents of a fused append) one address per lane.
    const bool dma_wave = wv >= 4;
    const int dw = wv & 3;
    const int dkey = 8 * dw + (lane >> 3);  // this lane's key in every round of this wave
    const uint32_t dvoff = dkey * kRowBytes + 16 * ((lane & 7) ^ ((lane >> 3) & 7));
    const bool in_page = a.page_size >= kChunkKeys;
    const int cached_end = a.new_kv != nullptr ? min(it.k1, it.p) : it.k1;
    auto page_of = [&](int t) {
        return s_pages[min(((it.k0 + t * kChunkKeys) >> a.log2_page) - lp0, kPageWindow - 1)];
    };
    auto issue = [&](int t, int slot, int page) {
        if (!dma_wave) return;
        const int kbase = it.k0 + t * kChunkKeys;
        const uint32_t dst = ring + slot * kChunkTileBytes + dw * 1024;  // round r = dw + 4 r'
        if (in_page && kbase + kChunkKeys <= cached_end) {
            const char *src = reinterpret_cast<const char *>(a.kv) +
                              ((size_t)__builtin_amdgcn_readfirstlane(page) * a.page_size +
                               (kbase & (a.page_size - 1))) * kRowBytes;
#define MLA_CHUNK_DMA_S(r) lds_dma16_sbase_imm<128 * (r)>(src, dvoff, __builtin_amdgcn_readfirstlane(dst + 4096 * (r)))
            MLA_CHUNK_DMA_S(0); MLA_CHUNK_DMA_S(1); MLA_CHUNK_DMA_S(2); MLA_CHUNK_DMA_S(3); MLA_CHUNK_DMA_S(4);
            MLA_CHUNK_DMA_S(5); MLA_CHUNK_DMA_S(6); MLA_CHUNK_DMA_S(7); MLA_CHUNK_DMA_S(8);
#undef MLA_CHUNK_DMA_S
        } else {
            // keys past the item's range repeat its last key (a finite cached latent)
            const int key = min(kbase + dkey, it.k1 - 1);
            const char *gs;
            if (a.new_kv != nullptr && key >= it.p) {
                gs = reinterpret_cast<const char *>(a.new_kv) + (size_t)(it.row0 + key - it.p) * kRowBytes;
            } else {
                const int pg = s_pages[min((key >> a.log2_page) - lp0, kPageWindow - 1)];
                gs = reinterpret_cast<const char *>(a.kv) +
                     ((size_t)pg * a.page_size + (key & (a.page_size - 1))) * kRowBytes;
            }
            gs += 16 * ((lane & 7) ^ ((lane >> 3) & 7));
#define MLA_CHUNK_DMA_V(r) lds_dma16_imm<128 * (r)>(gs, __builtin_amdgcn_readfirstlane(dst + 4096 * (r)))
            MLA_CHUNK_DMA_V(0); MLA_CHUNK_DMA_V(1); MLA_CHUNK_DMA_V(2); MLA_CHUNK_DMA_V(3); MLA_CHUNK_DMA_V(4);
            MLA_CHUNK_DMA_V(5); MLA_CHUNK_DMA_V(6); MLA_CHUNK_DMA_V(7); MLA_CHUNK_DMA_V(8);
#undef MLA_CHUNK_DMA_V
        }
    };

    float m_ref = kNegInf, m_lane = kNegInf, l_run = 0.f;
    f32x4 acc[kCT][4];  // [token][value block db]
    bool bad = false;

    // S^T of tile t for this wave's token: lane l, element i of block kb =
    // key 16 kb + 4 g + i of the tile, head hd.  Two accumulation chains.
    auto scores = [&](int slot, f32x4 (&s)[2]) {
        const char *tile = smem + __builtin_amdgcn_readfirstlane(slot * kChunkTileBytes);
        s[0] = s[1] = f32x4{0.f, 0.f, 0.f, 0.f};
        constexpr int D = 2;  // steps whose K operands are in flight
        u32x4 av[D][2];
#pragma unroll
        for (int st = 0; st < D; ++st)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
                av[st][kb] = *reinterpret_cast<const u32x4 *>(tile + kq_off[st & 1] + 2048 * kb + 4096 * (st >> 1));
#pragma unroll
        for (int st = 0; st < kQSteps; ++st) {
            u32x4 cur[2] = {av[st % D][0], av[st % D][1]};
            if (st + D < kQSteps) {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
                    av[st % D][kb] = *reinterpret_cast<const u32x4 *>(tile + kq_off[(st + D) & 1] + 2048 * kb +
                                                                      4096 * ((st + D) >> 1));
            }
            u32x4 qb;
            if (st < kQRegSteps)
                qb = qreg[st];
            else
                qb = *reinterpret_cast<const u32x4 *>(s_q + (((st - kQRegSteps) * kCT + wv) * 64 + lane) * 16);
            s[0] = mfma_bf16(cur[0], qb, s[0]);
            s[1] = mfma_bf16(cur[1], qb, s[1]);
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // masked raw scores of tile t
    auto masked = [&](int t, const f32x4 (&s)[2], float (&x)[8]) {
        const int kbase = it.k0 + t * kChunkKeys;
        if (kbase + kChunkKeys - 1 <= lim) {
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = s[e >> 2][e & 3];
        } else {
            const int rel = lim - kbase - 4 * g;
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = (16 * (e >> 2) + (e & 3) <= rel) ? s[e >> 2][e & 3] : kNegInf;
        }
    };
    auto lane_max = [&](const float (&x)[8]) {
        return fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])), fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
    };
    auto softmax = [&](int t, int pbuf, const f32x4 (&s)[2], bool main_pass) {
        float x[8];
        masked(t, s, x);
        const float xm = lane_max(x) * a.scale_log2;
        m_lane = fmaxf(m_lane, xm);
        // also true for a first visible key after the first tile
        bad |= main_pass && xm - m_ref > kMaxPExp;
        // the scaled score is rounded before the max is subtracted, so the max
        // key gets p = 1 exactly; masked scores give p = 0
        const float mref = m_ref == kNegInf ? 0.f : m_ref;
        float p[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
#pragma clang fp contract(off)
            p[e] = __builtin_amdgcn_exp2f(x[e] * a.scale_log2 - mref);
        }
        l_run += ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
        *reinterpret_cast<u32x4 *>(s_pbuf + __builtin_amdgcn_readfirstlane(pbuf * kPTile) + (wv * 64 + lane) * 16) =
            u32x4{f16x2_bits(p[0], p[1]), f16x2_bits(p[2], p[3]), f16x2_bits(p[4], p[5]), f16x2_bits(p[6], p[7])};
    };
    // O^T += V^T P^T for tile t (P from buffer t & 1)
    auto pv = [&](int slot, int pbuf) {
        const char *tile = smem + __builtin_amdgcn_readfirstlane(slot * kChunkTileBytes);
        const char *pb = s_pbuf + __builtin_amdgcn_readfirstlane(pbuf * kPTile) + lane * 16;
        constexpr int PD = 3;  // P operands in flight
        u32x4 bp[PD];
#pragma unroll
        for (int tb = 0; tb < PD; ++tb) bp[tb] = *reinterpret_cast<const u32x4 *>(pb + tb * 64 * 16);
        u32x4 av[4];
#pragma unroll
        for (int db = 0; db < 4; ++db) {
            const u32x2 lo = lds_read_tr16(tile + vt_off[db]);
            const u32x2 hi = lds_read_tr16(tile + vt_off[db] + 2048);
            av[db] = u32x4{bf16x2_to_f16x2(lo[0]), bf16x2_to_f16x2(lo[1]), bf16x2_to_f16x2(hi[0]),
                           bf16x2_to_f16x2(hi[1])};
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int tb = 0; tb < kCT; ++tb) {
            const u32x4 cur = bp[tb % PD];
            if (tb + PD < kCT) bp[tb % PD] = *reinterpret_cast<const u32x4 *>(pb + (tb + PD) * 64 * 16);
#pragma unroll
            for (int db = 0; db < 4; ++db) acc[tb][db] = mfma_f16(av[db], cur, acc[tb][db]);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    TRACE(3);
    const bool main_pass = !exact;
    if (exact) m_ref = s_mx[wv * kHeads + hd];
    if (tid == 0) *s_abort = 0;
    __syncthreads();  // page window and abort flag ready; the ring is idle
    for (int t = 0; t < 2 && t < ntiles; ++t) issue(t, t, page_of(t));
    // queries and tile 0 landed (tile 1's nine rounds may still be in flight)
    if (ntiles == 1 || !dma_wave)
        wait_dma_all();
    else
        wait_dma_keep9();
    __syncthreads();
#pragma unroll
    for (int tb = 0; tb < kCT; ++tb)
#pragma unroll
        for (int db = 0; db < 4; ++db) acc[tb][db] = f32x4{0.f, 0.f, 0.f, 0.f};

    // tile 0: scores, the reference max, probabilities
    TRACE_TILE(0, 11);
    {
        f32x4 s0[2];
        scores(0, s0);
        if (main_pass) {
            float x[8];
            masked(0, s0, x);
            m_ref = wave_max16(lane_max(x) * a.scale_log2);
        }
        softmax(0, 0, s0, main_pass);
    }
    int slot = 0;  // ring slot of tile t (t % 3)
    // steady state: after the barrier, P*V of tile t and the scores of t + 1,
    // then the softmax of t + 1
    for (int t = 0; t < ntiles; ++t) {
        TRACE_TILE(t, 11);
        const int next_page = page_of(min(t + 2, ntiles - 1));
        if (t + 1 < ntiles) wait_dma_all();  // tile t + 1 (this wave's part)
        if (__builtin_amdgcn_ballot_w64(bad) != 0 && lane == 0) *s_abort = 1;
        __syncthreads();  // tile t + 1 and P of tile t complete; slot (t + 2) % 3 and P buffer (t + 1) & 1 free
        TRACE_TILE(t, 12);
        const int slot1 = slot == kChunkRing - 1 ? 0 : slot + 1;
        const int slot2 = slot1 == kChunkRing - 1 ? 0 : slot1 + 1;
        if (t + 2 < ntiles) issue(t + 2, slot2, next_page);
        TRACE_TILE(t, 14);
        pv(slot, t & 1);
        TRACE_TILE(t, 15);
        if (t + 1 < ntiles) {
            f32x4 s1[2];
            scores(slot1, s1);
            softmax(t + 1, (t + 1) & 1, s1, main_pass);
        }
        slot = slot1;
        TRACE_TILE(t, 13);
    }
    __syncthreads();  // every wave's last flag write and P*V reads are done
    if (main_pass && __builtin_amdgcn_readfirstlane(*s_abort) != 0) {
        // abandoned: publish the exact maxima for the exact pass
        const float mx = wave_max16(m_lane);
        if (g == 0) s_mx[wv * kHeads + hd] = mx;
        __syncthreads();
        return true;
    }

    TRACE(4);
    // row sums of this wave's token
    {
        const float lt = wave_sum16(l_run);
        if (g == 0) s_l[wv * kHeads + hd] = lt;
    }
    __syncthreads();
    TRACE(6);
    // acc[tb][db] element i: value dim 64 wv + 16 db + 4 g + i of token tb, head hd
#pragma unroll
    for (int tb = 0; tb < kCT; ++tb) {
        if (tb >= nt) break;
        const int row = it.row0 + it.i0 + tb;
        if (it.nks_eff == 1) {
            const float inv = 1.f / s_l[tb * kHeads + hd];
#pragma unroll
            for (int db = 0; db < 4; ++db) store_out4(a, row, hd, 64 * wv + 16 * db + 4 * g, acc[tb][db] * inv);
        } else {
            const size_t prow = (size_t)item * kCT + tb;
            float *po = a.ws_chunk_o + (prow * kHeads + hd) * kDv + 64 * wv + 4 * g;
#pragma unroll
            for (int db = 0; db < 4; ++db) *reinterpret_cast<f32x4 *>(po + 16 * db) = acc[tb][db];
        }
    }
    if (g == 0 && wv < nt) {
        const int row = it.row0 + it.i0 + wv;
        const float l = s_l[wv * kHeads + hd];
        if (it.nks_eff == 1) {
            if (a.lse) a.lse[(size_t)row * kHeads + hd] = (m_ref + log2f(l)) * kLn2;
        } else {
            const size_t prow = (size_t)item * kCT + wv;
            a.ws_chunk_ml[(prow * kHeads + hd) * 2 + 0] = m_ref;
            a.ws_chunk_ml[(prow * kHeads + hd) * 2 + 1] = l;
        }
    }
    // fused append: split 0 of a block writes the block's own new latents
    // (nothing in this launch reads those slots, so it can come last)
    if (a.new_kv != nullptr && it.ks == 0) append_rows(a, r, it.p + it.i0, it.row0 + it.i0, it.i1 - it.i0);
    TRACE(5);
    return false;
}

constexpr int kMainLds = kDecLds > kChunkLds ? kDecLds : kChunkLds;

// Persistent workgroups (one per CU) take work items from two counters in
// the workspace, one per queue: the chunk items (largest blocks first) and
// the decode items.  Workgroups below dec_first_wgs start on the decode
// queue, the others on the chunk queue, and each moves to the other queue
// once its own is empty: with no decode-first workgroups the decode units
// fill the tail after the chunk items; with some, decode streaming runs
// beside the chunk tiles from the start.  An item's results and partial
// slots depend only on its index, so the schedule never changes the output
// bits.  The last workgroup to finish zeroes the counters for the next call.
__global__ __launch_bounds__(kAttnThreads, 1) void attention_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) char smem[kMainLds];
    __shared__ int s_tmp[16];
    __shared__ int s_pages[2][kPageWindow];  // chunk items use the first window
    __shared__ DecSeg s_seg[2][kMaxSeg];
    __shared__ int s_gbar[2];
    __shared__ int s_item;
    bool on_dec = (int)blockIdx.x < a.dec_first_wgs;  // thread 0's current queue
    for (;;) {
        if (threadIdx.x == 0) {
            // the current queue, then the other one: -1 once both are empty
            int it = -1;
            for (int k = 0; k < 2 && it < 0; ++k) {
                if (on_dec) {
                    const int d = __hip_atomic_fetch_add(a.work + 2, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (d < a.n_dec_units) it = a.n_chunk_items + d;
                } else {
                    const int c = __hip_atomic_fetch_add(a.work, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (c < a.n_chunk_items) it = c;
                }
                if (it < 0) on_dec = !on_dec;
            }
            s_item = it;
        }
        __syncthreads();
        const int item = s_item;
        if (item < 0) break;
        TRACE_ITEM(item);
        if (item < a.n_chunk_items) {
            // a second, exact pass only if the main one was abandoned
            for (int pass = 0; pass < 2; ++pass) {
                if (!chunk_item(a, item, smem, s_tmp, s_pages[0], pass != 0)) break;
                __syncthreads();
            }
        }
        else
            decode_wg(a, item - a.n_chunk_items, smem, s_tmp, s_pages, s_seg, s_gbar);
        TRACE(7);
        __syncthreads();  // LDS (and s_item) free for the next item
    }
    if (threadIdx.x == 0) {
        const int done = __hip_atomic_fetch_add(a.work + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (done == (int)gridDim.x - 1) {  // every workgroup has taken its last item
            __hip_atomic_store(a.work, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(a.work + 1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(a.work + 2, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// Merge workgroups of split decode rows (none when no decode row was split).
__host__ __device__ __forceinline__ int merge_dec_wgs(const AttnArgs &a) {
    return a.ws_dec_o != nullptr ? a.num_reqs * a.merge_hsplit : 0;
}

// Split merges, after the attention kernel (the kernel boundary makes every
// partial visible): first merge_hsplit workgroups per request (decode rows
// split across units), then one per (chunk item, block row).
__global__ __launch_bounds__(kThreads) void combine_kernel(AttnArgs a) {
    __shared__ int s_tmp[16];
    const int b = blockIdx.x;
    const int n_dec = merge_dec_wgs(a);
    if (b < n_dec) {
        decode_merge(a, b / a.merge_hsplit, b % a.merge_hsplit, s_tmp);
        return;
    }
    // one workgroup per (chunk item, row of its block): the item with key split
    // 0 merges that row over the block's splits
    const int item = (b - n_dec) / kChunkBlockTokens, j = (b - n_dec) % kChunkBlockTokens;
    Located lc;
    if (!locate_item(item, a.num_reqs, ReqLens{a.cu_q, a.prefix, a.chunk_rev != 0}, ChunkCount{a.ks_chunk, a.route}, s_tmp, lc)) return;
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
        if (k >= nrows) continue;
        if ((unsigned)page[k] >= (unsigned)a.num_pages) {
            raise_flag(kFlagBadPage);
            continue;
        }
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

hipError_t noalloc_scratch(void **ptr) {
    static std::mutex mu;
    static void *addr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(mu);
    if (addr[dev] == nullptr) {
        // once per device, with that device current: its copy's address, and
        // the work-queue counters cleared (every completed call leaves them zero)
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        static const unsigned char zeros[256] = {};
        e = hipMemcpy(p, zeros, sizeof zeros, hipMemcpyHostToDevice);
        if (e != hipSuccess) return e;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

hipError_t read_flags(int *flags, bool clear) {
    hipError_t e = hipMemcpyFromSymbol(flags, HIP_SYMBOL(g_flags), sizeof(int), 0, hipMemcpyDeviceToHost);
    if (e != hipSuccess || !clear || *flags == 0) return e;
    const int zero = 0;
    return hipMemcpyToSymbol(HIP_SYMBOL(g_flags), &zero, sizeof(int), 0, hipMemcpyHostToDevice);
}

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
    hipLaunchKernelGGL(attention_kernel, dim3(grid), dim3(kAttnThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_combine(const AttnArgs &a, hipStream_t s) {
    // only the kinds that left partials get workgroups
    const long long grid_ll =
        (long long)merge_dec_wgs(a) + (a.ws_chunk_o != nullptr ? (long long)a.n_chunk_items * kChunkBlockTokens : 0);
    if (grid_ll > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const int grid = (int)grid_ll;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL(combine_kernel, dim3(grid), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace mla
