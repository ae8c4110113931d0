// C ABI of libmlastep: argument checks, work planning and launches.
// The entry points and their contracts are declared in include/mla_step.h.
#include "mla_step.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <algorithm>
#include <mutex>
#include <vector>

#include "mla_kernels.h"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int hip_fail(hipError_t e, const char *what) {
    return fail(MLA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Compute units of the current device (cached per device ordinal).
int cu_count(int *status) {
    static std::mutex mu;
    static int cache[64] = {0};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        *status = hip_fail(e, "hipGetDevice");
        return 0;
    }
    if (dev < 0 || dev >= 64) dev = 0;
    std::lock_guard<std::mutex> lk(mu);
    if (cache[dev] == 0) {
        int n = 0;
        e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess || n <= 0) {
            *status = hip_fail(e, "hipDeviceGetAttribute(multiProcessorCount)");
            return 0;
        }
        cache[dev] = n;
    }
    return cache[dev];
}

int ilog2_exact(int v) {
    int l = 0;
    while ((1 << l) < v) ++l;
    return (1 << l) == v ? l : -1;
}

long long ceil_div_ll(long long a, long long b) { return (a + b - 1) / b; }

struct Shape {
    int R = 0;
    int T = 0;
    int log2_page = 0;
};

// Host checks shared by both entry points.
int check_batch(const mla_batch *b, Shape *sh) {
    g_err[0] = '\0';
    if (!b) return fail(MLA_ERR_INVALID_ARG, "batch is NULL");
    if (b->num_reqs < 0) return fail(MLA_ERR_INVALID_ARG, "num_reqs = %d < 0", b->num_reqs);
    sh->R = b->num_reqs;
    if (b->num_reqs == 0) return MLA_OK;
    const int lg = ilog2_exact(b->page_size);
    if (b->page_size < 1 || b->page_size > 1024 || lg < 0)
        return fail(MLA_ERR_UNSUPPORTED, "page_size = %d is not a power of two in [1, 1024]", b->page_size);
    sh->log2_page = lg;
    if (b->num_pages < 1) return fail(MLA_ERR_INVALID_ARG, "num_pages = %d < 1", b->num_pages);
    if (b->max_pages_per_req < 1)
        return fail(MLA_ERR_INVALID_ARG, "max_pages_per_req = %d < 1", b->max_pages_per_req);
    if (!b->q_lens || !b->prefix_lens) return fail(MLA_ERR_INVALID_ARG, "host q_lens / prefix_lens is NULL");
    if (!b->cu_q_dev || !b->prefix_lens_dev || !b->block_table_dev)
        return fail(MLA_ERR_INVALID_ARG, "a device batch array is NULL");
    const long long cap = (long long)b->max_pages_per_req * b->page_size;
    long long T = 0;
    for (int r = 0; r < b->num_reqs; ++r) {
        const long long c = b->q_lens[r], p = b->prefix_lens[r];
        if (c < 1) return fail(MLA_ERR_INVALID_ARG, "q_lens[%d] = %lld < 1", r, c);
        if (p < 0) return fail(MLA_ERR_INVALID_ARG, "prefix_lens[%d] = %lld < 0", r, p);
        if (p + c > cap)
            return fail(MLA_ERR_INVALID_ARG, "request %d: prefix %lld + q_len %lld exceeds the block table (%lld keys)",
                        r, p, c, cap);
        if (p + c > (1LL << 30)) return fail(MLA_ERR_INVALID_ARG, "request %d: more than 2^30 keys", r);
        T += c;
        if (T > (1LL << 30) / mla::kHeads) return fail(MLA_ERR_INVALID_ARG, "too many rows in the step");
    }
    sh->T = (int)T;
    return MLA_OK;
}

struct Plan {
    int ks_chunk = 0, n_chunk_items = 0;
    int n_dec_wg = 0, dec_tiles_per_wg = 0, dec_total_tiles = 0;
    bool chunk_split = false, dec_split = false;
    size_t off_chunk_o = 0, off_chunk_ml = 0, off_dec_o = 0, off_dec_ml = 0, bytes = 0;
};

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// Rough per-CU costs used only to balance the two kinds of work (us).
constexpr double kChunkTileUs = 3.2;      // 4 tokens x 32 keys on one CU
constexpr double kCuStreamGBs = 50.0;     // one CU streaming alone
constexpr double kChipStreamGBs = 6300.0; // all CUs streaming together

struct DecReq {
    long long first_tile, tiles, p;
};

// Does a decode share of S tiles per workgroup respect the kernel's limits
// (segments and page-window entries per workgroup)?
bool dec_share_fits(const std::vector<DecReq> &reqs, long long total, long long S, int page_size) {
    size_t k = 0;
    for (long long R0 = 0; R0 < total; R0 += S) {
        const long long R1 = std::min(R0 + S, total);
        while (k < reqs.size() && reqs[k].first_tile + reqs[k].tiles <= R0) ++k;
        long long segs = 0, pages = 0;
        for (size_t j = k; j < reqs.size() && reqs[j].first_tile < R1; ++j) {
            const long long t0 = std::max(R0 - reqs[j].first_tile, 0LL);
            const long long t1 = std::min(R1 - reqs[j].first_tile, reqs[j].tiles);
            const long long k0 = t0 * mla::kKeysPerTile;
            const long long klast = std::min(t1 * mla::kKeysPerTile, reqs[j].p + 1) - 1;
            pages += klast / page_size - k0 / page_size + 1;
            ++segs;
        }
        if (segs > mla::kMaxDecSegments || pages > mla::kPageWindow) return false;
    }
    return true;
}

// Work layout of one call.
//  * chunk requests -> items of (4 tokens) x (ks_chunk keys), longest rows
//    first; key ranges are split only when the chunk is too small to give the
//    chip enough items.
//  * decode requests -> one list of 32-key tiles cut into equal shares for
//    n_dec_wg persistent workgroups; n_dec_wg balances the decode stream
//    against the chunk work that runs on the remaining compute units.
// The device recomputes the same mapping from the device copies of the lengths.
int make_plan(const mla_batch *b, const Shape &sh, Plan *pl) {
    if (sh.R == 0) return MLA_OK;
    int st = MLA_OK;
    const int ncu = cu_count(&st);
    if (st != MLA_OK) return st;
    const long long P = b->page_size;
    long long cap = ((long long)(mla::kPageWindow - 1) * P) / 64 * 64;  // keys per chunk item
    if (cap < 64) cap = 64;
    const int BM = mla::kChunkBlockTokens, KT = mla::kKeysPerTile;

    std::vector<DecReq> dec;
    long long chunk_blocks = 0, chunk_block_keys = 0, dec_total = 0;
    for (int r = 0; r < sh.R; ++r) {
        const long long c = b->q_lens[r], p = b->prefix_lens[r];
        if (c == 1) {
            const long long nt = ceil_div_ll(p + 1, KT);
            dec.push_back(DecReq{dec_total, nt, p});
            dec_total += nt;
        } else {
            const long long nrb = ceil_div_ll(c, BM);
            chunk_blocks += nrb;
            for (long long rb = 0; rb < nrb; ++rb) chunk_block_keys += p + std::min(c, (rb + 1) * BM);
        }
    }
    if (dec_total > (1LL << 30)) return fail(MLA_ERR_INVALID_ARG, "too many decode keys in the step");
    // chunk items
    const long long target = 2LL * ncu;
    long long ks_chunk = cap;
    if (chunk_blocks > 0 && chunk_blocks < target) {
        ks_chunk = std::max<long long>(128, ceil_div_ll(ceil_div_ll(chunk_block_keys, target), 64) * 64);
        ks_chunk = std::min(ks_chunk, cap);
    }
    long long nci = 0;
    for (int r = 0; r < sh.R; ++r) {
        const long long c = b->q_lens[r], p = b->prefix_lens[r];
        if (c == 1) continue;
        nci += ceil_div_ll(c, BM) * ceil_div_ll(p + c, ks_chunk);
        if (p + c > ks_chunk) pl->chunk_split = true;
    }
    if (nci > (1LL << 27)) return fail(MLA_ERR_INVALID_ARG, "step needs too many work items");
    pl->ks_chunk = (int)ks_chunk;
    pl->n_chunk_items = (int)nci;
    // decode shares
    if (dec_total > 0) {
        const double chunk_us = (double)ceil_div_ll(chunk_block_keys, KT) * kChunkTileUs;
        long long best_g = std::min<long long>(ncu, dec_total);
        if (chunk_us > 0.0 && ncu > 1) {
            double best = 1e300;
            for (long long g = 1; g < ncu && g <= dec_total; ++g) {
                const double bw = std::min(kCuStreamGBs, kChipStreamGBs / g);  // GB/s per CU
                const double t_dec = (double)ceil_div_ll(dec_total, g) * (KT * mla::kRowBytes) / (bw * 1e3);
                const double t_chunk = chunk_us / (double)(ncu - g);
                const double t = std::max(t_dec, t_chunk);
                if (t < best) {
                    best = t;
                    best_g = g;
                }
            }
        }
        long long S = ceil_div_ll(dec_total, best_g);
        while (S > 1 && !dec_share_fits(dec, dec_total, S, (int)P)) S = std::max(1LL, S * 3 / 4);
        if (!dec_share_fits(dec, dec_total, S, (int)P))
            return fail(MLA_ERR_UNSUPPORTED, "decode work does not fit the per-workgroup segment / page limits");
        const long long G = ceil_div_ll(dec_total, S);
        if (G > (1LL << 24)) return fail(MLA_ERR_INVALID_ARG, "too many decode workgroups");
        pl->n_dec_wg = (int)G;
        pl->dec_tiles_per_wg = (int)S;
        pl->dec_total_tiles = (int)dec_total;
        for (const DecReq &d : dec)
            if (d.first_tile / S != (d.first_tile + d.tiles - 1) / S) pl->dec_split = true;
    }
    size_t off = 0;
    if (pl->chunk_split) {
        pl->off_chunk_o = off;
        off = align256(off + (size_t)nci * BM * mla::kPartialFloats * sizeof(float));
        pl->off_chunk_ml = off;
        off = align256(off + (size_t)nci * BM * mla::kPartialStats * sizeof(float));
    }
    if (pl->dec_split) {
        pl->off_dec_o = off;
        off = align256(off + (size_t)2 * pl->n_dec_wg * mla::kPartialFloats * sizeof(float));
        pl->off_dec_ml = off;
        off = align256(off + (size_t)2 * pl->n_dec_wg * mla::kPartialStats * sizeof(float));
    }
    pl->bytes = off;
    return MLA_OK;
}

}  // namespace

extern "C" {

int mla_abi_version(void) { return MLA_ABI_VERSION; }

const char *mla_last_error(void) { return g_err; }

size_t mixed_step_workspace_bytes(const mla_batch *batch) {
    Shape sh;
    if (check_batch(batch, &sh) != MLA_OK) return 0;
    Plan pl;
    if (make_plan(batch, sh, &pl) != MLA_OK) return 0;
    return pl.bytes;
}

int append_latent_kv(const mla_batch *batch, const uint16_t *new_latents, uint16_t *kv_cache, void *stream) {
    Shape sh;
    int st = check_batch(batch, &sh);
    if (st != MLA_OK || sh.R == 0) return st;
    if (!new_latents || !kv_cache) return fail(MLA_ERR_INVALID_ARG, "new_latents / kv_cache is NULL");
    if ((reinterpret_cast<uintptr_t>(new_latents) | reinterpret_cast<uintptr_t>(kv_cache)) & 15)
        return fail(MLA_ERR_INVALID_ARG, "new_latents / kv_cache must be 16-byte aligned");
    mla::AppendArgs a;
    a.src = new_latents;
    a.kv = kv_cache;
    a.cu_q = batch->cu_q_dev;
    a.prefix = batch->prefix_lens_dev;
    a.bt = batch->block_table_dev;
    a.num_reqs = sh.R;
    a.num_rows = sh.T;
    a.page_size = batch->page_size;
    a.log2_page = sh.log2_page;
    a.max_pages = batch->max_pages_per_req;
    a.num_pages = batch->num_pages;
    hipError_t e = mla::launch_append(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "append kernel launch");
    return MLA_OK;
}

}  // extern "C"

namespace {

// Shared by mixed_step_attn (new_latents == NULL) and mixed_step (fused append).
int attend(const mla_batch *batch, const uint16_t *q, const uint16_t *new_latents, uint16_t *kv_cache,
           float softmax_scale, void *out, int32_t out_dtype, float *lse, void *workspace, size_t workspace_bytes,
           void *stream) {
    Shape sh;
    int st = check_batch(batch, &sh);
    if (st != MLA_OK || sh.R == 0) return st;
    if (!q || !kv_cache || !out) return fail(MLA_ERR_INVALID_ARG, "q / kv_cache / out is NULL");
    if (reinterpret_cast<uintptr_t>(new_latents) & 15)
        return fail(MLA_ERR_INVALID_ARG, "new_latents must be 16-byte aligned");
    if (out_dtype != MLA_OUT_F32 && out_dtype != MLA_OUT_BF16)
        return fail(MLA_ERR_INVALID_ARG, "out_dtype = %d is neither MLA_OUT_F32 nor MLA_OUT_BF16", out_dtype);
    if (!std::isfinite(softmax_scale) || softmax_scale <= 0.f)
        return fail(MLA_ERR_INVALID_ARG, "softmax_scale must be finite and > 0");
    if ((reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(kv_cache) | reinterpret_cast<uintptr_t>(out) |
         reinterpret_cast<uintptr_t>(workspace)) & 15)
        return fail(MLA_ERR_INVALID_ARG, "q / kv_cache / out / workspace must be 16-byte aligned");
    if (reinterpret_cast<uintptr_t>(lse) & 3) return fail(MLA_ERR_INVALID_ARG, "lse must be 4-byte aligned");
    Plan pl;
    st = make_plan(batch, sh, &pl);
    if (st != MLA_OK) return st;
    if (pl.bytes > 0 && (!workspace || workspace_bytes < pl.bytes))
        return fail(MLA_ERR_WORKSPACE, "workspace of %zu bytes at %p; this batch needs %zu", workspace_bytes,
                    workspace, pl.bytes);
    mla::AttnArgs a;
    a.q = q;
    a.kv = kv_cache;
    a.new_kv = new_latents;
    a.kv_out = new_latents ? kv_cache : nullptr;
    a.cu_q = batch->cu_q_dev;
    a.prefix = batch->prefix_lens_dev;
    a.bt = batch->block_table_dev;
    a.out = out;
    a.lse = lse;
    char *ws = static_cast<char *>(workspace);
    a.ws_chunk_o = pl.chunk_split ? reinterpret_cast<float *>(ws + pl.off_chunk_o) : nullptr;
    a.ws_chunk_ml = pl.chunk_split ? reinterpret_cast<float *>(ws + pl.off_chunk_ml) : nullptr;
    a.ws_dec_o = pl.dec_split ? reinterpret_cast<float *>(ws + pl.off_dec_o) : nullptr;
    a.ws_dec_ml = pl.dec_split ? reinterpret_cast<float *>(ws + pl.off_dec_ml) : nullptr;
    a.num_reqs = sh.R;
    a.num_rows = sh.T;
    a.page_size = batch->page_size;
    a.log2_page = sh.log2_page;
    a.max_pages = batch->max_pages_per_req;
    a.num_pages = batch->num_pages;
    a.scale_log2 = (float)((double)softmax_scale * 1.4426950408889634);
    a.ks_chunk = pl.ks_chunk;
    a.n_chunk_items = pl.n_chunk_items;
    a.n_dec_wg = pl.n_dec_wg;
    a.dec_tiles_per_wg = pl.dec_tiles_per_wg;
    a.dec_total_tiles = pl.dec_total_tiles;
    a.out_bf16 = out_dtype == MLA_OUT_BF16 ? 1 : 0;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = mla::launch_attention(a, s);
    if (e != hipSuccess) return hip_fail(e, "attention kernel launch");
    if (pl.chunk_split || pl.dec_split) {
        e = mla::launch_combine(a, s);
        if (e != hipSuccess) return hip_fail(e, "merge kernel launch");
    }
    return MLA_OK;
}

}  // namespace

extern "C" {

int mixed_step_attn(const mla_batch *batch, const uint16_t *q, const uint16_t *kv_cache, float softmax_scale,
                    void *out, int32_t out_dtype, float *lse, void *workspace, size_t workspace_bytes,
                    void *stream) {
    return attend(batch, q, nullptr, const_cast<uint16_t *>(kv_cache), softmax_scale, out, out_dtype, lse, workspace,
                  workspace_bytes, stream);
}

int mixed_step(const mla_batch *batch, const uint16_t *q, const uint16_t *new_latents, uint16_t *kv_cache,
               float softmax_scale, void *out, int32_t out_dtype, float *lse, void *workspace,
               size_t workspace_bytes, void *stream) {
    if (batch && batch->num_reqs > 0 && !new_latents) {
        g_err[0] = '\0';
        return fail(MLA_ERR_INVALID_ARG, "new_latents is NULL");
    }
    return attend(batch, q, new_latents, kv_cache, softmax_scale, out, out_dtype, lse, workspace, workspace_bytes,
                  stream);
}

}  // extern "C"
