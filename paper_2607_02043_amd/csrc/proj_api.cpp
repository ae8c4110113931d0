// C ABI of the projections around the mixed-step attention and of the whole
// attention layer: argument checks, workspace layout and launches.  The entry
// points and their contracts are declared in include/mla_layer.h.
#include "mla_layer.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <atomic>

#include "api_util.h"
#include "proj_kernels.h"

namespace {

using proj::GemmArgs;

size_t a256(size_t v) { return (v + 255) & ~size_t(255); }

// Projection workspace: before attention qn bf16 [T][16][128], qpe fp32
// [T][16][64] and kvf fp32 [T][576]; after attention o bf16 [T][2048] at the
// start (the two phases never overlap in time).
struct ProjLayout {
    size_t qn = 0, qpe = 0, kvf = 0, o = 0, total = 0;
};

ProjLayout proj_layout(long long T) {
    ProjLayout l;
    size_t off = 0;
    l.qn = off;
    off = a256(off + (size_t)T * proj::kHeads * proj::kNope * 2);
    l.qpe = off;
    off = a256(off + (size_t)T * proj::kHeads * proj::kRope * 4);
    l.kvf = off;
    off = a256(off + (size_t)T * proj::kDqk * 4);
    l.o = 0;
    l.total = std::max(off, a256((size_t)T * proj::kOCols * 2));
    return l;
}

// Tuning overrides (mla_layer_tune), process-wide.  Their first values come
// from the environment, read once: MLA_GEMM_BM / MLA_GEMM_BN / MLA_GEMM_D and
// MLA_LAYER_MHA_MIN / MLA_LAYER_MHA_PAIRS (see mla_layer.h).  -1 = the
// library's own choice.
struct Tuning {
    std::atomic<int> v[MLA_TUNE_COUNT];
};

int env_or(const char *name, int dflt) {
    const char *e = std::getenv(name);
    return e ? std::atoi(e) : dflt;
}

Tuning &tuning() {
    static Tuning *t = [] {
        Tuning *n = new Tuning;
        const int bm = env_or("MLA_GEMM_BM", 0), bn = env_or("MLA_GEMM_BN", 0);
        n->v[MLA_TUNE_GEMM_BM].store(bm > 0 ? bm : -1);
        n->v[MLA_TUNE_GEMM_BN].store(bn > 0 ? bn : -1);
        n->v[MLA_TUNE_GEMM_DEPTH].store(std::getenv("MLA_GEMM_D") ? std::max(0, env_or("MLA_GEMM_D", 0)) : -1);
        const int m = env_or("MLA_LAYER_MHA_MIN", 0);
        n->v[MLA_TUNE_MHA_MIN_ROWS].store(m >= 2 ? m : -1);
        n->v[MLA_TUNE_MHA_PAIRS].store(std::getenv("MLA_LAYER_MHA_PAIRS") ? std::max(0, env_or("MLA_LAYER_MHA_PAIRS", 0))
                                                                        : -1);
        return n;
    }();
    return *t;
}

int tuned(int knob) { return tuning().v[knob].load(std::memory_order_relaxed); }

int cu_count() {
    int ncu = 256, dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
        ncu = v;
    return ncu;
}

// Tile shape of a GEMM launch, from measurements of the layer's GEMMs at 256
// to 4160 rows: the largest of the LDS-ring tiles 128 x 128 (2 stages),
// 64 x 128 (3), 64 x 64 (4), 32 x 64 (6) that still gives at least 0.85
// workgroups per CU (fewer leaves CUs idle; more is a second round of
// workgroups for large tiles), and the register-staged 256 x 128 tile for the
// narrow batched value up-projection once it has 1024 rows.  fp32 activations
// use 64-column tiles.  MLA_GEMM_BM / MLA_GEMM_BN / MLA_GEMM_D override the
// choice (for tuning; a shape that is not instantiated fails the launch).
proj::GemmShape pick_shape(long long M, int N, int batch, int epi, bool a_f32) {
    struct Cand {
        int bm, bn, depth;
    };
    static const Cand ring[] = {{128, 128, 2}, {64, 128, 3}, {64, 64, 4}, {32, 64, 6}};
    proj::GemmShape t{32, 64, 6, epi};
    const long long need = (long long)cu_count() * 85 / 100;
    if (!a_f32 && N <= 128 && M >= 1024) {
        t = {256, 128, 0, epi};
    } else {
        for (const Cand &c : ring) {
            t = {c.bm, c.bn, c.depth, epi};
            if ((M + c.bm - 1) / c.bm * ((N + c.bn - 1) / c.bn) * batch >= need) break;
        }
    }
    if (a_f32) {
        t.bn = proj::kBN;
        t.bm = std::min(t.bm, 128);
    }
    if (int v = tuned(MLA_TUNE_GEMM_BM); v > 0) t.bm = v;
    if (!a_f32)
        if (int v = tuned(MLA_TUNE_GEMM_BN); v > 0) t.bn = v;
    if (int v = tuned(MLA_TUNE_GEMM_DEPTH); v >= 0) t.depth = v;
    return t;
}

bool misaligned(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) != 0; }

int check_weights(const mla_proj_weights *w, bool pre) {
    if (!w) return mla::set_error(MLA_ERR_INVALID_ARG, "weights is NULL");
    const void *ptrs[3] = {pre ? w->w_q : w->w_uv, pre ? w->w_dkv : w->w_o, pre ? w->kv_gain : w->w_uv};
    const char *names = pre ? "w_q / w_dkv / kv_gain / w_uk_t" : "w_uv / w_o";
    for (const void *p : ptrs)
        if (!p || misaligned(p)) return mla::set_error(MLA_ERR_INVALID_ARG, "%s must be non-NULL and 16-byte aligned", names);
    if (pre) {
        if (!w->w_uk_t || misaligned(w->w_uk_t))
            return mla::set_error(MLA_ERR_INVALID_ARG, "%s must be non-NULL and 16-byte aligned", names);
        if (!std::isfinite(w->rms_eps) || w->rms_eps <= 0.f)
            return mla::set_error(MLA_ERR_INVALID_ARG, "rms_eps must be finite and > 0");
        if (!std::isfinite(w->rope_base) || w->rope_base <= 1.f)
            return mla::set_error(MLA_ERR_INVALID_ARG, "rope_base must be finite and > 1");
    }
    return MLA_OK;
}

int launch(const GemmArgs &g, int epi, bool a_f32, int batch, hipStream_t s, const char *what) {
    const proj::GemmShape t = pick_shape(g.M, g.N, batch, epi, a_f32);
    if (g.n_split < g.N && g.n_split % t.bn != 0)
        return mla::set_error(MLA_ERR_INVALID_ARG, "%s GEMM: column split %d is not a multiple of the tile width %d",
                              what, g.n_split, t.bn);
    const hipError_t e = proj::launch_gemm(g, t, a_f32, batch, s);
    if (e != hipSuccess) return mla::set_error(MLA_ERR_HIP, "%s GEMM launch: %s", what, hipGetErrorString(e));
    return MLA_OK;
}

int pre_attn(const mla_batch *batch, int T, const uint16_t *hidden, const mla_proj_weights *w, uint16_t *q_abs,
             uint16_t *new_latents, void *workspace, size_t workspace_bytes, hipStream_t s) {
    using namespace proj;
    if (T == 0) return MLA_OK;
    int st = check_weights(w, true);
    if (st != MLA_OK) return st;
    if (!hidden || !q_abs || !new_latents || misaligned(hidden) || misaligned(q_abs) || misaligned(new_latents))
        return mla::set_error(MLA_ERR_INVALID_ARG, "hidden / q_abs / new_latents must be non-NULL and 16-byte aligned");
    const ProjLayout L = proj_layout(T);
    if (!workspace || misaligned(workspace) || workspace_bytes < L.total)
        return mla::set_error(MLA_ERR_WORKSPACE, "workspace of %zu bytes at %p; %d rows need %zu", workspace_bytes,
                              workspace, T, L.total);
    char *ws = static_cast<char *>(workspace);
    uint16_t *qn = reinterpret_cast<uint16_t *>(ws + L.qn);
    float *qpe = reinterpret_cast<float *>(ws + L.qpe);
    float *kvf = reinterpret_cast<float *>(ws + L.kvf);

    GemmArgs g{};
    g.a = hidden;
    g.lda = kHidden;
    g.b = w->w_q;
    g.b2 = w->w_dkv;
    g.ldb = kHidden;
    g.n_split = kQCols;
    g.M = T;
    g.N = kQCols + kDqk;
    g.K = kHidden;
    g.qn = qn;
    g.qpe = qpe;
    g.kvf = kvf;
    st = launch(g, kQkvSplit, false, 1, s, "query / latent projection");
    if (st != MLA_OK) return st;

    RowArgs r{};
    r.qpe = qpe;
    r.kvf = kvf;
    r.gamma = w->kv_gain;
    r.cu_q = batch->cu_q_dev;
    r.prefix = batch->prefix_lens_dev;
    r.q_abs = q_abs;
    r.latent = new_latents;
    r.num_reqs = batch->num_reqs;
    r.num_rows = T;
    r.eps = w->rms_eps;
    r.log2_base = std::log2((double)w->rope_base);
    GemmArgs u{};
    // the rope / norm rows ride along as extra workgroups of the absorption launch
    u.rope = r;
    u.rope_wgs = rope_norm_wgs(T);
    u.a = qn;
    u.lda = kHeads * kNope;
    u.a_bstride = kNope;
    u.b = w->w_uk_t;
    u.b2 = w->w_uk_t;
    u.ldb = kNope;
    u.b_bstride = (long long)kLatent * kNope;
    u.n_split = kLatent;
    u.M = T;
    u.N = kLatent;
    u.K = kNope;
    u.c = q_abs;
    u.ldc = (long long)kHeads * kDqk;
    u.c_bstride = kDqk;
    return launch(u, kStoreBf16, false, kHeads, s, "query absorption");
}

// o[r] = concat_h W_UV[h] attn_out[r][h] for rows r0 .. r1 - 1 (bf16 o [T][2048]).
int uv_gemm(int r0, int r1, const void *attn_out, bool a_f32, const mla_proj_weights *w, uint16_t *o, hipStream_t s) {
    using namespace proj;
    if (r1 <= r0) return MLA_OK;
    GemmArgs v{};
    v.a = static_cast<const char *>(attn_out) + (size_t)r0 * kHeads * kLatent * (a_f32 ? 4 : 2);
    v.lda = (long long)kHeads * kLatent;
    v.a_bstride = kLatent;
    v.b = w->w_uv;
    v.b2 = w->w_uv;
    v.ldb = kLatent;
    v.b_bstride = (long long)kVHead * kLatent;
    v.n_split = kVHead;
    v.M = r1 - r0;
    v.N = kVHead;
    v.K = kLatent;
    v.c = o + (size_t)r0 * kOCols;
    v.ldc = kOCols;
    v.c_bstride = kVHead;
    return launch(v, kStoreBf16, a_f32, kHeads, s, "value up-projection");
}

// out = o W_o^T for T rows.
int o_gemm(int T, const uint16_t *o, const mla_proj_weights *w, void *out, int32_t out_dtype, hipStream_t s) {
    using namespace proj;
    GemmArgs g{};
    g.a = o;
    g.lda = kOCols;
    g.b = w->w_o;
    g.b2 = w->w_o;
    g.ldb = kOCols;
    g.n_split = kHidden;
    g.M = T;
    g.N = kHidden;
    g.K = kOCols;
    g.c = out;
    g.ldc = kHidden;
    return launch(g, out_dtype == MLA_OUT_F32 ? kStoreF32 : kStoreBf16, false, 1, s, "output projection");
}

int post_attn(int T, const void *attn_out, int32_t attn_dtype, const mla_proj_weights *w, void *out,
              int32_t out_dtype, void *workspace, size_t workspace_bytes, hipStream_t s) {
    using namespace proj;
    if (T < 0) return mla::set_error(MLA_ERR_INVALID_ARG, "num_rows = %d < 0", T);
    if (T == 0) return MLA_OK;
    int st = check_weights(w, false);
    if (st != MLA_OK) return st;
    if (attn_dtype != MLA_OUT_F32 && attn_dtype != MLA_OUT_BF16)
        return mla::set_error(MLA_ERR_INVALID_ARG, "attn_dtype = %d is neither MLA_OUT_F32 nor MLA_OUT_BF16", attn_dtype);
    if (out_dtype != MLA_OUT_F32 && out_dtype != MLA_OUT_BF16)
        return mla::set_error(MLA_ERR_INVALID_ARG, "out_dtype = %d is neither MLA_OUT_F32 nor MLA_OUT_BF16", out_dtype);
    if (!attn_out || !out || misaligned(attn_out) || misaligned(out))
        return mla::set_error(MLA_ERR_INVALID_ARG, "attn_out / out must be non-NULL and 16-byte aligned");
    const ProjLayout L = proj_layout(T);
    if (!workspace || misaligned(workspace) || workspace_bytes < L.total)
        return mla::set_error(MLA_ERR_WORKSPACE, "workspace of %zu bytes at %p; %d rows need %zu", workspace_bytes,
                              workspace, T, L.total);
    uint16_t *o = reinterpret_cast<uint16_t *>(static_cast<char *>(workspace) + L.o);
    st = uv_gemm(0, T, attn_out, attn_dtype == MLA_OUT_F32, w, o, s);
    if (st != MLA_OK) return st;
    return o_gemm(T, o, w, out, out_dtype, s);
}

// Which chunk requests take the multi-head path in the layer (up-projected
// keys and values, 192 + 128 dims per head: about 30% of the absorbed form's
// flops per query-key pair, for one up-projection of the request's keys).
// By default none do: every row runs on the absorbed kernel.  The route is
// opt-in (mla_layer_tune): a row minimum alone sends every chunk request of
// that many rows; with a pairs-per-key bar too, only requests whose query-key
// pairs per key, c (p + c / 2) / (p + c), reach it (the up-projection costs a
// fixed time per key, the multi-head form saves a fixed time per pair).
mla::ChunkRoute mha_route() {
    const int m = tuned(MLA_TUNE_MHA_MIN_ROWS), k = tuned(MLA_TUNE_MHA_PAIRS);
    mla::ChunkRoute r = mla::kAbsorbAll;
    if (m >= 2) {
        r.min_rows = m;
        r.pair_keys = k >= 0 ? k : 0;
    }
    return r;
}

// Layer workspace: the attention's (counters first) at offset 0, then the
// absorbed queries, the new latents, the attention output (bf16: the value
// up-projection reads it as bf16 in any case), the per-head values o (bf16
// [T][2048]), the up-projected keys and values of the largest multi-head
// chunk request (fp16 [p + c][4096]) and its rope keys (fp16 [p + c][64]),
// and the projection workspace.
struct LayerLayout {
    size_t attn = 0, q = 0, lat = 0, olat = 0, o = 0, kv = 0, kpe = 0, proj = 0, total = 0;
};

LayerLayout layer_layout(size_t attn_bytes, long long T, long long max_mha_keys) {
    LayerLayout l;
    l.attn = attn_bytes;
    size_t off = a256(attn_bytes);
    l.q = off;
    off = a256(off + (size_t)T * proj::kHeads * proj::kDqk * 2);
    l.lat = off;
    off = a256(off + (size_t)T * proj::kDqk * 2);
    l.olat = off;
    off = a256(off + (size_t)T * proj::kHeads * proj::kLatent * 2);
    l.o = off;
    off = a256(off + (size_t)T * proj::kOCols * 2);
    l.kv = off;
    off = a256(off + (size_t)max_mha_keys * 2 * proj::kOCols * 2);
    l.kpe = off;
    off = a256(off + (size_t)max_mha_keys * proj::kRope * 2);
    l.proj = off;
    l.total = off + proj_layout(T).total;
    return l;
}

// Sizes of a layer step: rows, the attention workspace (largest of the plans
// with and without the multi-head requests) and the keys of the largest
// multi-head request.
int layer_sizes(const mla_batch *b, mla::ChunkRoute route, int *T, size_t *attn, long long *max_keys) {
    int st = mla::batch_rows(b, T);
    if (st != MLA_OK || *T == 0) return st;
    *max_keys = 0;
    for (int r = 0; r < b->num_reqs; ++r)
        if (route.multi_head(b->prefix_lens[r], b->q_lens[r]))
            *max_keys = std::max<long long>(*max_keys, (long long)b->prefix_lens[r] + b->q_lens[r]);
    size_t a_all = 0, a_part = 0;
    st = mla::attn_workspace(b, &a_all);
    if (st == MLA_OK && *max_keys > 0) st = mla::attn_workspace(b, &a_part, route);
    *attn = std::max(a_all, a_part);
    return st;
}

}  // namespace

extern "C" {

size_t mla_proj_workspace_bytes(int32_t num_rows) { return num_rows > 0 ? proj_layout(num_rows).total : 0; }

int mla_pre_attn(const mla_batch *batch, const uint16_t *hidden, const mla_proj_weights *w, uint16_t *q_abs,
                 uint16_t *new_latents, void *workspace, size_t workspace_bytes, void *stream) {
    int T = 0;
    const int st = mla::batch_rows(batch, &T);
    if (st != MLA_OK) return st;
    return pre_attn(batch, T, hidden, w, q_abs, new_latents, workspace, workspace_bytes,
                    static_cast<hipStream_t>(stream));
}

int mla_post_attn(int32_t num_rows, const void *attn_out, int32_t attn_dtype, const mla_proj_weights *w, void *out,
                  int32_t out_dtype, void *workspace, size_t workspace_bytes, void *stream) {
    mla::set_error(MLA_OK, "");
    return post_attn(num_rows, attn_out, attn_dtype, w, out, out_dtype, workspace, workspace_bytes,
                     static_cast<hipStream_t>(stream));
}

int mla_layer_tune(int32_t knob, int32_t value) {
    mla::set_error(MLA_OK, "");
    if (knob < 0 || knob >= MLA_TUNE_COUNT) return mla::set_error(MLA_ERR_INVALID_ARG, "unknown tuning knob %d", knob);
    if (value < -1) return mla::set_error(MLA_ERR_INVALID_ARG, "tuning value %d < -1", value);
    tuning().v[knob].store(value);
    return MLA_OK;
}

size_t mla_layer_workspace_bytes(const mla_batch *batch) {
    int T = 0;
    size_t attn = 0;
    long long max_keys = 0;
    if (layer_sizes(batch, mha_route(), &T, &attn, &max_keys) != MLA_OK || T == 0) return 0;
    return layer_layout(attn, T, max_keys).total;
}

int mla_attention_layer(const mla_batch *batch, const uint16_t *hidden, const mla_proj_weights *w,
                        uint16_t *kv_cache, float softmax_scale, void *out, int32_t out_dtype, void *workspace,
                        size_t workspace_bytes, void *stream) {
    using namespace proj;
    const mla::ChunkRoute route = mha_route();
    int T = 0;
    size_t attn = 0;
    long long max_keys = 0;
    int st = layer_sizes(batch, route, &T, &attn, &max_keys);
    if (st != MLA_OK || T == 0) return st;
    if (max_keys > 0 && (!w || !w->w_uk || misaligned(w->w_uk)))
        return mla::set_error(MLA_ERR_INVALID_ARG, "w_uk must be non-NULL and 16-byte aligned");
    const LayerLayout L = layer_layout(attn, T, max_keys);
    if (!workspace || misaligned(workspace) || workspace_bytes < L.total)
        return mla::set_error(MLA_ERR_WORKSPACE, "workspace of %zu bytes at %p; this batch needs %zu",
                              workspace_bytes, workspace, L.total);
    char *ws = static_cast<char *>(workspace);
    uint16_t *q = reinterpret_cast<uint16_t *>(ws + L.q);
    uint16_t *lat = reinterpret_cast<uint16_t *>(ws + L.lat);
    uint16_t *olat = reinterpret_cast<uint16_t *>(ws + L.olat);
    uint16_t *o = reinterpret_cast<uint16_t *>(ws + L.o);
    char *pws = ws + L.proj;
    const size_t pws_bytes = L.total - L.proj;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    st = pre_attn(batch, T, hidden, w, q, lat, pws, pws_bytes, s);
    if (st != MLA_OK) return st;
    if (max_keys == 0) {
        // every row on the absorbed kernel: append and attention in one launch
        st = mixed_step(batch, q, lat, kv_cache, softmax_scale, olat, MLA_OUT_BF16, nullptr, attn > 0 ? ws : nullptr,
                        attn, stream);
        if (st != MLA_OK) return st;
        st = uv_gemm(0, T, olat, false, w, o, s);
        if (st != MLA_OK) return st;
        return o_gemm(T, o, w, out, out_dtype, s);
    }

    // Long chunk requests take the multi-head path; the other rows the
    // absorbed kernel, which also appends their new latents.  The multi-head
    // requests' latents are appended by their up-projection launch.
    st = mla::attend_rows(batch, q, lat, kv_cache, softmax_scale, olat, MLA_OUT_BF16, attn > 0 ? ws : nullptr, attn,
                          stream, route);
    if (st != MLA_OK) return st;
    // value up-projection of the absorbed rows: the span from the first to
    // the last row that is not in a multi-head request
    int lo = T, hi = 0;
    {
        int row = 0;
        for (int r = 0; r < batch->num_reqs; ++r) {
            const int c = batch->q_lens[r];
            if (!route.multi_head(batch->prefix_lens[r], c)) {
                lo = std::min(lo, row);
                hi = std::max(hi, row + c);
            }
            row += c;
        }
    }
    st = uv_gemm(lo, hi, olat, false, w, o, s);
    if (st != MLA_OK) return st;
    const uint16_t *qn = reinterpret_cast<const uint16_t *>(pws + proj_layout(T).qn);
    uint16_t *kvu = reinterpret_cast<uint16_t *>(ws + L.kv);
    uint16_t *kpe = reinterpret_cast<uint16_t *>(ws + L.kpe);
    int lg = 0;
    while ((1 << lg) < batch->page_size) ++lg;
    int row = 0;
    for (int r = 0; r < batch->num_reqs; ++r) {
        const int c = batch->q_lens[r], p = batch->prefix_lens[r];
        if (route.multi_head(p, c)) {
            // keys 0 .. p + c - 1 of the request: k = W_UK c, v = W_UV c (fp16)
            GemmArgs u{};
            u.a = kv_cache;
            u.lda = kDqk;
            u.a_bt = batch->block_table_dev + (size_t)r * batch->max_pages_per_req;
            u.a_log2p = lg;
            u.a_npages = batch->num_pages;
            u.a_new = lat + (size_t)row * kDqk;  // the chunk's own keys: its new latents
            u.a_new_from = p;
            u.keys = KeyRowsJob{kv_cache, lat + (size_t)row * kDqk, u.a_bt, lg, batch->num_pages, p, p + c, kpe};
            u.keys_wgs = (p + c + kKeyRowsPerWg - 1) / kKeyRowsPerWg;
            u.b = w->w_uk;
            u.b2 = w->w_uv;
            u.ldb = kLatent;
            u.n_split = kOCols;
            u.M = p + c;
            u.N = 2 * kOCols;
            u.K = kLatent;
            u.c = kvu;
            u.ldc = 2 * kOCols;
            st = launch(u, kStoreF16, false, 1, s, "key / value up-projection");
            if (st != MLA_OK) return st;
            MhaArgs m{};
            m.qn = qn;
            m.q_abs = q;
            m.kv = kvu;
            m.kpe = kpe;
            m.o = o;
            m.row0 = row;
            m.c = c;
            m.p = p;
            m.scale_log2 = (float)((double)softmax_scale * 1.4426950408889634);
            const hipError_t e = launch_mha_prefill(m, s);
            if (e != hipSuccess)
                return mla::set_error(MLA_ERR_HIP, "multi-head prefill launch: %s", hipGetErrorString(e));
        }
        row += c;
    }
    return o_gemm(T, o, w, out, out_dtype, s);
}

}  // extern "C"
