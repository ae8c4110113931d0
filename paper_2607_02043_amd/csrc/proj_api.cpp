// C ABI of the projections around the mixed-step attention and of the whole
// attention layer: argument checks, workspace layout and launches.  The entry
// points and their contracts are declared in include/mla_layer.h.
#include "mla_layer.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>

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

int env_int(const char *name) {
    const char *e = std::getenv(name);
    return e ? std::atoi(e) : 0;
}

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
    if (int v = env_int("MLA_GEMM_BM")) t.bm = v;
    if (!a_f32)
        if (int v = env_int("MLA_GEMM_BN")) t.bn = v;
    if (const char *e = std::getenv("MLA_GEMM_D")) t.depth = std::atoi(e);
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

    GemmArgs v{};
    v.a = attn_out;
    v.lda = (long long)kHeads * kLatent;
    v.a_bstride = kLatent;
    v.b = w->w_uv;
    v.b2 = w->w_uv;
    v.ldb = kLatent;
    v.b_bstride = (long long)kVHead * kLatent;
    v.n_split = kVHead;
    v.M = T;
    v.N = kVHead;
    v.K = kLatent;
    v.c = o;
    v.ldc = kOCols;
    v.c_bstride = kVHead;
    st = launch(v, kStoreBf16, attn_dtype == MLA_OUT_F32, kHeads, s, "value up-projection");
    if (st != MLA_OK) return st;

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

// Layer workspace: the attention's (counters first) at offset 0, then the
// absorbed queries, the new latents, the attention output (bf16: the value
// up-projection reads it as bf16 in any case) and the projection workspace.
struct LayerLayout {
    size_t attn = 0, q = 0, lat = 0, o = 0, proj = 0, total = 0;
};

LayerLayout layer_layout(size_t attn_bytes, long long T) {
    LayerLayout l;
    l.attn = attn_bytes;
    size_t off = a256(attn_bytes);
    l.q = off;
    off = a256(off + (size_t)T * proj::kHeads * proj::kDqk * 2);
    l.lat = off;
    off = a256(off + (size_t)T * proj::kDqk * 2);
    l.o = off;
    off = a256(off + (size_t)T * proj::kHeads * proj::kLatent * 2);
    l.proj = off;
    l.total = off + proj_layout(T).total;
    return l;
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

size_t mla_layer_workspace_bytes(const mla_batch *batch) {
    int T = 0;
    if (mla::batch_rows(batch, &T) != MLA_OK || T == 0) return 0;
    size_t attn = 0;
    if (mla::attn_workspace(batch, &attn) != MLA_OK) return 0;
    return layer_layout(attn, T).total;
}

int mla_attention_layer(const mla_batch *batch, const uint16_t *hidden, const mla_proj_weights *w,
                        uint16_t *kv_cache, float softmax_scale, void *out, int32_t out_dtype, void *workspace,
                        size_t workspace_bytes, void *stream) {
    int T = 0;
    int st = mla::batch_rows(batch, &T);
    if (st != MLA_OK || T == 0) return st;
    size_t attn = 0;
    st = mla::attn_workspace(batch, &attn);
    if (st != MLA_OK) return st;
    const LayerLayout L = layer_layout(attn, T);
    if (!workspace || misaligned(workspace) || workspace_bytes < L.total)
        return mla::set_error(MLA_ERR_WORKSPACE, "workspace of %zu bytes at %p; this batch needs %zu",
                              workspace_bytes, workspace, L.total);
    char *ws = static_cast<char *>(workspace);
    uint16_t *q = reinterpret_cast<uint16_t *>(ws + L.q);
    uint16_t *lat = reinterpret_cast<uint16_t *>(ws + L.lat);
    uint16_t *o = reinterpret_cast<uint16_t *>(ws + L.o);
    const hipStream_t s = static_cast<hipStream_t>(stream);
    st = pre_attn(batch, T, hidden, w, q, lat, ws + L.proj, L.total - L.proj, s);
    if (st != MLA_OK) return st;
    st = mixed_step(batch, q, lat, kv_cache, softmax_scale, o, MLA_OUT_BF16, nullptr, attn > 0 ? ws : nullptr,
                    attn, stream);
    if (st != MLA_OK) return st;
    return post_attn(T, o, MLA_OUT_BF16, w, out, out_dtype, ws + L.proj, L.total - L.proj, s);
}

}  // extern "C"
