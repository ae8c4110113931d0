"""Projections and the whole attention layer: HIP path vs the fp64 oracle
(oracle/proj_oracle.py), through the C ABI (needs an MI355X).

Tolerances.  The GPU accumulates in fp32 and rounds to bf16 at the same
points as the oracle's rounded mode, which rounds the exact value once.  Each
GPU result is checked against the exact value (float64, no intermediate
rounding) with an elementwise bound built from what the path may do:
  * a value rounded to bf16 moves by at most one ulp of itself (half an ulp,
    doubled for the case where fp32 error pushes it across a binade);
  * a GEMM over an input that was itself rounded to bf16 moves by at most
    sum_k ulp(x_k) |w_k| (every input off by its full rounding step);
  * fp32 accumulation over K <= 2048 terms moves by at most 2^-16 sum_k |x_k w_k|.
On top of the bound, at most 1 % of stored bf16 values may differ from the
oracle's (a flip needs the exact value within fp32 error of a rounding
boundary), and fp32 results keep a mean relative error <= 2^-10 against the
oracle's rounded mode.  The whole layer keeps the attention output's bars
(max-abs 1e-2 at unit scale, mean relative error 2e-3).
Layers whose chunks take the multi-head path (up-projected fp16 keys and
values) are checked against the oracle's multi-head rounded mode, which rounds
at that path's own storage points, at the same bars (max-abs 1e-2 at unit
scale, mean relative error 2e-3).  A second, looser guard compares them with
the exact layer: within 1.5 times the absorbed rounded mode's own distance
from it, a sanity bound only (the two forms round at different points, so
neither error bounds the other).
Every instantiated GEMM tile shape is exercised through the tuning knobs
(mla_layer_tune).
"""
import numpy as np
import pytest

import oracle
from harness import from_dev_u16, log, sample_rows, to_dev
from oracle import proj_oracle as PO
import paper_2607_02043_amd as mla
from paper_2607_02043_amd import workloads as W

pytestmark = pytest.mark.gpu

SCALE = W.SOFTMAX_SCALE


@pytest.fixture(scope="module")
def weights():
    wb = W.make_proj_weights(seed=11)
    return wb, PO.Weights.from_bits(wb), mla.DeviceProjWeights(wb)


# GEMM tile shapes (rows, columns, LDS stages) forced through the library's
# tuning variables; None keeps the library's own choice.
SHAPES = [None, (32, 64, 6), (64, 64, 4), (128, 64, 3), (32, 128, 4), (64, 128, 3), (128, 128, 2), (128, 128, 3),
          (32, 128, 0), (64, 128, 0), (128, 128, 0), (128, 256, 0), (256, 128, 0)]
_KNOBS = (mla.TUNE_GEMM_BM, mla.TUNE_GEMM_BN, mla.TUNE_GEMM_DEPTH)


@pytest.fixture
def gemm_shape(request):
    settings = {k: -1 for k in _KNOBS} if request.param is None else dict(zip(_KNOBS, request.param))
    with mla.tuned(settings):
        yield request.param


@pytest.fixture
def mha_route():
    """Sets the layer's multi-head route for one test: mha_route(min_rows, pairs=-1)."""
    keys = (mla.TUNE_MHA_MIN_ROWS, mla.TUNE_MHA_PAIRS)
    for k in keys:
        mla.layer_tune(k, -1)

    def set_route(min_rows, pairs=-1):
        mla.layer_tune(mla.TUNE_MHA_MIN_ROWS, min_rows)
        mla.layer_tune(mla.TUNE_MHA_PAIRS, pairs)

    yield set_route
    for k in keys:
        mla.layer_tune(k, -1)


def _ulp_bf16(x):
    a = np.maximum(np.abs(x), 2.0 ** -126)
    return np.ldexp(1.0, np.frexp(a)[1] - 8)


def _gemm_bound(x_exact, w):
    """(sum_k ulp(x_k) |w_k|, sum_k |x_k w_k|) for y = x . w^T over the last axis."""
    aw = np.abs(w)
    return _ulp_bf16(x_exact) @ aw.T, np.abs(x_exact) @ aw.T


def check_bf16(gpu_bits, ref_bits, exact, what, upstream=None, mags=None):
    """gpu_bits: stored bf16 results; exact: their float64 values with no
    intermediate rounding; upstream / mags: _gemm_bound terms when the value is
    a GEMM over rounded inputs (or over fp32-accumulated inputs)."""
    g = PO.bf16_value(gpu_bits)
    assert np.isfinite(g).all(), f"{what}: non-finite"
    tol = _ulp_bf16(exact)
    if upstream is not None:
        tol = tol + upstream
    if mags is not None:
        tol = tol + 2.0 ** -16 * mags
    else:
        tol = tol + 2.0 ** -16 * np.abs(exact)
    d = np.abs(g - exact)
    frac = float(np.mean(gpu_bits != ref_bits))
    log(f"  {what}: max |d|/tol = {float((d / tol).max()):.3f}, bits differing from the oracle {100 * frac:.3f} %")
    assert (d <= tol).all(), f"{what}: {int((d > tol).sum())} elements beyond the bound"
    assert frac <= 0.01, f"{what}: {100 * frac:.2f} % of bf16 values differ from the oracle"


def check_f32(gpu, ref, what, max_abs=None, mean_rel=2.0 ** -10):
    assert np.isfinite(gpu).all(), f"{what}: non-finite"
    rms = float(np.sqrt(np.mean(ref ** 2)))
    d = np.abs(gpu - ref)
    ma = float(d.max()) if d.size else 0.0
    mr = float(d.sum() / max(np.abs(ref).sum(), 1e-300))
    log(f"  {what}: max_abs={ma:.3e} (limit {max_abs}) mean_rel={mr:.3e} rms={rms:.3f}")
    if max_abs is not None:
        assert ma <= max_abs, f"{what}: max_abs {ma} > {max_abs}"
    assert mr <= mean_rel, f"{what}: mean_rel {mr} > {mean_rel}"


def check_vs_exact(got, exact, rounded, what):
    """A layer output against the exact (fp64, unrounded) layer.  The ABI
    stores queries, latents and the attention output in bf16, which leaves an
    error floor that the oracle's own rounded mode measures; a path that
    rounds at other points must stay within 1.5 times that floor (and within
    the attention bars where the floor is lower)."""
    assert np.isfinite(got).all(), f"{what}: non-finite"
    scale = max(1.0, float(np.sqrt(np.mean(exact ** 2))))
    den = max(np.abs(exact).sum(), 1e-300)
    floor_rel = float(np.abs(rounded - exact).sum() / den)
    floor_abs = float(np.abs(rounded - exact).max())
    mr = float(np.abs(got - exact).sum() / den)
    ma = float(np.abs(got - exact).max())
    lim_rel, lim_abs = max(2e-3, 1.5 * floor_rel), max(1e-2 * scale, 1.5 * floor_abs)
    log(f"  {what} vs exact: mean_rel={mr:.3e} (rounding floor {floor_rel:.3e}, limit {lim_rel:.3e}) "
        f"max_abs={ma:.3e} (floor {floor_abs:.3e}, limit {lim_abs:.3e})")
    assert mr <= lim_rel, f"{what}: mean_rel {mr} > {lim_rel}"
    assert ma <= lim_abs, f"{what}: max_abs {ma} > {lim_abs}"


def _run_pre(batch, hidden_bits, dw):
    import torch
    db = mla.DeviceBatch.from_batch(batch)
    T = batch.num_rows
    q = torch.full((T, 16, 576), -1, dtype=torch.int16, device="cuda")
    lat = torch.full((T, 576), -1, dtype=torch.int16, device="cuda")
    ws = torch.empty(mla.mla_proj_workspace_bytes(T), dtype=torch.uint8, device="cuda")
    mla.mla_pre_attn(db, to_dev(hidden_bits), dw, q, lat, ws)
    torch.cuda.synchronize()
    return from_dev_u16(q), from_dev_u16(lat)


PRE_CASES = {
    "tiny": ([37, 0, 5], [1, 9, 3], 16),
    "ragged_multi_tile": (list(np.random.default_rng(3).integers(0, 20000, 200)) + [3000], [1] * 200 + [137], 64),
    "one_row": ([32767], [1], 64),
}


@pytest.mark.parametrize("gemm_shape", SHAPES, indirect=True)
@pytest.mark.parametrize("case", sorted(PRE_CASES))
def test_pre_attn_parity(case, gemm_shape, weights):
    wb, wo, dw = weights
    prefix, qlen, page = PRE_CASES[case]
    wl = W.custom(prefix, qlen, page_size=page, seed=21)
    b = wl.batch
    log(f"[gpu] pre_attn {case}: T={b.num_rows} tile={gemm_shape}")
    hidden = W.random_hidden(b.num_rows, seed=21)
    q_gpu, lat_gpu = _run_pre(b, hidden, dw)
    pos = PO.positions(b.q_lens, b.prefix_lens)
    q_ref, lat_ref = PO.pre_attn(pos, PO.bf16_value(hidden), wo, rounded=True)
    q_exact, lat_exact = PO.pre_attn(pos, PO.bf16_value(hidden), wo, rounded=False)
    q_nope = (PO.bf16_value(hidden) @ wo.w_q.T).reshape(-1, 16, 192)[:, :, :128]
    up = np.stack([_gemm_bound(q_nope[:, h], wo.w_uk_t[h])[0] for h in range(16)], axis=1)
    mags = np.stack([_gemm_bound(q_nope[:, h], wo.w_uk_t[h])[1] for h in range(16)], axis=1)
    check_bf16(q_gpu[:, :, :512], q_ref[:, :, :512], q_exact[:, :, :512], "q_abs latent part", up, mags)
    # fp32 accumulation sizes of the rope parts (a rotation mixes the two dims of a pair)
    x = PO.bf16_value(hidden)
    m_q = (np.abs(x) @ np.abs(wo.w_q).T).reshape(-1, 16, 192)[:, :, 128:]
    m_kv = np.abs(x) @ np.abs(wo.w_dkv).T
    check_bf16(q_gpu[:, :, 512:], q_ref[:, :, 512:], q_exact[:, :, 512:], "q_abs rope part",
               mags=np.repeat(m_q[..., 0::2] + m_q[..., 1::2], 2, axis=-1))
    kv = x @ wo.w_dkv.T
    inv = 1.0 / np.sqrt(np.mean(kv[:, :512] ** 2, axis=1, keepdims=True) + wo.eps)
    m_lat = np.concatenate([m_kv[:, :512] * inv * np.abs(wo.kv_gain) + np.abs(lat_exact[:, :512]),
                            np.repeat(m_kv[:, 512::2] + m_kv[:, 513::2], 2, axis=-1)], axis=1)
    check_bf16(lat_gpu, lat_ref, lat_exact, "new latents", mags=m_lat)


@pytest.mark.parametrize("gemm_shape", [None, (32, 64, 6), (64, 128, 3), (128, 128, 2), (32, 128, 0), (128, 256, 0)],
                         indirect=True)
@pytest.mark.parametrize("attn_bf16,out_bf16", [(False, False), (True, False), (False, True)])
def test_post_attn_parity(attn_bf16, out_bf16, gemm_shape, weights):
    import torch
    wb, wo, dw = weights
    T = 301
    log(f"[gpu] post_attn T={T} attn_bf16={attn_bf16} out_bf16={out_bf16} tile={gemm_shape}")
    a = W.random_attn_out(T, seed=31)
    a_dev = torch.from_numpy(a).cuda()
    if attn_bf16:
        a_dev = a_dev.to(torch.bfloat16)
        a = a_dev.float().cpu().numpy()  # the bf16 values the GPU reads (torch rounds to nearest even)
    out = torch.full((T, 2048), float("nan"), dtype=torch.bfloat16 if out_bf16 else torch.float32, device="cuda")
    ws = torch.empty(mla.mla_proj_workspace_bytes(T), dtype=torch.uint8, device="cuda")
    mla.mla_post_attn(a_dev, dw, out, ws)
    torch.cuda.synchronize()
    ref = PO.post_attn(a.astype(np.float64), wo, rounded=True, out_bf16=out_bf16)
    got = out.float().cpu().numpy().astype(np.float64)
    # exact from the bf16-rounded attention output (both sides round it identically)
    ab = PO.through_bf16(a.astype(np.float64))
    o_exact = np.concatenate([ab[:, h] @ wo.w_uv[h].T for h in range(16)], axis=1)
    up, mags = _gemm_bound(o_exact, wo.w_o)
    exact = o_exact @ wo.w_o.T
    tol = up + 2.0 ** -16 * mags + (_ulp_bf16(exact) if out_bf16 else 0.0)
    d = np.abs(got - exact)
    log(f"  out: max |d|/tol = {float((d / tol).max()):.3f}")
    assert np.isfinite(got).all() and (d <= tol).all()
    check_f32(got, ref, "out vs rounded oracle", mean_rel=2.0 ** -10 if not out_bf16 else 2.0 ** -8)


def _route_fn(route):
    """The multi-head route (min_rows, pairs) as the oracle's predicate (None: every row absorbed)."""
    if route is None:
        return None
    m, k = route
    k = max(k, 0)
    return lambda p, c: c >= m and c * (2 * p + c) >= 2 * k * (p + c)


def _layer_case(prefix, qlen, page, seed, weights, rows=None, out_bf16=False, exact=False, route=None):
    """One mla_attention_layer call against the oracle's rounded mode (the
    multi-head rounded mode for the requests `route` sends there).  Returns
    (got, ref, pool after (GPU), pool after (oracle), batch[, exact layer][,
    the step's latents from mla_pre_attn on the GPU])."""
    import torch
    wb, wo, dw = weights
    wl = W.custom(prefix, qlen, page_size=page, seed=seed)
    b = wl.batch
    li = wl.layer(0)
    hidden = W.random_hidden(b.num_rows, seed=seed)
    db = mla.DeviceBatch.from_batch(b)
    pool = to_dev(li.pool)
    out = torch.full((b.num_rows, 2048), float("nan"), dtype=torch.bfloat16 if out_bf16 else torch.float32,
                     device="cuda")
    ws = mla.layer_workspace_for(db)
    mla.mla_attention_layer(db, to_dev(hidden), dw, pool, SCALE, out, ws)
    torch.cuda.synchronize()
    ref, pool_ref, _, _ = PO.layer(b, hidden, wo, li.pool, SCALE, out_bf16=out_bf16, rows=rows)
    if route is not None:
        ref = PO.layer_multihead(b, hidden, wo, li.pool, SCALE, _route_fn(route), rows=rows)
    got = out.float().cpu().numpy().astype(np.float64)
    if rows is not None:
        got = got[np.asarray(rows)]
    res = [got, ref, from_dev_u16(pool), pool_ref, b]
    if exact:
        res.append(PO.layer_exact(b.q_lens, b.prefix_lens, PO.bf16_value(hidden), wo, PO.logical_cache(b, li.pool),
                                  SCALE, rows=rows))
    if route is not None:
        _, lat_gpu = _run_pre(b, hidden, dw)
        res.append(lat_gpu)
    return tuple(res)


def _written(b, shape):
    w = np.zeros(shape, dtype=bool)
    for r in range(b.num_reqs):
        for t in range(int(b.prefix_lens[r]), int(b.prefix_lens[r] + b.q_lens[r])):
            w[b.block_table[r][t // b.page_size], t % b.page_size] = True
    return w


def _check_pool_bits(b, pool_gpu, pool_before, lat_gpu):
    """The step writes exactly its own slots, each with the latent that
    mla_pre_attn computes for that row (bit for bit); every other slot keeps
    its bits."""
    written = _written(b, pool_gpu.shape[:2])
    assert np.array_equal(pool_gpu[~written], pool_before[~written]), "a slot outside the step changed"
    row = 0
    for r in range(b.num_reqs):
        for i in range(int(b.q_lens[r])):
            t = int(b.prefix_lens[r]) + i
            slot = pool_gpu[b.block_table[r][t // b.page_size], t % b.page_size]
            assert np.array_equal(slot, lat_gpu[row + i]), f"request {r} slot {t}: not the step's latent"
        row += int(b.q_lens[r])


LAYER_CASES = {
    "tiny_page16": ([37, 0, 5, 200], [1, 9, 3, 1], 16),
    "decode_and_chunk": ([100, 700, 2500, 64, 0], [1, 1, 1, 1, 150], 64),
    "chunk_after_prefix": ([1000, 9], [77, 1], 64),
}


@pytest.mark.parametrize("case", sorted(LAYER_CASES))
def test_layer_parity(case, weights):
    prefix, qlen, page = LAYER_CASES[case]
    log(f"[gpu] attention layer {case}: prefix={prefix} q_lens={qlen} page={page}")
    got, ref, pool_gpu, pool_ref, b = _layer_case(prefix, qlen, page, 41, weights)
    check_f32(got, ref, "layer out", max_abs=1e-2 * max(1.0, float(np.sqrt(np.mean(ref ** 2)))), mean_rel=2e-3)
    # slots the step did not write are untouched; written slots hold the step's latents to one bf16 step
    written = _written(b, pool_ref.shape[:2])
    assert np.array_equal(pool_gpu[~written], pool_ref[~written])
    gw, rw = PO.bf16_value(pool_gpu[written]), PO.bf16_value(pool_ref[written])
    assert (np.abs(gw - rw) <= 2 * _ulp_bf16(rw) + 1e-3).all()


def test_layer_bf16_out(weights):
    got, ref, *_ = _layer_case([300, 0], [1, 40], 64, 43, weights, out_bf16=True)
    check_f32(got, ref, "layer out bf16", mean_rel=3e-3)
    # the fp32 bar plus one bf16 step of the stored result
    lim = 1e-2 * max(1.0, float(np.sqrt(np.mean(ref ** 2)))) + _ulp_bf16(ref)
    assert (np.abs(got - ref) <= lim).all()


@pytest.mark.parametrize("route", ["default", "multi_head"])
def test_layer_full_size_sampled_rows(route, weights, mha_route):
    """128 decode rows with lognormal contexts plus a 2048-token chunk over a
    6144-token prefix (T = 2176), the chunk on the absorbed kernel (default)
    or the multi-head path: sampled rows against the rounded oracle."""
    r = None
    if route == "multi_head":
        r = (256, 0)
        mha_route(256)
    wl = W.config(3)
    b = wl.batch
    rows = sample_rows(b, n_decode=24, seed=3)
    log(f"[gpu] attention layer at full size ({route}): T={b.num_rows}, {len(rows)} sampled rows")
    res = _layer_case(list(b.prefix_lens), list(b.q_lens), b.page_size, wl.seed, weights, rows=rows, exact=True,
                      route=r)
    got, ref, ex = res[0], res[1], res[5]
    if r is None:
        check_f32(got, ref, "layer out (sampled)", max_abs=1e-2 * max(1.0, float(np.sqrt(np.mean(ref ** 2)))),
                  mean_rel=2e-3)
    else:
        _check_mha(got, ref, ex, "layer out (sampled)")


# Chunk requests of many rows can take the multi-head path in the layer (keys
# and values up-projected per head, fp16; opt-in through the layer's tuning
# knobs).  The oracle is the same layer in its multi-head rounded mode (fp16
# keys and values, bf16 query parts and per-head output at the GPU path's
# storage points), at the attention bars; the exact layer is a second guard.
MHA_CASES = {
    "chunk_only_prefix0": ([0], [150], 64),
    "decode_chunk_decode_page16": ([300, 40, 1000], [1, 97, 1], 16),
    "two_chunks": ([0, 70, 5], [64, 130, 1], 64),
    "ragged_page1": ([9, 0, 17], [33, 1, 2], 1),
    "long_prefix_short_chunk": ([4000], [9], 64),
}


def _check_mha(got, ref, ex, what):
    check_f32(got, ref, what + " vs multi-head rounded oracle",
              max_abs=1e-2 * max(1.0, float(np.sqrt(np.mean(ref ** 2)))), mean_rel=2e-3)
    check_vs_exact(got, ex, ref, what)


@pytest.mark.parametrize("case", sorted(MHA_CASES))
def test_layer_multihead_path_parity(case, weights, mha_route):
    mha_route(2)
    prefix, qlen, page = MHA_CASES[case]
    log(f"[gpu] attention layer, multi-head chunks {case}: prefix={prefix} q_lens={qlen} page={page}")
    wl = W.custom(prefix, qlen, page_size=page, seed=47)
    got, ref, pool_gpu, pool_ref, b, ex, lat = _layer_case(prefix, qlen, page, 47, weights, exact=True, route=(2, 0))
    _check_mha(got, ref, ex, "layer out")
    _check_pool_bits(b, pool_gpu, wl.layer(0).pool, lat)


def test_layer_multihead_pairs_route(weights, mha_route):
    """With a pairs-per-key bar, a 1536-row chunk over a 4096-token prefix
    takes the multi-head path and the decode rows around it do not.  Sampled
    rows."""
    mha_route(256, 950)
    prefix, qlen = [50, 4096, 3000], [1, 1536, 1]
    wl = W.custom(prefix, qlen, page_size=64, seed=49)
    rows = sample_rows(wl.batch, n_decode=2, seed=49)
    got, ref, pool_gpu, pool_ref, b, ex, lat = _layer_case(prefix, qlen, 64, 49, weights, rows=rows, exact=True,
                                                           route=(256, 950))
    _check_mha(got, ref, ex, "layer out (sampled)")
    _check_pool_bits(b, pool_gpu, wl.layer(0).pool, lat)


def test_layer_default_route_is_absorbed(weights):
    """By default every row runs on the absorbed kernel: the same long chunk
    matches the absorbed rounded oracle at the attention bars."""
    prefix, qlen = [50, 4096, 3000], [1, 1536, 1]
    wl = W.custom(prefix, qlen, page_size=64, seed=49)
    rows = sample_rows(wl.batch, n_decode=2, seed=49)
    got, ref, *_ = _layer_case(prefix, qlen, 64, 49, weights, rows=rows)
    check_f32(got, ref, "layer out (sampled)", max_abs=1e-2 * max(1.0, float(np.sqrt(np.mean(ref ** 2)))),
              mean_rel=2e-3)


def test_layer_mixed_routing(weights, mha_route):
    """One chunk request on each path in the same step: with 100 pairs per key
    required, the 120-row chunk over 2000 keys goes multi-head and the 150-row
    chunk at prefix 0 stays on the absorbed kernel."""
    mha_route(2, 100)
    wl = W.custom([2000, 7, 0], [120, 1, 150], page_size=64, seed=51)
    got, ref, pool_gpu, pool_ref, b, ex, lat = _layer_case([2000, 7, 0], [120, 1, 150], 64, 51, weights, exact=True,
                                                           route=(2, 100))
    _check_mha(got, ref, ex, "layer out")
    _check_pool_bits(b, pool_gpu, wl.layer(0).pool, lat)


@pytest.mark.parametrize("route", ["default", "multi_head"])
def test_layer_four_chunks_full_size_sampled_rows(route, weights, mha_route):
    """One layer of the 27-layer workload: 64 decode rows and four 1024-token
    chunks at prefixes 0 / 1024 / 3072 / 8192 (by default every row on the
    absorbed kernel; with a 256-row minimum, all four chunks multi-head)."""
    r = None
    if route == "multi_head":
        r = (256, 0)
        mha_route(256)
    wl = W.config(5)
    b = wl.batch
    rows = sample_rows(b, n_decode=16, seed=5)
    log(f"[gpu] attention layer, four chunks at full size ({route}): T={b.num_rows}, {len(rows)} sampled rows")
    res = _layer_case(list(b.prefix_lens), list(b.q_lens), b.page_size, wl.seed, weights, rows=rows, exact=True,
                      route=r)
    got, ref, ex = res[0], res[1], res[5]
    if r is None:
        check_f32(got, ref, "layer out (sampled)", max_abs=1e-2 * max(1.0, float(np.sqrt(np.mean(ref ** 2)))),
                  mean_rel=2e-3)
    else:
        _check_mha(got, ref, ex, "layer out (sampled)")


def test_layer_multihead_bad_page_id_writes_nothing(weights, mha_route):
    """A block-table entry outside the pool in a multi-head chunk request
    (keys 128..191, all new): those new latents are written nowhere (page 0
    and every other slot keep their bits, no fault), and every other new
    latent of the step lands in its own slot.  Outputs are not checked."""
    import torch
    mha_route(2)
    wb, wo, dw = weights
    wl = W.custom([70, 100], [150, 1], page_size=64, seed=53, name="mha_bad_page")
    b = wl.batch
    li = wl.layer(0)
    b.block_table = b.block_table.copy()
    assert b.block_table.shape[1] >= 4
    b.block_table[0, 2] = b.num_pages + 3
    log(f"[gpu] attention layer, multi-head chunk with block-table entry {b.num_pages + 3} of {b.num_pages} pages")
    hidden = W.random_hidden(b.num_rows, seed=53)
    db = mla.DeviceBatch.from_batch(b)
    pool = to_dev(li.pool)
    out = torch.empty((b.num_rows, 2048), dtype=torch.float32, device="cuda")
    mla.mla_attention_layer(db, to_dev(hidden), dw, pool, SCALE, out, mla.layer_workspace_for(db))
    torch.cuda.synchronize()
    _, lat = _run_pre(b, hidden, dw)
    expect = li.pool.copy()
    cu = b.cu_q
    for r in range(b.num_reqs):
        for i in range(int(b.q_lens[r])):
            t = int(b.prefix_lens[r]) + i
            pg = int(b.block_table[r, t // b.page_size])
            if 0 <= pg < b.num_pages:
                expect[pg, t % b.page_size] = lat[cu[r] + i]
    assert np.array_equal(from_dev_u16(pool), expect)
