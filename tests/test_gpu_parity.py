"""HIP path vs the fp64 oracle, through the C ABI (needs an MI355X).

Small workloads are compared on every output row; the full-size workloads
(256-request decode batches, 2048-token chunks over a 6144-token prefix, the
27-layer step) on sampled rows that the oracle computes one by one.  Append is
compared bit for bit on the whole pool (NaN canaries included).
"""
import zlib

import numpy as np
import pytest

import oracle
from harness import GpuLayer, assert_close, log, run_layer, sample_rows
import paper_2607_02043_amd as mla
from paper_2607_02043_amd import workloads as W

pytestmark = pytest.mark.gpu

EDGE_CASES = {
    # name: (prefix_lens, q_lens, page_size)
    "decode_single_key": ([0], [1], 64),
    "decode_tile_edges": ([30, 31, 32, 63, 64, 65, 95, 127, 128, 255, 256, 257], [1] * 12, 64),
    "page16_mixed": ([15, 0, 100, 3], [1, 37, 1, 70], 16),
    "page1": ([5, 0, 40], [1, 9, 1], 1),
    "page2_ragged_chunk": ([7, 0], [13, 2], 2),
    "chunk_of_two": ([0], [2], 64),
    "chunk_unaligned_prefix": ([70, 1], [45, 3], 64),
    "chunk_long_prefix": ([5000], [37], 64),
    "page256": ([600, 0, 1000], [1, 300, 1], 256),
    "chunk_first": ([0, 9, 300], [33, 1, 1], 32),
    "page512": ([1030, 0, 511], [1, 513, 1], 512),
    "page1024": ([3000, 0, 1500, 10], [1, 200, 1, 1], 1024),
    "decode_100k_keys": ([100000, 7], [1, 1], 64),
}


def _compare_all_rows(wl, li, out_bf16=False):
    b = wl.batch
    g = run_layer(b, li, out_bf16=out_bf16)
    pool_ref, out_ref, lse_ref = oracle.step(b, li, W.SOFTMAX_SCALE)
    assert np.array_equal(g.pool_np(), pool_ref), "append: pool differs from the oracle"
    assert_close(g.out_np(), out_ref, g.lse_np(), lse_ref, what=wl.name + (" bf16" if out_bf16 else ""))


@pytest.mark.parametrize("name", sorted(EDGE_CASES))
def test_edge_cases_all_rows(name):
    prefix, qlen, page = EDGE_CASES[name]
    log(f"[gpu] edge case {name}: prefix={prefix} q_lens={qlen} page={page}")
    wl = W.custom(prefix, qlen, page_size=page, seed=zlib.crc32(name.encode()) % 1000, name=name)
    _compare_all_rows(wl, wl.layer(0))


def test_many_requests():
    rng = np.random.default_rng(5)
    prefix = list(rng.integers(0, 3000, 300)) + [100, 0]
    qlen = [1] * 300 + [64, 129]
    log("[gpu] 302 requests (300 decode + 2 chunks), page 64")
    wl = W.custom(prefix, qlen, page_size=64, seed=8, name="many_requests")
    _compare_all_rows(wl, wl.layer(0))


def _plant_spike(b, li, key_pos_req, req, token_row, scale=8.0):
    """Overwrite the latent of key `key_pos_req` of request `req` with
    scale * sign(q[token_row][head 0]): its score then exceeds every earlier
    score of that row by far more than 2^15 in log2 units."""
    q0 = W.bf16_bits_to_f32(li.q.reshape(-1, W.NUM_HEADS, W.D_QK)[token_row, 0])
    spike = W.f32_to_bf16_bits(np.where(q0 >= 0, scale, -scale).astype(np.float32))
    p, c = int(b.prefix_lens[req]), int(b.q_lens[req])
    if key_pos_req < p:  # cached: write it into the pool through the block table
        pg = int(b.block_table[req][key_pos_req // b.page_size])
        li.pool[pg, key_pos_req % b.page_size] = spike
    else:  # appended this step
        row0 = int(np.concatenate([[0], np.cumsum(b.q_lens)])[req])
        li.new_latents.reshape(-1, W.D_QK)[row0 + key_pos_req - p] = spike


def test_chunk_late_score_spike():
    """Chunk rows whose later keys outscore the first tile by more than the
    fp16 probability range take the exact-max pass."""
    wl = W.custom([100, 5, 0], [40, 1, 70], page_size=16, seed=11, name="score_spike")
    b, li = wl.batch, wl.layer(0)
    _plant_spike(b, li, 90, 0, token_row=30)   # cached key, request 0
    _plant_spike(b, li, 125, 0, token_row=35)  # appended key, request 0
    _plant_spike(b, li, 40, 2, token_row=41 + 60)  # appended key of the prefix-0 chunk
    log("[gpu] chunk rows with late score spikes")
    _compare_all_rows(wl, li)


def _fused_vs_two_calls(wl, li, what):
    """mixed_step (fused append) against append + mixed_step_attn: identical
    bits for out, lse and the whole pool; and the oracle's tolerance."""
    b = wl.batch
    g2 = run_layer(b, li)
    g1 = run_layer(b, li, fused=True)
    assert np.array_equal(g1.pool_np(), g2.pool_np()), f"{what}: fused append pool differs"
    assert np.array_equal(g1.out.cpu().numpy(), g2.out.cpu().numpy()), f"{what}: fused output bits differ"
    assert np.array_equal(g1.lse.cpu().numpy(), g2.lse.cpu().numpy()), f"{what}: fused lse bits differ"
    pool_ref, out_ref, lse_ref = oracle.step(b, li, W.SOFTMAX_SCALE)
    assert np.array_equal(g1.pool_np(), pool_ref), f"{what}: fused append differs from the oracle"
    assert_close(g1.out_np(), out_ref, g1.lse_np(), lse_ref, what=what + " fused")


@pytest.mark.parametrize("name", sorted(EDGE_CASES))
def test_fused_step_edge_cases(name):
    prefix, qlen, page = EDGE_CASES[name]
    log(f"[gpu] fused step, edge case {name}")
    wl = W.custom(prefix, qlen, page_size=page, seed=zlib.crc32(name.encode()) % 1000, name=name)
    _fused_vs_two_calls(wl, wl.layer(0), name)


@pytest.mark.parametrize("idx", [1, 2])
def test_fused_step_configs(idx):
    wl = W.config(idx)
    log(f"[gpu] fused step, config {idx}")
    _fused_vs_two_calls(wl, wl.layer(0), wl.name)


def test_fused_step_score_spike():
    wl = W.custom([100, 5, 0], [40, 1, 70], page_size=16, seed=11, name="score_spike")
    b, li = wl.batch, wl.layer(0)
    _plant_spike(b, li, 90, 0, token_row=30)
    _plant_spike(b, li, 125, 0, token_row=35)
    _plant_spike(b, li, 40, 2, token_row=41 + 60)
    log("[gpu] fused step with late score spikes")
    _fused_vs_two_calls(wl, li, "score_spike")


@pytest.mark.parametrize("idx", [1, 2])
def test_config_all_rows(idx):
    wl = W.config(idx)
    log(f"[gpu] config {idx}: {wl.name}, all rows")
    _compare_all_rows(wl, wl.layer(0))


@pytest.mark.parametrize("idx", [1, 2])
def test_config_bf16_output(idx):
    """bf16 output (round to nearest even) at the same bars as fp32: the
    rounding itself adds about 1.3e-3 aggregate relative error (half an ulp
    of 8 significant bits, averaged over a binade), the kernel's own error is
    about 1e-4."""
    wl = W.config(idx)
    log(f"[gpu] config {idx}, bf16 output")
    _compare_all_rows(wl, wl.layer(0), out_bf16=True)


def _compare_sampled(b, li, g, what, seed=0):
    rows = sample_rows(b, seed=seed)
    pool_ref = oracle.append(b, li.new_latents, li.pool)
    assert np.array_equal(g.pool_np(), pool_ref), f"{what}: append pool differs"
    out_ref, lse_ref = oracle.attend(b, li.q, pool_ref, W.SOFTMAX_SCALE, rows=rows)
    assert_close(g.out_np()[rows], out_ref, g.lse_np()[rows], lse_ref, what=f"{what} ({len(rows)} sampled rows)")


def test_config3_full_size_sampled():
    wl = W.config(3)
    log(f"[gpu] config 3 full size: {wl.name}")
    li = wl.layer(0)
    g = run_layer(wl.batch, li)
    _compare_sampled(wl.batch, li, g, "config 3")


@pytest.mark.parametrize("chunk", [0, 256, 512, 1024, 2048, 4096])
def test_config4_full_size_sampled(chunk):
    wl = W.config(4, chunk=chunk)
    log(f"[gpu] config 4 full size, chunk {chunk}")
    li = wl.layer(0)
    g = run_layer(wl.batch, li)
    _compare_sampled(wl.batch, li, g, f"config 4 C={chunk}", seed=chunk)


def test_config5_27_layers_sampled():
    import torch
    wl = W.config(5)
    log(f"[gpu] config 5: {wl.name}")
    db = mla.DeviceBatch.from_batch(wl.batch)
    check = {0: None, 13: None, 26: None}
    layers = []
    for layer in range(wl.num_layers):
        li = wl.layer(layer)
        layers.append(GpuLayer(db, li))
        if layer in check:
            check[layer] = li
    for g in layers:  # back to back on one stream, as the benchmark runs them
        g.run()
    torch.cuda.synchronize()
    log("  27 layers done")
    for layer, li in check.items():
        _compare_sampled(wl.batch, li, layers[layer], f"config 5 layer {layer}", seed=layer)


@pytest.mark.parametrize("prefix,chunk", [(24576, 8192), (57344, 4096)])
def test_prefill_node_step_sampled(prefix, chunk):
    """A prefill node's step (no decode rows): one long chunk over a long
    cached prefix, the shapes of the prefill-node step time of Eq. 3."""
    wl = W.custom([prefix], [chunk], page_size=64, seed=prefix % 997, name=f"prefill node {chunk}@{prefix}")
    log(f"[gpu] prefill-node step: chunk {chunk} at prefix {prefix}")
    li = wl.layer(0)
    g = run_layer(wl.batch, li, fused=True)
    _compare_sampled(wl.batch, li, g, wl.name, seed=1)


def test_chunk_value_range():
    """Chunk rows carry V through fp16 (values |v| <= 65504 exact; below
    2^-14 the fp16 subnormals keep at least 2^-24 absolute).  Keys with
    value dims at the largest bf16 magnitudes inside that range and at fp16
    subnormal magnitudes; the query is zero on those dims, so the scores come
    from the other dims only.  Both the decode and the chunk rows must keep
    them: relative error at the fp16 probability rounding on the large dims,
    absolute error at the subnormal spacing on the small ones."""
    wl = W.custom([300, 40, 0, 77], [1, 70, 45, 1], page_size=16, seed=5, name="value_range")
    b, li = wl.batch, wl.layer(0)
    rng = np.random.default_rng(3)
    big = np.array([0x477F, 0x4770, 0x4700, 0x46FF], dtype=np.uint16)  # 65280, 61440, 32768, 32640
    tiny = np.array([0x3380, 0x3400, 0x3480, 0x3800, 0x3880], dtype=np.uint16)  # 2^-24 .. 2^-14
    sign = np.uint16(0x8000)

    def plant(x):  # x: [..., 576] latents
        shp = x.shape[:-1] + (32,)
        x[..., 0:32] = rng.choice(big, size=shp) | (rng.integers(0, 2, size=shp, dtype=np.uint16) * sign)
        x[..., 32:64] = rng.choice(tiny, size=shp) | (rng.integers(0, 2, size=shp, dtype=np.uint16) * sign)

    finite = ~np.isnan(W.bf16_bits_to_f32(li.pool[..., 0]))
    pool = li.pool.copy()
    sub = pool[finite]
    plant(sub)
    pool[finite] = sub
    li.pool = pool
    plant(li.new_latents.reshape(-1, W.D_QK))
    li.q.reshape(-1, W.NUM_HEADS, W.D_QK)[..., 0:64] = 0
    g = run_layer(b, li, fused=True)
    pool_ref, out_ref, lse_ref = oracle.step(b, li, W.SOFTMAX_SCALE)
    assert np.array_equal(g.pool_np(), pool_ref), "append: pool differs from the oracle"
    out = g.out_np()
    assert np.isfinite(out).all()
    d_big = np.abs(out[..., 0:32] - out_ref[..., 0:32])
    d_tiny = np.abs(out[..., 32:64] - out_ref[..., 32:64])
    log(f"  value range: large dims max_abs={d_big.max():.3e} (scale 65280), "
        f"tiny dims max_abs={d_tiny.max():.3e} (scale 2^-14)")
    assert d_big.max() <= 65280 * 2.0 ** -10, "large value dims lost precision (clamped?)"
    assert d_tiny.max() <= 2.0 ** -22, "fp16-subnormal value dims lost more than the subnormal spacing"
    assert_close(out[..., 64:], out_ref[..., 64:], g.lse_np(), lse_ref, what="value range, other dims")


@pytest.mark.parametrize("keys", [64, 192, 1024])
def test_forced_chunk_key_splits(keys):
    """Every block of 8 chunk tokens cut into many key ranges (equal 64-aligned
    ranges, the last ones shorter or empty), merged by the split combine: the
    result must not depend on the split.  Page 16 and ragged chunk tails."""
    wl = W.custom([5000, 15, 0, 1300, 333], [37, 1, 70, 9, 1], page_size=16, seed=keys, name=f"split{keys}")
    log(f"[gpu] forced chunk key split {keys}")
    mla.debug_set(mla.MLA_DEBUG_CHUNK_KEYS, keys)
    try:
        _compare_all_rows(wl, wl.layer(0))
    finally:
        mla.debug_set(mla.MLA_DEBUG_CHUNK_KEYS, 0)


@pytest.mark.parametrize("unit", [1, 2, 3])
def test_forced_small_decode_units(unit):
    """Decode units of 1-3 tiles: every request is cut into many parts (up to
    ~100 for the longest), each a partial row merged by the split combine,
    several requests inside one unit where they are short.  Page 16, a chunk
    beside them."""
    wl = W.custom([3100, 15, 0, 700, 33, 64, 2000], [1, 1, 40, 1, 1, 1, 1], page_size=16, seed=40 + unit,
                  name=f"unit{unit}")
    log(f"[gpu] forced decode unit {unit}")
    mla.debug_set(mla.MLA_DEBUG_DEC_UNIT, unit)
    try:
        _compare_all_rows(wl, wl.layer(0))
    finally:
        mla.debug_set(mla.MLA_DEBUG_DEC_UNIT, 0)


@pytest.mark.parametrize("first", [1, 5, 64, 100000])
def test_decode_first_schedule_same_bits(first):
    """Workgroups that start on the decode queue (1, 5, 64, or every one of
    the launch) change only which workgroup runs which item: output, LSE and
    cache are bit-identical to the chunk-first schedule (none forced), which
    matches the oracle.  Chunks long enough to be split beside decode rows that are
    split too (small forced units)."""
    wl = W.custom([4000, 15, 0, 700, 2600, 64, 9000, 300], [1, 1, 300, 1, 1, 1, 1, 129], page_size=16,
                  seed=50 + first % 97, name=f"first{first}")
    b, li = wl.batch, wl.layer(0)
    log(f"[gpu] decode-first workgroups {first}")
    mla.debug_set(mla.MLA_DEBUG_DEC_UNIT, 7)
    mla.debug_set(mla.MLA_DEBUG_CHUNK_KEYS, 512)
    mla.debug_set(mla.MLA_DEBUG_DEC_FIRST, 0)
    try:
        base = run_layer(b, li, fused=True)
        mla.debug_set(mla.MLA_DEBUG_DEC_FIRST, first)
        g = run_layer(b, li, fused=True)
    finally:
        mla.debug_set(mla.MLA_DEBUG_DEC_FIRST, -1)
        mla.debug_set(mla.MLA_DEBUG_DEC_UNIT, 0)
        mla.debug_set(mla.MLA_DEBUG_CHUNK_KEYS, 0)
    assert np.array_equal(g.out_np().view(np.uint32), base.out_np().view(np.uint32)), "output bits differ"
    assert np.array_equal(g.lse_np().view(np.uint32), base.lse_np().view(np.uint32)), "LSE bits differ"
    assert np.array_equal(g.pool_np(), base.pool_np()), "cache differs"
    pool_ref, out_ref, lse_ref = oracle.step(b, li, W.SOFTMAX_SCALE)
    assert np.array_equal(g.pool_np(), pool_ref), "append: pool differs from the oracle"
    assert_close(g.out_np(), out_ref, g.lse_np(), lse_ref, what=wl.name)


def test_serving_steps_with_warm_plans():
    """Consecutive steps whose decode lengths grow by one token, as a decode
    node serves them: every step is a new batch, planned warm from the first
    one's plan (same key split and unit size, counts recomputed)."""
    import dataclasses
    wl = W.config(2)
    b0, li = wl.batch, wl.layer(0)
    dec = b0.q_lens == 1
    for k in range(3):
        p = b0.prefix_lens.astype(np.int64).copy()
        p[dec] = np.maximum(0, p[dec] - 2 + k)
        b = dataclasses.replace(b0, prefix_lens=p.astype(np.int32))
        log(f"[gpu] serving step {k}: decode prefixes {int(p[dec].min())}..{int(p[dec].max())}")
        g = run_layer(b, li, fused=True)
        _compare_sampled(b, li, g, f"serving step {k}", seed=k)
