"""Pins of the CPU oracle against things other than itself (no GPU needed).

* brute force: dense NumPy attention over the generator's logical key arrays
  (tests/bruteforce.py), on tiny random batches with ragged prefixes and page
  sizes 1, 2, 16 and 64;
* exact arithmetic: Python decimal at 50 digits for rows with <= 4 keys;
* closed forms: q = 0 (uniform weights), identical keys, a two-key score gap
  (logistic weights), rope-only scores, scale/q exchange;
* the step's invariants: any chunk split of a prompt equals one full
  prefill, a one-token decode equals the last prefill row, weights sum to 1,
  physical page order does not matter (all bit-exact in the oracle);
* append: a per-slot Python loop, with NaN canaries elsewhere untouched.
"""
import decimal
import math

import numpy as np
import pytest

import oracle
from bruteforce import dense_step
from paper_2607_02043_amd import workloads as W

SCALE = W.SOFTMAX_SCALE


def _bf(x):
    return W.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def _val(bits):
    return W.bf16_bits_to_f32(bits).astype(np.float64)


def _tiny(prefix, qlen, page, seed, vscale=1.0):
    wl = W.custom(prefix, qlen, page_size=page, seed=seed, value_scale=vscale)
    li = wl.layer(0, keep_cached=True)
    return wl, li


# --------------------------------------------------------------- brute force
BRUTE_CASES = [
    # (prefix_lens, q_lens, page_size)
    ([0], [1], 1),
    ([5, 0, 17], [1, 9, 1], 2),
    ([16, 31, 0], [1, 1, 7], 16),
    ([40, 3], [13, 1], 16),
    ([63, 64, 0, 10], [1, 1, 33, 5], 64),
    ([2, 0, 1], [3, 2, 1], 1),
]


@pytest.mark.parametrize("case", range(len(BRUTE_CASES)))
def test_oracle_matches_dense_bruteforce(case):
    prefix, qlen, page = BRUTE_CASES[case]
    wl, li = _tiny(prefix, qlen, page, seed=100 + case)
    pool_after, out, lse = oracle.step(wl.batch, li, SCALE)
    ref_out, ref_lse = dense_step(wl.batch, li, SCALE)
    assert out.shape == ref_out.shape
    err = np.abs(out - ref_out).max() / max(np.abs(ref_out).max(), 1e-300)
    assert err < 1e-12, err
    assert np.abs(lse - ref_lse).max() < 1e-11


# ------------------------------------------------------------------ decimal
def test_oracle_matches_decimal_small_rows():
    decimal.getcontext().prec = 50
    D = decimal.Decimal
    wl, li = _tiny([0, 2, 3], [2, 1, 1], 2, seed=7)
    pool_after, out, lse = oracle.step(wl.batch, li, SCALE)
    keys_by_req = []
    for r in range(wl.batch.num_reqs):
        p, c, row0 = int(wl.batch.prefix_lens[r]), int(wl.batch.q_lens[r]), int(wl.batch.cu_q[r])
        keys = [li.cached[r][j] for j in range(p)] + [li.new_latents[row0 + i] for i in range(c)]
        keys_by_req.append(keys)
    sc = D(float(np.float32(SCALE)))
    row = 0
    for r in range(wl.batch.num_reqs):
        p, c = int(wl.batch.prefix_lens[r]), int(wl.batch.q_lens[r])
        for i in range(c):
            for h in (0, 5, 15):
                qv = [D(float(x)) for x in _val(li.q[row, h])]
                s = []
                for j in range(p + i + 1):
                    kv = [D(float(x)) for x in _val(keys_by_req[r][j])]
                    s.append(sc * sum(a * b for a, b in zip(qv, kv)))
                m = max(s)
                w = [(x - m).exp() for x in s]
                l = sum(w)
                for e in (0, 1, 255, 511):
                    o = sum(w[j] * D(float(_val(keys_by_req[r][j][e:e + 1])[0])) for j in range(len(w))) / l
                    assert abs(float(o) - out[row, h, e]) <= 1e-14 * max(1.0, abs(float(o)))
                ls = m + l.ln()
                assert abs(float(ls) - lse[row, h]) <= 1e-13 * max(1.0, abs(float(ls)))
            row += 1


# ------------------------------------------------------------- closed forms
def _explicit_step(keys_bits, q_bits, page=4, prefix=None):
    """One request whose logical keys are keys_bits [n][576]: the first
    n - c are cached, the last c are new; q_bits is [c][16][576]."""
    n = keys_bits.shape[0]
    c = q_bits.shape[0]
    p = n - c if prefix is None else prefix
    batch = W.make_batch([p], [c], page, seed=3)
    pool = np.full((batch.num_pages, page, W.D_QK), W.CANARY_BF16, dtype=np.uint16)
    for j in range(p):
        pool[batch.block_table[0, j // page], j % page] = keys_bits[j]
    li = W.LayerInputs(pool=pool, new_latents=keys_bits[p:].copy(), q=q_bits)
    return batch, li


def test_zero_query_gives_mean_of_visible_values():
    rng = np.random.default_rng(11)
    keys = _bf(rng.standard_normal((9, W.D_QK)))
    q = np.zeros((4, W.NUM_HEADS, W.D_QK), dtype=np.uint16)  # +0.0
    batch, li = _explicit_step(keys, q)
    _, out, lse = oracle.step(batch, li, SCALE)
    vals = _val(keys)
    for i in range(4):
        n_vis = 5 + i + 1
        np.testing.assert_allclose(out[i], np.broadcast_to(vals[:n_vis, :512].mean(axis=0), (16, 512)),
                                   rtol=0, atol=1e-14)
        np.testing.assert_allclose(lse[i], math.log(n_vis), rtol=0, atol=1e-14)


def test_identical_keys_return_that_value():
    rng = np.random.default_rng(12)
    one = _bf(rng.standard_normal(W.D_QK))
    keys = np.tile(one, (7, 1))
    q = _bf(rng.standard_normal((2, W.NUM_HEADS, W.D_QK)))
    batch, li = _explicit_step(keys, q)
    _, out, lse = oracle.step(batch, li, SCALE)
    v = _val(one)
    qv = _val(q).astype(np.float64)
    for i in range(2):
        np.testing.assert_allclose(out[i], np.broadcast_to(v[:512], (16, 512)), rtol=1e-15, atol=1e-15)
        s = float(np.float32(SCALE)) * (qv[i] @ v)
        np.testing.assert_allclose(lse[i], s + math.log(6 + i), rtol=1e-13, atol=1e-13)


def test_two_key_gap_gives_logistic_weights():
    # q has a single non-zero dim d; s_j = scale * a * k_j[d] -> weights are logistic in the gap
    d, a = 100, 2.0
    x0, x1 = 3.0, -1.5
    keys = np.zeros((2, W.D_QK), dtype=np.float32)
    keys[0, d], keys[1, d] = x0, x1
    keys[0, :50] = 1.0
    keys[1, 200:300] = -2.0
    q = np.zeros((1, W.NUM_HEADS, W.D_QK), dtype=np.float32)
    q[0, :, d] = a
    q[0, 3, d] = -a  # head 3 prefers key 1
    batch, li = _explicit_step(_bf(keys), _bf(q))
    _, out, lse = oracle.step(batch, li, SCALE)
    sc = float(np.float32(SCALE))
    for h in range(16):
        sign = -1.0 if h == 3 else 1.0
        gap = sc * sign * a * (x0 - x1)
        w0 = 1.0 / (1.0 + math.exp(-gap))
        k64 = keys.astype(np.float64)
        expect = w0 * k64[0, :512] + (1 - w0) * k64[1, :512]
        np.testing.assert_allclose(out[0, h], expect, rtol=0, atol=1e-14)
        s0, s1 = sc * sign * a * x0, sc * sign * a * x1
        np.testing.assert_allclose(lse[0, h], max(s0, s1) + math.log1p(math.exp(-abs(s0 - s1))),
                                   rtol=0, atol=1e-14)


def test_rope_dims_score_but_never_reach_the_output():
    # keys equal in the 512 value dims' score contribution (q is zero there) but differ
    # in the 64 rope dims; values differ.  Output = rope-weighted mix of values.
    rng = np.random.default_rng(13)
    keys = _bf(rng.standard_normal((3, W.D_QK)))
    q = np.zeros((1, W.NUM_HEADS, W.D_QK), dtype=np.float32)
    q[0, :, 512:] = W.bf16_bits_to_f32(_bf(rng.standard_normal((16, 64))))
    qb = _bf(q)
    batch, li = _explicit_step(keys, qb)
    _, out, _ = oracle.step(batch, li, SCALE)
    kv = _val(keys)
    qv = _val(qb)
    sc = float(np.float32(SCALE))
    for h in range(16):
        s = sc * (kv[:, 512:] @ qv[0, h, 512:])
        w = np.exp(s - s.max())
        w /= w.sum()
        np.testing.assert_allclose(out[0, h], w @ kv[:, :512], rtol=0, atol=1e-13)
    # and the rope dims of the latent never appear: changing them moves weights only
    keys2 = keys.copy()
    keys2[:, 512:] = keys[::-1, 512:]
    batch2, li2 = _explicit_step(keys2, qb)
    _, out2, _ = oracle.step(batch2, li2, SCALE)
    assert not np.allclose(out, out2)


def test_scale_and_query_are_exchangeable():
    # doubling the query is exact in bf16; scale * (2q).k == (2 scale) * q.k
    wl, li = _tiny([5, 0], [1, 6], 4, seed=21)
    li2 = W.LayerInputs(pool=li.pool, new_latents=li.new_latents,
                        q=_bf(2.0 * W.bf16_bits_to_f32(li.q)))
    _, o1, l1 = oracle.step(wl.batch, li, 2 * SCALE)
    _, o2, l2 = oracle.step(wl.batch, li2, SCALE)
    np.testing.assert_allclose(o1, o2, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(l1, l2, rtol=1e-13, atol=1e-13)


# --------------------------------------------------------------- invariants
def _prompt_keys_and_q(n, seed):
    rng = np.random.default_rng(seed)
    keys = _bf(rng.standard_normal((n, W.D_QK)).astype(np.float32))
    q = _bf(rng.standard_normal((n, W.NUM_HEADS, W.D_QK)).astype(np.float32))
    return keys, q


@pytest.mark.parametrize("splits", [[37], [10, 27], [1, 1, 35], [16, 16, 5], [7, 9, 11, 10]])
def test_any_chunk_split_equals_one_full_prefill(splits):
    n = sum(splits)
    page = 8
    keys, q = _prompt_keys_and_q(n, 31)
    # one full prefill
    full = W.make_batch([0], [n], page, seed=5)
    pool0 = np.full((full.num_pages, page, W.D_QK), W.CANARY_BF16, dtype=np.uint16)
    li_full = W.LayerInputs(pool=pool0, new_latents=keys, q=q)
    _, out_full, lse_full = oracle.step(full, li_full, SCALE)
    # successive steps on one pool and block-table row, one chunk each
    pool = pool0.copy()
    outs, lses = [], []
    off = 0
    for c in splits:
        b = W.Batch(page_size=page, prefix_lens=np.array([off], np.int32), q_lens=np.array([c], np.int32),
                    block_table=full.block_table, num_pages=full.num_pages)
        pool = oracle.append(b, keys[off:off + c], pool)
        o, l = oracle.attend(b, q[off:off + c], pool, SCALE)
        outs.append(o)
        lses.append(l)
        off += c
    assert np.array_equal(np.concatenate(outs), out_full)
    assert np.array_equal(np.concatenate(lses), lse_full)


@pytest.mark.parametrize("n", [1, 2, 63, 64, 65, 130])
def test_decode_equals_last_prefill_row(n):
    page = 16
    keys, q = _prompt_keys_and_q(n, 41 + n)
    full = W.make_batch([0], [n], page, seed=6)
    pool0 = np.full((full.num_pages, page, W.D_QK), W.CANARY_BF16, dtype=np.uint16)
    _, out_full, lse_full = oracle.step(full, W.LayerInputs(pool=pool0, new_latents=keys, q=q), SCALE)
    # decode: n-1 cached keys, the last token is the step's one new row
    dec = W.Batch(page_size=page, prefix_lens=np.array([n - 1], np.int32), q_lens=np.array([1], np.int32),
                  block_table=full.block_table, num_pages=full.num_pages)
    pool = oracle.append(W.Batch(page_size=page, prefix_lens=np.array([0], np.int32),
                                 q_lens=np.array([n - 1], np.int32), block_table=full.block_table,
                                 num_pages=full.num_pages), keys[:n - 1], pool0) if n > 1 else pool0
    pool = oracle.append(dec, keys[n - 1:], pool)
    o, l = oracle.attend(dec, q[n - 1:], pool, SCALE)
    assert np.array_equal(o[0], out_full[n - 1])
    assert np.array_equal(l[0], lse_full[n - 1])


def test_softmax_weights_sum_to_one():
    wl, li = _tiny([70, 0], [1, 20], 16, seed=51)
    pool_after = oracle.append(wl.batch, li.new_latents, li.pool)
    for r, row, nk in [(0, 0, 71), (1, 1, 1), (1, 20, 20)]:
        out, lse, w = oracle.attend_row_weights(wl.batch, r, nk, li.q[row], pool_after, SCALE)
        assert (w >= 0).all()
        assert np.abs(w.sum(axis=1) - 1.0).max() <= 1e-13
        o2, l2 = oracle.attend(wl.batch, li.q, pool_after, SCALE, rows=[row])
        np.testing.assert_allclose(o2[0], out, rtol=0, atol=0)


@pytest.mark.parametrize("seed", [0, 1])
def test_page_permutation_leaves_output_unchanged(seed):
    wl, li = _tiny([30, 0, 77, 5], [1, 19, 1, 4], 8, seed=61 + seed)
    b = wl.batch
    _, out, lse = oracle.step(b, li, SCALE)
    rng = np.random.default_rng(seed)
    perm = rng.permutation(b.num_pages)  # new page id of old page i is perm[i]
    pool2 = np.empty_like(li.pool)
    pool2[perm] = li.pool
    bt2 = np.where(b.block_table >= 0, perm[np.maximum(b.block_table, 0)], -1).astype(np.int32)
    b2 = W.Batch(page_size=b.page_size, prefix_lens=b.prefix_lens, q_lens=b.q_lens, block_table=bt2,
                 num_pages=b.num_pages)
    _, out2, lse2 = oracle.step(b2, W.LayerInputs(pool=pool2, new_latents=li.new_latents, q=li.q), SCALE)
    assert np.array_equal(out, out2)
    assert np.array_equal(lse, lse2)


# ------------------------------------------------------------------- append
@pytest.mark.parametrize("case", range(3))
def test_append_is_a_slot_copy_and_leaves_canaries(case):
    prefix, qlen, page = [([0], [5], 4), ([3, 9, 0], [1, 8, 2], 4), ([63, 1], [1, 70], 64)][case]
    wl, li = _tiny(prefix, qlen, page, seed=70 + case)
    b = wl.batch
    got = oracle.append(b, li.new_latents, li.pool)
    expect = li.pool.copy()
    row = 0
    written = np.zeros(expect.shape[:2], dtype=bool)
    for r in range(b.num_reqs):
        for t in range(int(b.prefix_lens[r]), int(b.prefix_lens[r] + b.q_lens[r])):
            page_id = int(b.block_table[r][t // page])
            for d in range(W.D_QK):
                expect[page_id, t % page, d] = li.new_latents[row, d]
            written[page_id, t % page] = True
            row += 1
    assert np.array_equal(got, expect)
    # nothing outside the written slots and the cached prefixes changed: canaries stay NaN
    cached = np.zeros_like(written)
    for r in range(b.num_reqs):
        for t in range(int(b.prefix_lens[r])):
            cached[b.block_table[r][t // page], t % page] = True
    untouched = ~(written | cached)
    assert (got[untouched] == W.CANARY_BF16).all()


def test_append_rejects_slot_outside_table():
    b = W.make_batch([0], [5], 4, seed=1)
    bad = W.Batch(page_size=4, prefix_lens=np.array([6], np.int32), q_lens=np.array([5], np.int32),
                  block_table=b.block_table, num_pages=b.num_pages)
    with pytest.raises(ValueError):
        oracle.append(bad, np.zeros((5, W.D_QK), np.uint16), np.zeros((b.num_pages, 4, W.D_QK), np.uint16))
