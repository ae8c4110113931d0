"""Pins of the projection oracle (oracle/proj_oracle.py) against things other
than itself (no GPU needed).

* bf16 rounding: torch's float32 -> bfloat16 conversion (a library routine)
  on values spread over every binade, subnormals included, and hand-worked
  ties and a case where rounding twice (through float32) differs;
* rope: identity at position 0, the complex-multiplication form of a
  rotation, the angle of the first pair (frequency 1), norm per pair,
  composition, and the relative-position property of scores;
* RMSNorm: unit mean square with unit gain, scale invariance, constants;
* the absorbed layer equals the plain multi-head attention with explicit
  per-head keys W_UK c and values W_UV c (the form the absorption rewrites);
* positions: a prompt run as two chunks, or ended by a one-token decode,
  gives the rows of a single full prefill;
* the rounded mode (bf16 at the storage points, paged C-oracle attention)
  stays within bf16 rounding of the exact mode.
"""
import math

import numpy as np
import pytest
import torch

from oracle import proj_oracle as PO
from paper_2607_02043_amd import workloads as W

SCALE = W.SOFTMAX_SCALE


@pytest.fixture(scope="module")
def weights():
    return PO.Weights.from_bits(W.make_proj_weights(seed=5))


# ------------------------------------------------------------------- bf16
def test_round_bf16_matches_torch_conversion():
    rng = np.random.default_rng(0)
    mant = rng.uniform(1.0, 2.0, 20000)
    expo = rng.integers(-140, 120, 20000)
    sign = rng.choice([-1.0, 1.0], 20000)
    x = (sign * np.ldexp(mant, expo)).astype(np.float32)
    x = np.concatenate([x, np.float32([0.0, -0.0, 1.0, 65504.0, 1e-40, -3e-39])])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = PO.round_bf16(x.astype(np.float64))
    assert np.array_equal(got, ref)


def test_round_bf16_ties_and_single_rounding():
    one = 1.0
    assert PO.round_bf16(one + 2.0 ** -8) == 0x3F80          # tie -> even (down)
    assert PO.round_bf16(one + 3 * 2.0 ** -8) == 0x3F82      # tie -> even (up)
    assert PO.round_bf16(-(one + 2.0 ** -8)) == 0xBF80
    # just above the tie: once-rounded goes up; through float32 it would be a tie and go down
    assert PO.round_bf16(one + 2.0 ** -8 + 2.0 ** -40) == 0x3F81
    assert PO.bf16_value(0x3F81) == 1.0 + 2.0 ** -7


# ------------------------------------------------------------------- rope
def test_rope_definition_pins():
    rng = np.random.default_rng(1)
    v = rng.standard_normal((5, 64))
    base = 10000.0
    assert np.array_equal(PO.rope(v, 0, base), v)
    # the first pair turns by exactly pos radians
    e0 = np.zeros(64)
    e0[0] = 1.0
    for p in (1, 7, 1000, 32767):
        y = PO.rope(e0, p, base)
        assert y[0] == pytest.approx(math.cos(p), abs=1e-12) and y[1] == pytest.approx(math.sin(p), abs=1e-12)
        assert np.all(y[2:] == 0)
    # complex form: pair i is multiplied by exp(1j * pos * base ** (-i / 32))
    pos = np.array([0, 3, 100, 4096, 20000])
    z = v[:, 0::2] + 1j * v[:, 1::2]
    freq = np.exp(-np.log(base) * np.arange(32) / 32.0)
    zr = z * np.exp(1j * pos[:, None] * freq[None, :])
    y = PO.rope(v, pos, base)
    assert np.allclose(y[:, 0::2], zr.real, atol=1e-9) and np.allclose(y[:, 1::2], zr.imag, atol=1e-9)
    # norms of every pair are kept; rotations compose
    assert np.allclose(y[:, 0::2] ** 2 + y[:, 1::2] ** 2, v[:, 0::2] ** 2 + v[:, 1::2] ** 2)
    assert np.allclose(PO.rope(PO.rope(v, 17, base), 250, base), PO.rope(v, 267, base), atol=1e-10)


def test_rope_scores_depend_on_relative_position_only():
    rng = np.random.default_rng(2)
    a, b = rng.standard_normal(64), rng.standard_normal(64)
    for m, n in ((5, 2), (1000, 1), (300, 299), (17000, 16000)):
        ref = np.dot(PO.rope(a, m - n, 10000.0), b)
        for k in (0, 1, n):
            assert np.dot(PO.rope(a, m - k, 10000.0), PO.rope(b, n - k, 10000.0)) == pytest.approx(ref, abs=1e-9)


# ---------------------------------------------------------------- RMSNorm
def test_rms_norm_pins():
    rng = np.random.default_rng(3)
    v = rng.standard_normal((4, 512)) * np.array([[0.01], [1.0], [30.0], [1e-4]])
    y = PO.rms_norm(v, np.ones(512), 1e-6)
    ms = np.mean(v * v, axis=1)
    assert np.allclose(np.mean(y * y, axis=1), ms / (ms + 1e-6), rtol=1e-12)
    assert np.allclose(PO.rms_norm(-7.5 * v, np.ones(512), 0.0), -PO.rms_norm(v, np.ones(512), 0.0), rtol=1e-12)
    g = rng.standard_normal(512)
    assert np.allclose(PO.rms_norm(v, g, 1e-6), y * g, rtol=1e-12)
    c = np.full(512, 3.0)
    assert np.allclose(PO.rms_norm(c, np.ones(512), 1e-6), 3.0 / math.sqrt(9.0 + 1e-6), rtol=1e-14)


# ------------------------------------------------------------- whole layer
def _cached(rng, prefix_lens):
    return [rng.standard_normal((p, PO.DQK)) for p in prefix_lens]


def test_absorbed_layer_equals_multihead_definition(weights):
    rng = np.random.default_rng(4)
    q_lens, prefix = [1, 4, 3, 1], [5, 0, 3, 9]
    T = sum(q_lens)
    hidden = rng.standard_normal((T, PO.HIDDEN))
    cached = _cached(rng, prefix)
    got = PO.layer_exact(q_lens, prefix, hidden, weights, cached, SCALE)
    ref = PO.layer_unabsorbed(q_lens, prefix, hidden, weights, cached, SCALE)
    assert np.max(np.abs(got - ref)) <= 1e-10 * np.max(np.abs(ref))


def test_layer_positions_chunk_split_and_decode(weights):
    """A 7-token prompt prefilled at once equals chunks 3 + 4 over the cache
    of the first chunk, and equals a prefill of 6 then a one-token decode."""
    rng = np.random.default_rng(6)
    hidden = rng.standard_normal((7, PO.HIDDEN))
    full = PO.layer_exact([7], [0], hidden, weights, [np.zeros((0, PO.DQK))], SCALE)
    _, lat_first = PO.pre_attn(np.arange(3), hidden[:3], weights, rounded=False)
    second = PO.layer_exact([4], [3], hidden[3:], weights, [lat_first], SCALE)
    assert np.allclose(second, full[3:], rtol=1e-11, atol=1e-11 * np.abs(full).max())
    _, lat6 = PO.pre_attn(np.arange(6), hidden[:6], weights, rounded=False)
    dec = PO.layer_exact([1], [6], hidden[6:], weights, [lat6], SCALE)
    assert np.allclose(dec, full[6:], rtol=1e-11, atol=1e-11 * np.abs(full).max())
    # and the positions matter: the second chunk computed as if at position 0 differs
    wrong = PO.layer_exact([4], [0], hidden[3:], weights, [np.zeros((0, PO.DQK))], SCALE)
    assert not np.allclose(wrong, full[3:], rtol=1e-3)


def test_rounded_mode_stays_within_bf16_rounding(weights):
    wl = W.custom([37, 0, 5], [1, 9, 3], page_size=16, seed=8)
    b = wl.batch
    li = wl.layer(0)
    hidden = W.random_hidden(b.num_rows, seed=8)
    out, pool_after, q_bits, lat_bits = PO.layer(b, hidden, weights, li.pool, SCALE)
    exact = PO.layer_exact(b.q_lens, b.prefix_lens, PO.bf16_value(hidden), weights, PO.logical_cache(b, li.pool),
                           SCALE)
    rel = np.sqrt(np.mean((out - exact) ** 2) / np.mean(exact ** 2))
    assert 0 < rel < 2.0 ** -6
    # the stored values are the exact ones rounded once
    pos = PO.positions(b.q_lens, b.prefix_lens)
    _, lat_exact = PO.pre_attn(pos, PO.bf16_value(hidden), weights, rounded=False)
    assert np.array_equal(lat_bits, PO.round_bf16(lat_exact))


def test_multihead_rounded_mode_pins(weights):
    """The multi-head rounded mode: with no request routed it is the absorbed
    rounded mode exactly; with every chunk routed, it stays within fp16 / bf16
    rounding of the exact layer computed the plain multi-head way
    (layer_unabsorbed: explicit per-head keys and values, one head at a time)
    and differs from the absorbed rounded mode only by rounding.  fp16
    rounding matches numpy's IEEE half conversion on hand-worked ties."""
    assert PO.round_f16(1.0 + 2.0 ** -11) == 1.0            # tie to even (down)
    assert PO.round_f16(1.0 + 3 * 2.0 ** -11) == 1.0 + 2.0 ** -9  # tie to even (up)
    assert PO.round_f16(2.0 ** -24) == 2.0 ** -24           # smallest subnormal
    assert PO.round_f16(65504.0) == 65504.0
    wl = W.custom([37, 0, 5, 20], [1, 9, 3, 6], page_size=16, seed=9)
    b = wl.batch
    li = wl.layer(0)
    hidden = W.random_hidden(b.num_rows, seed=9)
    absorbed, *_ = PO.layer(b, hidden, weights, li.pool, SCALE)
    none = PO.layer_multihead(b, hidden, weights, li.pool, SCALE, lambda p, c: False)
    assert np.array_equal(none, absorbed)
    mh = PO.layer_multihead(b, hidden, weights, li.pool, SCALE, lambda p, c: c >= 2)
    ref = PO.layer_unabsorbed(b.q_lens, b.prefix_lens, PO.bf16_value(hidden), weights, PO.logical_cache(b, li.pool),
                              SCALE)
    rel = np.sqrt(np.mean((mh - ref) ** 2) / np.mean(ref ** 2))
    assert 0 < rel < 2.0 ** -6
    # the decode rows (c = 1) are the absorbed ones; the chunk rows differ by rounding only
    dec = np.concatenate([np.arange(int(b.cu_q[r]), int(b.cu_q[r + 1])) for r in range(b.num_reqs)
                          if b.q_lens[r] == 1])
    assert np.array_equal(mh[dec], absorbed[dec])
    d = np.abs(mh - absorbed)
    assert 0 < d.max() < 2.0 ** -5 * np.abs(ref).max()
