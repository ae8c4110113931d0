"""Plain fp64 reference of the projections around the mixed-step attention,
which with it make one attention layer of the model the paper serves
(DeepSeek-V2-Lite, section 6: multi-head latent attention with 16 heads,
hidden width 2048, no query compression).

TEST INFRASTRUCTURE ONLY: imported by tests/ and the smoke check, never by
the product path.  It shares no code with the package: numpy in float64, the
formulas written out as they are defined, one request and one head at a time
where the definition is per request or per head.

Definitions (the paper only names the model; these are that model's
published attention, read as follows):
  row t of request r sits at position pos_t = p_r + (t - first row of r);
  q[t]      = W_q x[t], viewed [16][192] (128 dims without position, 64 rope);
  kv[t]     = W_dkv x[t] (512 compressed + 64 rope);
  latent[t] = (kv[t][:512] / sqrt(mean(kv[t][:512]^2) + eps) * gain,
               rope(kv[t][512:], pos_t));
  key of head h for cached latent c:  (W_UK[h] c[:512], c[512:]),  value: W_UV[h] c[:512];
  query of head h: (q[t][h][:128], rope(q[t][h][128:], pos_t));
  rope(v, pos) rotates the pairs (v[2i], v[2i+1]) by pos * base^(-2i/64);
  the absorbed query puts W_UK[h]^T q[t][h][:128] in front of the rope part,
  so that its dot product with the whole latent equals the per-head score;
  attention per head with scale sigma over keys 0 .. p_r + i (causal);
  o[t][h]   = W_UV[h] (sum_j softmax_j c_j[:512]);   out[t] = W_o concat_h o[t][h].
Weight layouts are those of the C ABI (mla_layer.h): w_q [3072][2048],
w_dkv [576][2048], kv_gain [512], w_uk_t[h][c][d] = W_UK[h][d][c],
w_uv[h][d][c] = W_UV[h][d][c], w_o [2048][2048].

Two modes.  `exact`: every value in float64, nothing rounded.  `rounded`:
the same arithmetic in float64, but each value that the GPU path stores in
bf16 is rounded to bf16 (nearest, ties to even) at that point: q[..][:128]
before the absorption, q_abs, latent, the attention output before W_UV, o,
and the result when a bf16 result is asked for.

The multi-head form of a chunk request (`layer_multihead`) has storage points
of its own, rounded the same way in the rounded mode: the per-head keys
W_UK[h] c and values W_UV[h] c of every visible latent c are stored in fp16
(round to nearest even; the rope key c[512:] is a bf16 value, exact in
fp16), the query is the bf16 q[..][:128] with the bf16 rope part of q_abs,
and the per-head output o is stored in bf16 before W_o.  The softmax
probabilities, which the GPU also holds in fp16 against a running maximum,
are not rounded here: their rounding depends on the order in which keys
arrive, which is not part of the definition.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence

import numpy as np

HIDDEN, HEADS, NOPE, ROPE, LATENT, VHEAD = 2048, 16, 128, 64, 512, 128
QK = NOPE + ROPE
DQK = LATENT + ROPE


# ------------------------------------------------------------------ bf16 values
def bf16_value(bits) -> np.ndarray:
    """float64 values of bf16 bit patterns."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def round_bf16(x) -> np.ndarray:
    """bf16 bit patterns of float64 values, rounded once to nearest, ties to
    even (8 significant bits; results below 2^-126 keep a fixed 2^-133 step)."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)  # x = m 2^e, 0.5 <= |m| < 1
    e = np.maximum(e, -125)  # the bf16 subnormal range has a fixed quantum
    step = np.ldexp(1.0, e - 8)
    y = np.rint(x / step) * step  # rint: ties to even
    return (y.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def through_bf16(x) -> np.ndarray:
    """The float64 value of round_bf16(x)."""
    return bf16_value(round_bf16(x))


# ---------------------------------------------------------------- definitions
def rope(v: np.ndarray, pos, base: float) -> np.ndarray:
    """Rotate pairs (2i, 2i+1) of the last axis (64 dims) by pos * base^(-2i/64).
    `pos` broadcasts against v's leading axes."""
    v = np.asarray(v, dtype=np.float64)
    pos = np.asarray(pos, dtype=np.float64)
    out = np.empty_like(v)
    for i in range(ROPE // 2):
        theta = float(base) ** (-(2.0 * i) / ROPE)
        ang = pos * theta
        c, s = np.cos(ang), np.sin(ang)
        x0, x1 = v[..., 2 * i], v[..., 2 * i + 1]
        out[..., 2 * i] = x0 * c - x1 * s
        out[..., 2 * i + 1] = x0 * s + x1 * c
    return out


def rms_norm(v: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    v = np.asarray(v, dtype=np.float64)
    return v / np.sqrt(np.mean(v * v, axis=-1, keepdims=True) + eps) * gain


def positions(q_lens: Sequence[int], prefix_lens: Sequence[int]) -> np.ndarray:
    """pos of every row of the step, request after request."""
    return np.concatenate([np.arange(p, p + c, dtype=np.int64) for c, p in zip(q_lens, prefix_lens)]
                          or [np.zeros(0, dtype=np.int64)])


@dataclasses.dataclass
class Weights:
    """float64 values of the layer's weights (layouts of the C ABI)."""

    w_q: np.ndarray     # [3072][2048]
    w_dkv: np.ndarray   # [576][2048]
    kv_gain: np.ndarray  # [512]
    w_uk_t: np.ndarray  # [16][512][128]
    w_uv: np.ndarray    # [16][128][512]
    w_o: np.ndarray     # [2048][2048]
    eps: float = 1e-6
    base: float = 10000.0

    @classmethod
    def from_bits(cls, bits, eps: float = 1e-6, base: float = 10000.0) -> "Weights":
        return cls(bf16_value(bits.w_q), bf16_value(bits.w_dkv), bf16_value(bits.kv_gain), bf16_value(bits.w_uk_t),
                   bf16_value(bits.w_uv), bf16_value(bits.w_o), float(np.float32(eps)), float(np.float32(base)))


# ------------------------------------------------------------- the projections
def pre_attn(pos: np.ndarray, hidden: np.ndarray, W: Weights, rounded: bool = True):
    """(q_abs [T][16][576], latent [T][576]) for hidden [T][2048] (float64
    values).  rounded: bf16 bit patterns; exact: float64."""
    x = np.asarray(hidden, dtype=np.float64)
    T = x.shape[0]
    q = (x @ W.w_q.T).reshape(T, HEADS, QK)
    kv = x @ W.w_dkv.T
    q_nope = q[:, :, :NOPE]
    if rounded:
        q_nope = through_bf16(q_nope)
    q_abs = np.empty((T, HEADS, DQK))
    for h in range(HEADS):
        q_abs[:, h, :LATENT] = q_nope[:, h, :] @ W.w_uk_t[h].T  # W_UK[h]^T q: sum over d of q[d] W_UK[h][d][c]
    q_abs[:, :, LATENT:] = rope(q[:, :, NOPE:], pos[:, None], W.base)
    latent = np.empty((T, DQK))
    latent[:, :LATENT] = rms_norm(kv[:, :LATENT], W.kv_gain, W.eps)
    latent[:, LATENT:] = rope(kv[:, LATENT:], pos, W.base)
    if rounded:
        return round_bf16(q_abs), round_bf16(latent)
    return q_abs, latent


def post_attn(attn_out: np.ndarray, W: Weights, rounded: bool = True, out_bf16: bool = False) -> np.ndarray:
    """out [T][2048] (float64 values; the bf16 values when out_bf16 and rounded)
    from the attention output [T][16][512]."""
    a = np.asarray(attn_out, dtype=np.float64)
    if rounded:
        a = through_bf16(a)
    T = a.shape[0]
    o = np.empty((T, HEADS, VHEAD))
    for h in range(HEADS):
        o[:, h, :] = a[:, h, :] @ W.w_uv[h].T
    o = o.reshape(T, HEADS * VHEAD)
    if rounded:
        o = through_bf16(o)
    out = o @ W.w_o.T
    if rounded and out_bf16:
        out = through_bf16(out)
    return out


# ------------------------------------------------------------- whole layer
def attend_logical(q_abs: np.ndarray, keys: np.ndarray, prefix: int, scale: float) -> np.ndarray:
    """Absorbed attention of one request's c rows over its logical keys
    [p + c][576]: row i sees keys 0 .. p + i.  Returns [c][16][512]."""
    c = q_abs.shape[0]
    out = np.empty((c, HEADS, LATENT))
    for i in range(c):
        k = keys[:prefix + i + 1]
        s = scale * (q_abs[i] @ k.T)  # [16][n]
        s -= s.max(axis=1, keepdims=True)
        w = np.exp(s)
        w /= w.sum(axis=1, keepdims=True)
        out[i] = w @ k[:, :LATENT]
    return out


def layer_exact(q_lens, prefix_lens, hidden, W: Weights, cached: List[np.ndarray], scale: float,
                rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """The layer in float64 with nothing rounded.  cached[r]: request r's
    cached latents [p_r][576] (float64), in logical order.  rows: only these
    output rows (every row's latent is still formed: later rows attend them)."""
    pos = positions(q_lens, prefix_lens)
    q_abs, lat = pre_attn(pos, hidden, W, rounded=False)
    want = list(range(len(pos))) if rows is None else [int(x) for x in rows]
    where = {t: k for k, t in enumerate(want)}
    o = np.empty((len(want), HEADS, LATENT))
    row = 0
    for r, (c, p) in enumerate(zip(q_lens, prefix_lens)):
        c, p = int(c), int(p)
        keys = np.concatenate([np.asarray(cached[r], dtype=np.float64).reshape(p, DQK), lat[row:row + c]])
        for i in range(c):
            if row + i in where:  # row i of the request sees keys 0 .. p + i
                o[where[row + i]] = attend_logical(q_abs[row + i:row + i + 1], keys, p + i, scale)[0]
        row += c
    return post_attn(o, W, rounded=False)


def layer(batch, hidden_bits, W: Weights, pool_bits, scale: float, out_bf16: bool = False, rows=None):
    """The layer on a paged cache with the GPU path's bf16 storage points
    (rounded mode); the attention is the C oracle's (oracle.attend, fp64).
    Returns (out [T or len(rows)][2048], pool after the append, q_abs bits,
    latent bits)."""
    from . import append, attend
    pos = positions(batch.q_lens, batch.prefix_lens)
    q_abs, lat = pre_attn(pos, bf16_value(hidden_bits), W, rounded=True)
    pool_after = append(batch, lat, pool_bits)
    o, _ = attend(batch, q_abs, pool_after, scale, rows=rows)
    return post_attn(o, W, rounded=True, out_bf16=out_bf16), pool_after, q_abs, lat


def layer_unabsorbed(q_lens, prefix_lens, hidden, W: Weights, cached: List[np.ndarray], scale: float) -> np.ndarray:
    """The same layer computed the plain multi-head way, for checking the
    absorbed form: every head gets explicit keys (W_UK[h] c, rope part) and
    values W_UV[h] c for every visible token, float64, one head at a time."""
    x = np.asarray(hidden, dtype=np.float64)
    pos = positions(q_lens, prefix_lens)
    T = x.shape[0]
    q = (x @ W.w_q.T).reshape(T, HEADS, QK)
    kv = x @ W.w_dkv.T
    out = np.zeros((T, HIDDEN))
    row = 0
    for r, (c, p) in enumerate(zip(q_lens, prefix_lens)):
        new_lat = np.empty((c, DQK))
        for i in range(c):
            v = kv[row + i, :LATENT]
            new_lat[i, :LATENT] = v / math.sqrt(float(np.dot(v, v)) / LATENT + W.eps) * W.kv_gain
            new_lat[i, LATENT:] = rope(kv[row + i, LATENT:], pos[row + i], W.base)
        lat = np.concatenate([np.asarray(cached[r], dtype=np.float64).reshape(p, DQK), new_lat])
        for i in range(c):
            t = row + i
            heads = []
            for h in range(HEADS):
                w_uk = W.w_uk_t[h].T  # [128][512]: W_UK[h][d][c]
                k_nope = lat[:p + i + 1, :LATENT] @ w_uk.T  # [n][128]
                k = np.concatenate([k_nope, lat[:p + i + 1, LATENT:]], axis=1)
                qh = np.concatenate([q[t, h, :NOPE], rope(q[t, h, NOPE:], pos[t], W.base)])
                s = scale * (k @ qh)
                pw = np.exp(s - s.max())
                pw /= pw.sum()
                vals = lat[:p + i + 1, :LATENT] @ W.w_uv[h].T  # [n][128]
                heads.append(pw @ vals)
            out[t] = W.w_o @ np.concatenate(heads)
        row += c
    return out


def logical_cache(batch, pool_bits) -> List[np.ndarray]:
    """Each request's cached prefix latents (float64), gathered through its block table."""
    pool = bf16_value(pool_bits)
    out = []
    for r in range(batch.num_reqs):
        p = int(batch.prefix_lens[r])
        rows = [pool[batch.block_table[r][j // batch.page_size], j % batch.page_size] for j in range(p)]
        out.append(np.array(rows, dtype=np.float64).reshape(p, DQK))
    return out


def round_f16(x) -> np.ndarray:
    """float64 values of x rounded once to IEEE half (nearest, ties to even)."""
    return np.asarray(x, dtype=np.float64).astype(np.float16).astype(np.float64)


def layer_multihead(batch, hidden_bits, W: Weights, pool_bits, scale: float, multi_head, rows=None):
    """The layer in the rounded mode where chunk requests with
    multi_head(p, c) true take the multi-head form (storage points in the
    module doc) and every other row the absorbed form (`layer`).  Returns
    out [T or len(rows)][2048] (float64)."""
    ref, pool_after, q_bits, lat_bits = layer(batch, hidden_bits, W, pool_bits, scale, rows=None)
    pos = positions(batch.q_lens, batch.prefix_lens)
    x = bf16_value(hidden_bits)
    q_nope = through_bf16((x @ W.w_q.T).reshape(-1, HEADS, QK)[:, :, :NOPE])  # [T][16][128]
    q_rope = bf16_value(q_bits)[:, :, LATENT:]  # [T][16][64], the rope part of q_abs
    pool = bf16_value(pool_after)
    w_uk = np.transpose(W.w_uk_t, (0, 2, 1))  # [16][128][512] = W_UK[h][d][c]
    row = 0
    for r in range(batch.num_reqs):
        c, p = int(batch.q_lens[r]), int(batch.prefix_lens[r])
        if c > 1 and multi_head(p, c):
            n = p + c
            lat = np.array([pool[batch.block_table[r][j // batch.page_size], j % batch.page_size] for j in range(n)])
            o = np.empty((c, HEADS, VHEAD))
            for h in range(HEADS):
                k_nope = round_f16(lat[:, :LATENT] @ w_uk[h].T)  # [n][128]
                vals = round_f16(lat[:, :LATENT] @ W.w_uv[h].T)  # [n][128]
                k_rope = lat[:, LATENT:]  # bf16 values, exact in fp16
                for i in range(c):
                    t = row + i
                    s = scale * (k_nope[:p + i + 1] @ q_nope[t, h] + k_rope[:p + i + 1] @ q_rope[t, h])
                    w = np.exp(s - s.max())
                    o[i, h] = (w @ vals[:p + i + 1]) / w.sum()
            o = through_bf16(o.reshape(c, HEADS * VHEAD))
            ref[row:row + c] = o @ W.w_o.T
        row += c
    return ref if rows is None else ref[np.asarray(rows)]
