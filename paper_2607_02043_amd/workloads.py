"""Seeded synthetic inputs for one decode-node mixed step.

This module only draws numbers and lays them out: request lengths, a
randomly permuted block table, a paged latent pool whose cached prefixes are
filled with random latents (every other slot holds a NaN canary), the new
latents of the step and the absorbed queries.  It holds none of the
attention arithmetic and is the one piece of code that both the oracle side
(tests, CPU baseline) and the HIP side (tests, bench) use.

Shapes follow the model the paper serves (DeepSeek-V2-Lite, section 6 of the
paper): 16 query heads, one shared latent of 512 compressed dims plus 64 rope
dims per token, value = the first 512 latent dims.  A step mixes in-flight
decode rows (one query token each) with the chunked-prefill rows of
deflected requests (section 2.3; section 4.3.1, Eq. 4: B_n decodes plus
chi - B_n prefill tokens).

Recipe (all integers and values reproducible from the seed alone):
  * lengths: fixed lists, lognormal L = clip(rint(median * exp(sigma * z)))
    with z ~ N(0,1) from numpy.random.default_rng(seed), or uniform integers;
  * decode request r with context L: prefix p = L - 1 cached keys, one new
    token (its own latent is appended in the step, so it sees L keys);
  * chunk request: prefix p cached keys, c new tokens;
  * request order: decode requests first, then the chunks in listed order;
  * pages: perm = default_rng([seed, 7]).permutation(num_pages); request r
    takes the next ceil((p_r + c_r) / P) entries of perm; table rows are
    padded with -1;
  * values: scale * N(0,1) in float32, rounded to bf16 (round to nearest
    even).  Every array has its own stream, cut into fixed 2^22-value blocks,
    block b drawn from default_rng([seed, layer, stream, b]); so results do
    not depend on the number of threads used to draw them.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import math
import os
from typing import List, Optional, Sequence

import numpy as np

NUM_HEADS = 16
D_LATENT = 512
D_ROPE = 64
D_QK = D_LATENT + D_ROPE  # 576
D_V = D_LATENT  # 512
# 1/sqrt(128 nope + 64 rope), the softmax scale of DeepSeek-V2 attention,
# rounded once to float32; both sides use exactly these bits.
SOFTMAX_SCALE = float(np.float32(1.0 / math.sqrt(192.0)))
CANARY_BF16 = 0x7FC0  # quiet NaN

_BLOCK = 1 << 22
_STREAM_CACHE, _STREAM_NEW, _STREAM_Q = 0, 1, 2
_STREAM_HIDDEN, _STREAM_ATTN_OUT = 3, 4
_STREAM_W = 10  # + index of the weight


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); NaN stays NaN."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        rounded[nan] = CANARY_BF16
    return rounded


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def random_bf16(n_values: int, scale: float, seed: int, layer: int, stream: int, offset: float = 0.0) -> np.ndarray:
    """n_values bf16 bit patterns of offset + scale * N(0,1), block-seeded (see module doc)."""
    out = np.empty(n_values, dtype=np.uint16)
    nblk = (n_values + _BLOCK - 1) // _BLOCK

    def work(b: int) -> None:
        lo = b * _BLOCK
        hi = min(n_values, lo + _BLOCK)
        rng = np.random.default_rng([seed, layer, stream, b])
        x = rng.standard_normal(hi - lo, dtype=np.float32)
        if scale != 1.0:
            x *= np.float32(scale)
        if offset != 0.0:
            x += np.float32(offset)
        out[lo:hi] = f32_to_bf16_bits(x)

    if nblk <= 1:
        for b in range(nblk):
            work(b)
    else:
        with _cf.ThreadPoolExecutor(max_workers=_threads()) as ex:
            list(ex.map(work, range(nblk)))
    return out


@dataclasses.dataclass
class Batch:
    """Lengths and page mapping of one step (identical for every layer)."""

    page_size: int
    prefix_lens: np.ndarray  # int32 [R]
    q_lens: np.ndarray  # int32 [R]
    block_table: np.ndarray  # int32 [R][max_pages_per_req], -1 padded
    num_pages: int

    @property
    def num_reqs(self) -> int:
        return int(self.q_lens.shape[0])

    @property
    def max_pages_per_req(self) -> int:
        return int(self.block_table.shape[1])

    @property
    def cu_q(self) -> np.ndarray:
        cu = np.zeros(self.num_reqs + 1, dtype=np.int32)
        np.cumsum(self.q_lens, out=cu[1:])
        return cu

    @property
    def num_rows(self) -> int:
        return int(self.q_lens.sum())

    @property
    def kv_lens(self) -> np.ndarray:
        return (self.prefix_lens + self.q_lens).astype(np.int64)


@dataclasses.dataclass
class LayerInputs:
    """Values of one layer: pool (prefixes filled, NaN elsewhere), new latents, queries."""

    pool: np.ndarray  # uint16 [num_pages][P][576]
    new_latents: np.ndarray  # uint16 [T][576]
    q: np.ndarray  # uint16 [T][16][576]
    cached: Optional[List[np.ndarray]] = None  # logical prefix latents per request (kept on request)


@dataclasses.dataclass
class Workload:
    name: str
    seed: int
    value_scale: float
    batch: Batch
    num_layers: int = 1
    # chunk requests as (prefix, length), listed after the decode requests
    chunks: Sequence = ()
    num_decode: int = 0

    def layer(self, layer: int = 0, keep_cached: bool = False) -> LayerInputs:
        return make_layer_inputs(self.batch, self.seed, layer, self.value_scale, keep_cached)


def lognormal_lengths(rng: np.random.Generator, n: int, median: float, sigma: float, lo: int, hi: int) -> np.ndarray:
    z = rng.standard_normal(n)
    return np.clip(np.rint(median * np.exp(sigma * z)), lo, hi).astype(np.int64)


def make_batch(prefix_lens: Sequence[int], q_lens: Sequence[int], page_size: int, seed: int,
               pool_factor: float = 1.25, extra_pages: int = 0, table_slack_pages: int = 0) -> Batch:
    p = np.asarray(prefix_lens, dtype=np.int64)
    c = np.asarray(q_lens, dtype=np.int64)
    if p.shape != c.shape:
        raise ValueError("prefix_lens and q_lens differ in length")
    if (c < 1).any() or (p < 0).any():
        raise ValueError("need q_len >= 1 and prefix_len >= 0")
    need = -(-(p + c) // page_size)
    total = int(need.sum())
    num_pages = max(int(math.ceil(pool_factor * total)), total) + int(extra_pages)
    num_pages = max(num_pages, 1)
    max_pages = int(need.max()) + int(table_slack_pages) if len(need) else 1
    max_pages = max(max_pages, 1)
    perm = np.random.default_rng([seed, 7]).permutation(num_pages).astype(np.int32)
    table = np.full((len(c), max_pages), -1, dtype=np.int32)
    off = 0
    for r, n in enumerate(need):
        table[r, :n] = perm[off:off + n]
        off += int(n)
    return Batch(page_size=int(page_size), prefix_lens=p.astype(np.int32), q_lens=c.astype(np.int32),
                 block_table=table, num_pages=int(num_pages))


def make_layer_inputs(batch: Batch, seed: int, layer: int, value_scale: float,
                      keep_cached: bool = False) -> LayerInputs:
    P = batch.page_size
    R = batch.num_reqs
    T = batch.num_rows
    pool = np.full((batch.num_pages, P, D_QK), CANARY_BF16, dtype=np.uint16)
    n_cached = int(batch.prefix_lens.astype(np.int64).sum())
    cached_all = random_bf16(n_cached * D_QK, value_scale, seed, layer, _STREAM_CACHE).reshape(n_cached, D_QK)
    flat = pool.reshape(batch.num_pages * P, D_QK)
    cached_list = [] if keep_cached else None
    off = 0
    for r in range(R):
        p = int(batch.prefix_lens[r])
        if p == 0:
            if keep_cached:
                cached_list.append(cached_all[0:0])
            continue
        t = np.arange(p, dtype=np.int64)
        slots = batch.block_table[r, t // P].astype(np.int64) * P + (t % P)
        flat[slots] = cached_all[off:off + p]
        if keep_cached:
            cached_list.append(cached_all[off:off + p])
        off += p
    new_latents = random_bf16(T * D_QK, value_scale, seed, layer, _STREAM_NEW).reshape(T, D_QK)
    q = random_bf16(T * NUM_HEADS * D_QK, value_scale, seed, layer, _STREAM_Q).reshape(T, NUM_HEADS, D_QK)
    return LayerInputs(pool=pool, new_latents=new_latents, q=q, cached=cached_list)


# ---------------------------------------------------------------------------
# The five workloads.  Lengths echo the paper's microbenchmark (section 3.2:
# decode batches with K cached tokens and chi total tokens per step) and its
# 32K-context model; the trace itself is private, so these seeded recipes
# stand in for it.
# ---------------------------------------------------------------------------
CHUNK_SWEEP = (0, 256, 512, 1024, 2048, 4096)


def _assemble(name: str, seed: int, value_scale: float, decode_ctx: np.ndarray, chunks, page_size: int,
              num_layers: int = 1, pool_factor: float = 1.25) -> Workload:
    decode_ctx = np.asarray(decode_ctx, dtype=np.int64)
    prefix = list(decode_ctx - 1) + [int(p) for p, _ in chunks]
    qlen = [1] * len(decode_ctx) + [int(c) for _, c in chunks]
    batch = make_batch(prefix, qlen, page_size, seed, pool_factor=pool_factor)
    return Workload(name=name, seed=seed, value_scale=value_scale, batch=batch, num_layers=num_layers,
                    chunks=tuple(chunks), num_decode=len(decode_ctx))


def config(idx: int, chunk: int = 2048) -> Workload:
    """Workload idx in 1..5.  `chunk` picks the prefill length of workload 4."""
    if idx == 1:
        return _assemble("tiny: 4 decode (64/96/128/256) + 32-token chunk at prefix 0, page 16",
                         0, 0.5, [64, 96, 128, 256], [(0, 32)], 16)
    if idx == 2:
        rng = np.random.default_rng(1)
        ctx = lognormal_lengths(rng, 32, 1024, 1.0, 16, 8192)
        return _assemble("32 decode (lognormal 1024, s=1.0) + 512-token chunk at prefix 0, page 64",
                         1, 1.0, ctx, [(0, 512)], 64)
    if idx == 3:
        rng = np.random.default_rng(2)
        ctx = lognormal_lengths(rng, 128, 2048, 1.2, 16, 32768)
        return _assemble("128 decode (lognormal 2048, s=1.2) + 2048-token chunk at prefix 6144, page 64",
                         2, 1.0, ctx, [(6144, 2048)], 64)
    if idx == 4:
        if chunk not in CHUNK_SWEEP:
            raise ValueError(f"chunk must be one of {CHUNK_SWEEP}")
        rng = np.random.default_rng(3)
        ctx = rng.integers(512, 16384, 256, endpoint=True)
        chunks = [(0, chunk)] if chunk > 0 else []
        return _assemble(f"256 decode (uniform 512..16384) + {chunk}-token chunk at prefix 0, page 64",
                         3, 1.0, ctx, chunks, 64)
    if idx == 5:
        rng = np.random.default_rng(4)
        ctx = lognormal_lengths(rng, 64, 4096, 1.0, 1, 32768)
        chunks = [(0, 1024), (1024, 1024), (3072, 1024), (8192, 1024)]
        return _assemble("27 layers x (64 decode (lognormal 4096, s=1.0) + 4 x 1024-token chunks "
                         "at prefixes 0/1024/3072/8192), page 64",
                         4, 1.0, ctx, chunks, 64, num_layers=27, pool_factor=1.0)
    raise ValueError("config index must be 1..5")


def custom(prefix_lens: Sequence[int], q_lens: Sequence[int], page_size: int = 64, seed: int = 0,
           value_scale: float = 1.0, name: str = "custom", pool_factor: float = 1.25,
           table_slack_pages: int = 0) -> Workload:
    batch = make_batch(prefix_lens, q_lens, page_size, seed, pool_factor=pool_factor,
                       table_slack_pages=table_slack_pages)
    nd = int((np.asarray(q_lens) == 1).sum())
    return Workload(name=name, seed=seed, value_scale=value_scale, batch=batch, num_decode=nd)


# ---------------------------------------------------------------------------
# Projection weights of one attention layer and its input, for the layer step
# (hidden width 2048, 16 heads, 128 + 64 query dims per head, 512 + 64 latent
# dims, 128 value dims per head).  Weights are random: the trained model is
# not used.  Each is offset + scale * N(0,1) with scale = 1/sqrt(fan-in), so
# every projection of unit-variance inputs has unit-variance outputs; the
# RMSNorm gain is 1 + 0.1 N(0,1).
# ---------------------------------------------------------------------------
HIDDEN = 2048
QK_NOPE, QK_ROPE, V_HEAD = 128, 64, 128


@dataclasses.dataclass
class ProjWeights:
    """bf16 bit patterns, in the layouts of the C ABI (mla_layer.h)."""

    w_q: np.ndarray      # [16 * 192][2048]
    w_dkv: np.ndarray    # [576][2048]
    kv_gain: np.ndarray  # [512]
    w_uk_t: np.ndarray   # [16][512][128]: w_uk transposed per head
    w_uv: np.ndarray     # [16][128][512]
    w_uk: np.ndarray     # [16][128][512]
    w_o: np.ndarray      # [2048][16 * 128]
    rms_eps: float = 1e-6
    rope_base: float = 10000.0


def make_proj_weights(seed: int = 0, layer: int = 0) -> ProjWeights:
    def draw(k, shape, fan_in, offset=0.0, scale=None):
        n = int(np.prod(shape))
        sc = scale if scale is not None else 1.0 / math.sqrt(fan_in)
        return random_bf16(n, sc, seed, layer, _STREAM_W + k, offset).reshape(shape)

    qk = QK_NOPE + QK_ROPE
    w_uk = draw(3, (NUM_HEADS, QK_NOPE, D_LATENT), QK_NOPE)
    return ProjWeights(
        w_q=draw(0, (NUM_HEADS * qk, HIDDEN), HIDDEN),
        w_dkv=draw(1, (D_QK, HIDDEN), HIDDEN),
        kv_gain=draw(2, (D_LATENT,), 1, offset=1.0, scale=0.1),
        w_uk_t=np.ascontiguousarray(w_uk.transpose(0, 2, 1)),
        w_uv=draw(4, (NUM_HEADS, V_HEAD, D_LATENT), D_LATENT),
        w_uk=w_uk,
        w_o=draw(5, (HIDDEN, NUM_HEADS * V_HEAD), NUM_HEADS * V_HEAD),
    )


def random_hidden(num_rows: int, seed: int = 0, layer: int = 0, scale: float = 1.0) -> np.ndarray:
    """Layer input: bf16 bits [T][2048] of scale * N(0,1)."""
    return random_bf16(num_rows * HIDDEN, scale, seed, layer, _STREAM_HIDDEN).reshape(num_rows, HIDDEN)


def random_attn_out(num_rows: int, seed: int = 0, layer: int = 0, scale: float = 1.0) -> np.ndarray:
    """An attention output to feed the post-attention projections alone:
    float32 [T][16][512] of scale * N(0,1) (block-seeded like random_bf16)."""
    n = num_rows * NUM_HEADS * D_V
    out = np.empty(n, dtype=np.float32)
    for b in range((n + _BLOCK - 1) // _BLOCK):
        lo, hi = b * _BLOCK, min(n, (b + 1) * _BLOCK)
        out[lo:hi] = np.random.default_rng([seed, layer, _STREAM_ATTN_OUT, b]).standard_normal(hi - lo, dtype=np.float32)
    if scale != 1.0:
        out *= np.float32(scale)
    return out.reshape(num_rows, NUM_HEADS, D_V)
