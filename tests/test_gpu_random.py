"""Seeded random batches against the fp64 oracle, and two steps on two
streams at once (needs an MI355X).

* Random ragged batches: page sizes 1 .. 256, up to 40 requests, decode rows
  with prefixes up to 3000 keys and chunks of 2 .. 300 rows over prefixes up
  to 2000, some with the chunk key split forced (64 .. 1024 keys) and some
  with the decode unit size forced (1 .. 64 tiles), some with the
  workgroups that start on the decode work forced (0 .. 256), the fused and the
  two-call entry points; every output row and the whole pool.
* Concurrency: two different batches, each with its own workspace, launched
  on two streams without a wait between them; each matches the oracle and
  its own sequential run bit for bit.
"""
import numpy as np
import pytest

import oracle
from harness import GpuLayer, assert_close, log, run_layer
import paper_2607_02043_amd as mla
from paper_2607_02043_amd import workloads as W

pytestmark = pytest.mark.gpu

PAGE_SIZES = [1, 2, 4, 16, 32, 64, 128, 256]


def random_batch(seed):
    rng = np.random.default_rng(1000 + seed)
    page = int(rng.choice(PAGE_SIZES))
    R = int(rng.integers(1, 41))
    prefix, qlen = [], []
    for _ in range(R):
        if rng.random() < 0.7:
            prefix.append(int(rng.integers(0, 3001)))
            qlen.append(1)
        else:
            prefix.append(int(rng.integers(0, 2001)))
            qlen.append(int(rng.integers(2, 301)))
    keys = int(rng.integers(1, 17)) * 64 if rng.random() < 0.4 else 0
    fused = bool(rng.random() < 0.5)
    unit = int(rng.choice([1, 2, 5, 13, 64])) if rng.random() < 0.4 else 0
    first = int(rng.choice([0, 1, 3, 40, 256])) if rng.random() < 0.5 else -1
    return prefix, qlen, page, keys, fused, unit, first


@pytest.mark.parametrize("seed", range(16))
def test_random_batch_all_rows(seed):
    prefix, qlen, page, keys, fused, unit, first = random_batch(seed)
    log(f"[gpu] random batch {seed}: R={len(qlen)} page={page} rows={sum(qlen)} "
        f"chunks={sum(c > 1 for c in qlen)} key split={keys or 'planned'} unit={unit or 'planned'} "
        f"decode-first={first if first >= 0 else 'planned'} fused={fused}")
    wl = W.custom(prefix, qlen, page_size=page, seed=seed, name=f"random{seed}")
    b, li = wl.batch, wl.layer(0)
    mla.debug_set(mla.MLA_DEBUG_CHUNK_KEYS, keys)
    mla.debug_set(mla.MLA_DEBUG_DEC_UNIT, unit)
    mla.debug_set(mla.MLA_DEBUG_DEC_FIRST, first)
    try:
        g = run_layer(b, li, fused=fused)
    finally:
        mla.debug_set(mla.MLA_DEBUG_CHUNK_KEYS, 0)
        mla.debug_set(mla.MLA_DEBUG_DEC_UNIT, 0)
        mla.debug_set(mla.MLA_DEBUG_DEC_FIRST, -1)
    pool_ref, out_ref, lse_ref = oracle.step(b, li, W.SOFTMAX_SCALE)
    assert np.array_equal(g.pool_np(), pool_ref), "append: pool differs from the oracle"
    assert_close(g.out_np(), out_ref, g.lse_np(), lse_ref, what=wl.name)


def test_two_streams_at_once():
    import torch
    cases = [W.custom([900, 0, 40, 2500], [1, 150, 1, 1], page_size=16, seed=21, name="stream A"),
             W.custom([3000, 64, 7], [1, 1, 77], page_size=64, seed=22, name="stream B")]
    layers = []
    for wl in cases:
        db = mla.DeviceBatch.from_batch(wl.batch)
        layers.append((wl, GpuLayer(db, wl.layer(0)), GpuLayer(db, wl.layer(0))))
    torch.cuda.synchronize()
    # sequential reference runs on the default stream
    for _, seq, _ in layers:
        seq.run(fused=True)
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    log("[gpu] two mixed steps on two streams")
    for (_, _, par), s in zip(layers, streams):
        mla.mixed_step(par.dbatch, par.q, par.new, par.pool, W.SOFTMAX_SCALE, par.out, par.lse, par.ws, s)
    torch.cuda.synchronize()
    for wl, seq, par in layers:
        pool_ref, out_ref, lse_ref = oracle.step(wl.batch, wl.layer(0), W.SOFTMAX_SCALE)
        assert np.array_equal(par.pool_np(), pool_ref), f"{wl.name}: pool differs from the oracle"
        assert_close(par.out_np(), out_ref, par.lse_np(), lse_ref, what=wl.name)
        assert np.array_equal(par.out_np(), seq.out_np()) and np.array_equal(par.lse_np(), seq.lse_np())


def test_serving_sequence_warm_plans_all_rows():
    """Five consecutive steps of one decode node: decode lengths grow by a
    token, a request leaves and another joins, the chunk moves to its next
    chunk.  Each step's batch is close enough to the first one's for the
    planner's warm start (same split and unit size, counts recomputed); every
    step matches the oracle on every row."""
    rng = np.random.default_rng(77)
    dec = [int(x) for x in rng.integers(200, 3000, 24)]
    chunk_p, chunk_c = 512, 96
    for step in range(5):
        dec = [d + 1 for d in dec]
        if step == 2:  # one request finishes, another joins
            dec = dec[1:] + [int(rng.integers(200, 3000))]
        if step == 3:  # the chunk request moves on
            chunk_p += chunk_c
        prefix, qlen = dec + [chunk_p], [1] * len(dec) + [chunk_c]
        wl = W.custom(prefix, qlen, page_size=16, seed=300 + step, name=f"serving step {step}")
        log(f"[gpu] serving step {step}: {len(dec)} decodes, chunk {chunk_c} at {chunk_p}")
        g = run_layer(wl.batch, wl.layer(0), fused=True)
        pool_ref, out_ref, lse_ref = oracle.step(wl.batch, wl.layer(0), W.SOFTMAX_SCALE)
        assert np.array_equal(g.pool_np(), pool_ref), f"step {step}: pool differs from the oracle"
        assert_close(g.out_np(), out_ref, g.lse_np(), lse_ref, what=wl.name)
