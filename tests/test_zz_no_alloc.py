"""mixed_step_noalloc (the entry point for callers that cannot allocate)
against mixed_step, through the C ABI (needs an MI355X): two calls in a row
on the library's shared scratch, the second with a smaller batch, each
bit-identical to mixed_step with its own workspace (same kernels and plan),
and within the oracle's tolerance."""
import numpy as np
import pytest

import oracle
from harness import GpuLayer, assert_close, log
import paper_2607_02043_amd as mla
from paper_2607_02043_amd import workloads as W

pytestmark = pytest.mark.gpu


def _noalloc_vs_workspace(wl):
    import torch
    b, li = wl.batch, wl.layer(0)
    db = mla.DeviceBatch.from_batch(b)
    ref = GpuLayer(db, li)
    ref.run(fused=True)
    g = GpuLayer(db, li)
    mla.mixed_step_noalloc(db, g.q, g.new, g.pool, W.SOFTMAX_SCALE, g.out, g.lse)
    torch.cuda.synchronize()
    assert np.array_equal(g.pool_np(), ref.pool_np()), f"{wl.name}: pool differs"
    assert np.array_equal(g.out.cpu().numpy(), ref.out.cpu().numpy()), f"{wl.name}: output bits differ"
    assert np.array_equal(g.lse.cpu().numpy(), ref.lse.cpu().numpy()), f"{wl.name}: lse bits differ"
    pool_ref, out_ref, lse_ref = oracle.step(b, li, W.SOFTMAX_SCALE)
    assert np.array_equal(g.pool_np(), pool_ref)
    assert_close(g.out_np(), out_ref, g.lse_np(), lse_ref, what=wl.name + " (no-alloc)")


@pytest.mark.parametrize("first", [-1, 64])
def test_noalloc_matches_mixed_step_twice(first):
    # the larger batch first (key splits: its partials use the scratch), then a
    # smaller one; the planner's schedule, then 64 workgroups forced to start on
    # the decode work (the scratch's decode-queue counter used and left zero)
    mla.debug_set(mla.MLA_DEBUG_DEC_FIRST, first)
    try:
        for wl in (W.config(2), W.config(1)):
            log(f"[gpu] mixed_step_noalloc: {wl.name} (decode-first {first if first >= 0 else 'planned'})")
            _noalloc_vs_workspace(wl)
    finally:
        mla.debug_set(mla.MLA_DEBUG_DEC_FIRST, -1)

