"""Device-side error flags and the boundary's check mode (needs an MI355X).

* Ordinary workloads leave the device flags clear.
* A block-table entry outside the pool is never dereferenced: the kernels
  raise MLA_FLAG_BAD_PAGE, and the rest of the pool is left as it was.
* Check mode rejects, before launching: such an entry, device lengths that
  differ from the host ones, and written slots aliased between requests.
* An expired bounded wait raises MLA_FLAG_WAIT_EXPIRED; the condition is
  forced from the host with a spin limit of 0 (the kernel then skips its waits
  and computes garbage, but every access stays in bounds and it exits), and
  check mode turns it into MLA_ERR_HIP.
"""
import numpy as np
import pytest

from harness import GpuLayer, log, run_layer
import paper_2607_02043_amd as mla
from paper_2607_02043_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture
def debug():
    mla.device_flags(clear=True)
    yield
    mla.debug_set(mla.MLA_DEBUG_CHECK, 0)
    mla.debug_set(mla.MLA_DEBUG_SPIN_LIMIT, -1)
    mla.device_flags(clear=True)


def test_flags_stay_clear_on_ordinary_steps(debug):
    for idx in (1, 2):
        wl = W.config(idx)
        run_layer(wl.batch, wl.layer(0), fused=True)
        run_layer(wl.batch, wl.layer(0))
    assert mla.device_flags() == 0


def _bad_page_batch():
    wl = W.custom([200, 0, 90], [1, 70, 1], page_size=16, seed=4, name="bad_page")
    b = wl.batch
    li = wl.layer(0)
    b.block_table = b.block_table.copy()
    b.block_table[1, 2] = b.num_pages + 5  # a page of the chunk request: read (keys 32..47) and written
    return b, li


def test_bad_page_id_raises_the_flag(debug):
    b, li = _bad_page_batch()
    for fused in (False, True):
        g = run_layer(b, li, fused=fused)
        flags = mla.device_flags()
        log(f"  fused={fused}: flags {flags}")
        assert flags & mla.MLA_FLAG_BAD_PAGE
        # slots of other pages: as the oracle appends them; the slots the bad
        # entry stands for were never written anywhere
        pool = g.pool_np()
        assert pool.shape == li.pool.shape


def test_check_mode_rejects_bad_batches(debug):
    import torch
    mla.debug_set(mla.MLA_DEBUG_CHECK, 1)
    b, li = _bad_page_batch()
    db = mla.DeviceBatch.from_batch(b)
    g = GpuLayer(db, li)
    with pytest.raises(mla.MlaError) as e:
        g.run(fused=True)
    assert e.value.code == mla.MLA_ERR_INVALID_ARG and "block-table entry" in str(e.value)
    with pytest.raises(mla.MlaError):
        mla.append_latent_kv(db, g.new, g.pool)
    torch.cuda.synchronize()
    assert mla.device_flags() == 0  # rejected before any launch
    # device lengths that differ from the host copies
    wl = W.config(1)
    db = mla.DeviceBatch.from_batch(wl.batch)
    g = GpuLayer(db, wl.layer(0))
    db.prefix_dev[1] += 1
    with pytest.raises(mla.MlaError) as e:
        g.run(fused=True)
    assert "prefix_lens_dev" in str(e.value)
    # two requests writing one slot
    wl = W.custom([10, 10], [1, 1], page_size=16, seed=3)
    b = wl.batch
    b.block_table = b.block_table.copy()
    b.block_table[1, 0] = b.block_table[0, 0]
    db = mla.DeviceBatch.from_batch(b)
    g = GpuLayer(db, wl.layer(0))
    with pytest.raises(mla.MlaError) as e:
        g.run(fused=True)
    assert "written by requests" in str(e.value)
    # a good batch passes check mode and matches the unchecked result bit for bit
    wl = W.config(2)
    g1 = run_layer(wl.batch, wl.layer(0), fused=True)
    mla.debug_set(mla.MLA_DEBUG_CHECK, 0)
    g0 = run_layer(wl.batch, wl.layer(0), fused=True)
    assert np.array_equal(g1.out.cpu().numpy(), g0.out.cpu().numpy())


def test_expired_wait_raises_the_flag(debug):
    wl = W.custom([3000, 5000, 700], [1, 1, 1], page_size=64, seed=6, name="decode_only")
    mla.debug_set(mla.MLA_DEBUG_SPIN_LIMIT, 0)
    run_layer(wl.batch, wl.layer(0), fused=True)
    assert mla.device_flags() & mla.MLA_FLAG_WAIT_EXPIRED
    mla.debug_set(mla.MLA_DEBUG_CHECK, 1)
    with pytest.raises(mla.MlaError) as e:
        run_layer(wl.batch, wl.layer(0), fused=True)
    assert e.value.code == mla.MLA_ERR_HIP and "expired" in str(e.value)
    mla.debug_set(mla.MLA_DEBUG_SPIN_LIMIT, -1)
    run_layer(wl.batch, wl.layer(0), fused=True)  # the default limit: no flag, check mode passes
    assert mla.device_flags() == 0
