"""Helpers shared by the GPU tests: upload one layer, run the HIP path through
the C ABI, read results back, and compare with the oracle."""
import sys

import numpy as np

import paper_2607_02043_amd as mla
from paper_2607_02043_amd import workloads as W

# Tolerances of the attention output against the fp64 oracle: elementwise
# max-abs 1e-2 and aggregate relative error sum|gpu - ref| / sum|ref| 2e-3.
MAX_ABS = 1e-2
MEAN_REL = 2e-3
LSE_ABS = 1e-3


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(arr_u16, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(arr_u16).view(np.int16)).to(device)


def from_dev_u16(t):
    return t.cpu().numpy().view(np.uint16)


class GpuLayer:
    """Device copies of one layer's inputs plus output buffers."""

    def __init__(self, dbatch, li, out_bf16=False, want_lse=True, device="cuda"):
        import torch
        self.dbatch = dbatch
        self.pool = to_dev(li.pool, device)
        self.new = to_dev(li.new_latents.reshape(-1, W.D_QK), device)
        self.q = to_dev(li.q.reshape(-1, W.NUM_HEADS, W.D_QK), device)
        T = dbatch.num_rows
        dt = torch.bfloat16 if out_bf16 else torch.float32
        self.out = torch.full((T, W.NUM_HEADS, W.D_V), float("nan"), dtype=dt, device=device)
        self.lse = torch.full((T, W.NUM_HEADS), float("nan"), dtype=torch.float32, device=device) if want_lse else None
        self.ws = mla.workspace_for(dbatch, device)

    def run(self, scale=W.SOFTMAX_SCALE, append=True, fused=False):
        if fused:  # append + attention in one launch
            mla.mixed_step(self.dbatch, self.q, self.new, self.pool, scale, self.out, self.lse, self.ws)
            return
        if append:
            mla.append_latent_kv(self.dbatch, self.new, self.pool)
        mla.mixed_step_attn(self.dbatch, self.q, self.pool, scale, self.out, self.lse, self.ws)

    def out_np(self):
        import torch
        return self.out.to(torch.float32).cpu().numpy().astype(np.float64)

    def lse_np(self):
        return None if self.lse is None else self.lse.cpu().numpy().astype(np.float64)

    def pool_np(self):
        return from_dev_u16(self.pool)


def run_layer(batch, li, out_bf16=False, scale=W.SOFTMAX_SCALE, fused=False):
    import torch
    db = mla.DeviceBatch.from_batch(batch)
    g = GpuLayer(db, li, out_bf16=out_bf16)
    g.run(scale, fused=fused)
    torch.cuda.synchronize()
    return g


def errors(gpu, ref):
    d = np.abs(gpu - ref)
    return float(d.max()) if d.size else 0.0, float(d.sum() / max(np.abs(ref).sum(), 1e-300)) if d.size else 0.0


def assert_close(gpu_out, ref_out, gpu_lse=None, ref_lse=None, what="", max_abs=MAX_ABS, mean_rel=MEAN_REL):
    assert np.isfinite(gpu_out).all(), f"{what}: non-finite output"
    ma, mr = errors(gpu_out, ref_out)
    log(f"  {what}: max_abs={ma:.3e} mean_rel={mr:.3e}")
    assert ma <= max_abs, f"{what}: max_abs {ma} > {max_abs}"
    assert mr <= mean_rel, f"{what}: mean_rel {mr} > {mean_rel}"
    if gpu_lse is not None and ref_lse is not None:
        assert np.isfinite(gpu_lse).all(), f"{what}: non-finite lse"
        la = float(np.abs(gpu_lse - ref_lse).max()) if gpu_lse.size else 0.0
        assert la <= LSE_ABS, f"{what}: lse max_abs {la} > {LSE_ABS}"


def sample_rows(batch, n_decode=48, seed=0):
    """Rows the oracle computes one by one at full size: every chunk's first,
    last and block-boundary rows, random chunk rows, the longest and shortest
    decode rows and random decode rows."""
    rng = np.random.default_rng(seed)
    cu = batch.cu_q
    rows = set()
    dec = [r for r in range(batch.num_reqs) if batch.q_lens[r] == 1]
    chk = [r for r in range(batch.num_reqs) if batch.q_lens[r] > 1]
    for r in chk:
        c = int(batch.q_lens[r])
        base = int(cu[r])
        for i in [0, 1, 2, 3, 4, 5, 31, 32, 33, c // 2, c - 5, c - 4, c - 3, c - 2, c - 1]:
            if 0 <= i < c:
                rows.add(base + i)
        for i in rng.choice(c, size=min(c, 24), replace=False):
            rows.add(base + int(i))
    if dec:
        lens = np.array([batch.prefix_lens[r] for r in dec])
        rows.add(int(cu[dec[int(lens.argmax())]]))
        rows.add(int(cu[dec[int(lens.argmin())]]))
        for k in rng.choice(len(dec), size=min(len(dec), n_decode), replace=False):
            rows.add(int(cu[dec[int(k)]]))
    return np.array(sorted(rows), dtype=np.int64)
