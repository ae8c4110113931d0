"""Dense NumPy attention used to pin the oracle.

A different algorithm from the oracle: keys are taken from the generator's
logical arrays (cached prefix latents of each request, then the step's new
latents), never through the block table or the pool; all rows of a request
are scored at once as one dense [rows, heads, keys] tensor with an explicit
causal mask (row i of a request with prefix p sees keys 0..p+i).
"""
import numpy as np

from paper_2607_02043_amd.workloads import bf16_bits_to_f32

HEADS, DQK, DV = 16, 576, 512


def logical_keys(batch, layer_inputs, r):
    p = int(batch.prefix_lens[r])
    c = int(batch.q_lens[r])
    row0 = int(batch.cu_q[r])
    cached = bf16_bits_to_f32(layer_inputs.cached[r]).astype(np.float64).reshape(p, DQK)
    new = bf16_bits_to_f32(layer_inputs.new_latents[row0:row0 + c]).astype(np.float64)
    return np.concatenate([cached, new], axis=0)


def dense_request(batch, layer_inputs, r, scale):
    p = int(batch.prefix_lens[r])
    c = int(batch.q_lens[r])
    row0 = int(batch.cu_q[r])
    K = logical_keys(batch, layer_inputs, r)  # [p+c, 576]
    Q = bf16_bits_to_f32(layer_inputs.q[row0:row0 + c]).astype(np.float64)  # [c, 16, 576]
    S = float(np.float32(scale)) * np.einsum("ihd,jd->ihj", Q, K)
    j = np.arange(p + c)[None, None, :]
    i = np.arange(c)[:, None, None]
    S = np.where(j <= p + i, S, -np.inf)
    m = S.max(axis=2, keepdims=True)
    W = np.exp(S - m)
    l = W.sum(axis=2, keepdims=True)
    out = np.einsum("ihj,je->ihe", W / l, K[:, :DV])
    lse = (m + np.log(l))[..., 0]
    return out, lse


def dense_step(batch, layer_inputs, scale):
    outs, lses = [], []
    for r in range(batch.num_reqs):
        o, s = dense_request(batch, layer_inputs, r, scale)
        outs.append(o)
        lses.append(s)
    if not outs:
        return np.zeros((0, HEADS, DV)), np.zeros((0, HEADS))
    return np.concatenate(outs, axis=0), np.concatenate(lses, axis=0)
