"""Measured step latencies of the mixed decode + chunked-prefill step on one GPU.

These are the measurements the step-latency model of the paper (section
4.3.1, Eq. 4; profiling and linear estimators in section 5) is fitted to:
the latency of one attention step (latent append + mixed-step attention, one
layer) for a decode batch of B requests with K cached tokens each, plus one
prefill chunk of c tokens whose own earlier chunks (prefix p) are already
cached, as in the paper's microbenchmark of section 3 (Q2): chi = B + c
tokens per step, chunk index i = 1..5 with prefix p = c (i - 1).  Pure
prefill steps (no decode rows: the prefill-node model T_step(chi_p,
chi_p * i) of Eq. 3) use B = 0.

Every step reads its keys from HBM: before each timed step a 512 MiB buffer
is written, which evicts the 256 MB last-level cache, and the step alone is
timed with HIP events on its stream.  Latent values are random (the time
does not depend on them); they are drawn on the device from a seeded
generator.

Run as a module to write the measurements as CSV:
    python -m paper_2607_02043_amd.steps --grid decode-node --out steps.csv
"""
from __future__ import annotations

import argparse
import csv
import math
import sys
import time
from typing import Iterable, List, Sequence, Tuple

import numpy as np

from .workloads import SOFTMAX_SCALE

PAGE = 64
ROW_BYTES = 576 * 2

# The paper's microbenchmark axes (section 3, Q2): decode batch size, cached
# tokens per decode request (the workloads' median prompt lengths), tokens per
# step; here extended to larger batches.
PAPER_B = (4, 8, 16, 32, 64, 128)
PAPER_K = (842, 998, 3569, 13968, 14013)
PAPER_CHI = (128, 256, 512, 1024, 2048)
N_CHUNKS = 5


def decode_node_grid(bs: Sequence[int] = PAPER_B, ks: Sequence[int] = PAPER_K,
                     chis: Sequence[int] = PAPER_CHI, n_chunks: int = N_CHUNKS) -> List[Tuple[int, int, int, int]]:
    """(B, K, c, p) configurations: decode-only steps (c = 0) and, for each
    chi > B, chunks 1..n_chunks of c = chi - B tokens at prefix c (i - 1)."""
    out = []
    for B in bs:
        for K in ks:
            out.append((B, K, 0, 0))
            for chi in chis:
                c = chi - B
                if c <= 0:
                    continue
                for i in range(1, n_chunks + 1):
                    out.append((B, K, c, c * (i - 1)))
    return out


def prefill_node_grid(chis: Sequence[int] = (512, 1024, 2048, 4096, 8192), n_chunks: int = 8):
    """(0, 0, chi_p, chi_p * i): pure prefill steps, chunk i of a long prompt."""
    return [(0, 0, chi, chi * i) for chi in chis for i in range(n_chunks)]


class StepBench:
    """Device buffers large enough for every configuration of a grid."""

    def __init__(self, configs: Iterable[Tuple[int, int, int, int]], device="cuda:0", seed: int = 0,
                 flush_mib: int = 512):
        import torch

        import paper_2607_02043_amd as mla
        self.torch, self.mla = torch, mla
        self.dev = torch.device(device)
        configs = list(configs)
        max_pages = 0
        max_rows = 1
        for B, K, c, p in configs:
            pages = B * math.ceil((K + 1) / PAGE) + (math.ceil((p + c) / PAGE) if c else 0)
            max_pages = max(max_pages, pages)
            max_rows = max(max_rows, B + c)
        self.num_pages = max_pages
        g = torch.Generator(device=self.dev)
        g.manual_seed(seed)
        # random latents (bf16), queries and new latents; scale 1 like the workloads
        self.pool = torch.randn((self.num_pages, PAGE, 576), generator=g, device=self.dev).to(torch.bfloat16)
        self.q = torch.randn((max_rows, 16, 576), generator=g, device=self.dev).to(torch.bfloat16)
        self.new = torch.randn((max_rows, 576), generator=g, device=self.dev).to(torch.bfloat16)
        self.out = torch.empty((max_rows, 16, 512), dtype=torch.float32, device=self.dev)
        self.lse = torch.empty((max_rows, 16), dtype=torch.float32, device=self.dev)
        self.flush = torch.empty(flush_mib << 20, dtype=torch.uint8, device=self.dev)
        self.rng = np.random.default_rng(seed)

    def batch(self, B: int, K: int, c: int, p: int):
        """Decode requests first (prefix K, one token), then the chunk."""
        q_lens = [1] * B + ([c] if c else [])
        prefix = [K] * B + ([p] if c else [])
        need = [math.ceil((pp + qq) / PAGE) for pp, qq in zip(prefix, q_lens)]
        width = max(need)
        perm = self.rng.permutation(self.num_pages)
        bt = np.full((len(q_lens), width), -1, dtype=np.int32)
        at = 0
        for r, n in enumerate(need):
            bt[r, :n] = perm[at:at + n]
            at += n
        return self.mla.DeviceBatch(q_lens, prefix, bt, PAGE, self.num_pages, device=self.dev)

    def time_config(self, B: int, K: int, c: int, p: int, steps: int = 6, warmup: int = 2) -> float:
        """Median µs of one mixed_step (append + attention) with a cold last-level cache."""
        torch, mla = self.torch, self.mla
        db = self.batch(B, K, c, p)
        ws = mla.workspace_for(db, device=self.dev)
        stream = torch.cuda.current_stream()
        times = []
        for k in range(warmup + steps):
            self.flush.fill_(k & 0xFF)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            mla.mixed_step(db, self.q, self.new, self.pool, SOFTMAX_SCALE, self.out, self.lse, ws, stream)
            e1.record(stream)
            if k >= warmup:
                times.append((e0, e1))
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in times])) * 1e3


def algorithmic_keys(B: int, K: int, c: int, p: int) -> int:
    return B * (K + 1) + (p + c if c else 0)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--grid", choices=["decode-node", "prefill-node", "both"], default="both")
    ap.add_argument("--out", required=True)
    ap.add_argument("--steps", type=int, default=6)
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args(argv)
    configs = []
    if args.grid in ("decode-node", "both"):
        configs += decode_node_grid()
    if args.grid in ("prefill-node", "both"):
        configs += prefill_node_grid()
    bench = StepBench(configs, seed=args.seed)
    t0 = time.time()
    with open(args.out, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["B", "K", "c", "p", "us"])
        for n, (B, K, c, p) in enumerate(configs):
            us = bench.time_config(B, K, c, p, steps=args.steps)
            w.writerow([B, K, c, p, f"{us:.2f}"])
            if n % 50 == 0:
                print(f"[steps] {n}/{len(configs)} B={B} K={K} c={c} p={p}: {us:.1f} us "
                      f"({time.time() - t0:.0f} s)", file=sys.stderr, flush=True)
    print(f"[steps] wrote {len(configs)} rows to {args.out}", file=sys.stderr, flush=True)


if __name__ == "__main__":
    main()
