"""How close the work planner's choice is to the fastest plan (tuning tool;
needs an MI355X).

For a set of steps (single-chunk steps of a decode node: 4 to 128 decode
requests with 998 or 13968 cached tokens beside one chunk of 124 to 2040
tokens at chunk index 1 or 3; further mixed and prefill-node steps; and
the benchmark workloads 2, 3, 5 and 4 at C = 256 .. 4096), every step is
timed with the planner's own plan and with each forced pair of chunk key
split (MLA_DEBUG_CHUNK_KEYS: 64 .. 8192 keys below the longest chunk's
keys, and unsplit) and decode unit size (MLA_DEBUG_DEC_UNIT: 1 .. 128
tiles and one, two and three units per CU) in the chunk-first schedule
(MLA_DEBUG_DEC_FIRST = 0), and, for steps with both kinds of work, with
each key split beside 2/8 .. 7/8 of the CUs starting on the decode work
(MLA_DEBUG_DEC_FIRST, one decode item each).  Each time is the median of
five mixed_step calls after two warm-up calls, the last-level cache
flushed before every call; the planner's own plan is timed before and
after the forced ones, the faster kept.  The fastest of some fifty noisy
forced times sits a little below the true fastest, so a regret of 1-2 %
is within noise.  Printed: per step the planner's time, the
fastest forced plan and the planner's regret (its time over the fastest,
minus one), then the mean, 90th percentile and maximum regret; --csv also
writes every measurement (decode-first workgroups in its last column).

Usage: python -m paper_2607_02043_amd.plan_sweep [--csv FILE] [--quick]
(--quick: every fourth step only).
"""
import argparse
import itertools
import math
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

KEY_SPLITS = [64, 128, 256, 512, 1024, 2048, 4096, 8192, 16320]

# (decode requests, their cached tokens, chunk tokens, chunk prefix)
MIXED_STEPS = [(4, 998, 124, 372), (16, 13968, 1008, 1008), (8, 3569, 504, 504), (4, 842, 124, 372),
               (4, 3569, 252, 504), (32, 3569, 992, 992), (64, 998, 448, 896), (128, 3569, 384, 768),
               (16, 842, 1008, 3024), (32, 13968, 224, 672), (8, 14013, 2040, 6120), (64, 3569, 1984, 1984),
               (4, 842, 508, 0), (128, 13968, 1920, 3840), (0, 0, 1024, 4096), (0, 0, 2048, 8192),
               (0, 0, 512, 1536), (32, 998, 248, 248), (128, 842, 1920, 0), (16, 3569, 496, 1984),
               (64, 13968, 960, 960), (8, 998, 1016, 4064), (0, 0, 4096, 4096), (0, 0, 256, 768)]


def steps():
    """(name, prefix lengths, query lengths, page size) of every step."""
    from paper_2607_02043_amd import workloads as W
    out = []
    for B, K, c, p in MIXED_STEPS:
        out.append((f"mixed B={B} K={K} c={c} p={p}", [K] * B + [p], [1] * B + [c], 64))
    for idx in (2, 3, 5):
        b = W.config(idx).batch
        out.append((f"workload {idx}", [int(x) for x in b.prefix_lens], [int(x) for x in b.q_lens], b.page_size))
    for ch in (256, 1024, 2048, 4096):
        b = W.config(4, chunk=ch).batch
        out.append((f"workload 4 C={ch}", [int(x) for x in b.prefix_lens], [int(x) for x in b.q_lens], b.page_size))
    for B, K, c, i in itertools.product((4, 16, 64, 128), (998, 13968), (124, 504, 2040), (1, 3)):
        p = c * (i - 1)
        out.append((f"grid B={B} K={K} c={c} p={p}", [K] * B + [p], [1] * B + [c], 64))
    return out


def unit_sizes(prefix, q):
    tiles = sum(math.ceil((p + 1) / 32) for p, c in zip(prefix, q) if c == 1)
    if tiles == 0:
        return [0]
    u = {1, 2, 4, 8, 16, 32, 64, 128, math.ceil(tiles / 768), math.ceil(tiles / 512), math.ceil(tiles / 256)}
    return sorted(x for x in u if x <= tiles)


def key_splits(prefix, q):
    longest = max((p + c for p, c in zip(prefix, q) if c > 1), default=0)
    if longest == 0:
        return [16320]
    return sorted({k for k in KEY_SPLITS if k < longest} | {16320})


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--csv", default=None)
    ap.add_argument("--quick", action="store_true")
    args = ap.parse_args(argv)
    import torch

    import paper_2607_02043_amd as mla
    from paper_2607_02043_amd import workloads as W
    dev = torch.device("cuda:0")
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    ncu = torch.cuda.get_device_properties(dev).multi_processor_count
    all_steps = steps()[::4] if args.quick else steps()
    csv = open(args.csv, "w") if args.csv else None
    if csv:
        csv.write("step,key_split,unit,us,dec_first\n")

    def timed(db, q, new, pool, out, n=5, warm=2):
        ws = mla.workspace_for(db, device=dev)
        ts = []
        for k in range(warm + n):
            flush.fill_(k & 0xFF)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            mla.mixed_step(db, q, new, pool, W.SOFTMAX_SCALE, out, None, ws)
            e1.record()
            torch.cuda.synchronize()
            if k >= warm:
                ts.append(e0.elapsed_time(e1) * 1e3)
        return float(np.median(ts))

    rows, regrets = [], []
    for si, (name, prefix, q, page) in enumerate(all_steps):
        wl = W.custom(prefix, q, page_size=page, seed=1, name=name)
        b, li = wl.batch, wl.layer(0)
        up = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev)
        db = mla.DeviceBatch.from_batch(b, device=dev)
        pool, new, qq = up(li.pool), up(li.new_latents), up(li.q)
        out = torch.empty((b.num_rows, 16, 512), dtype=torch.float32, device=dev)
        timed(db, qq, new, pool, out, n=20, warm=10)  # page in the new buffers
        own = timed(db, qq, new, pool, out)
        best = (math.inf, None)
        forced = [(ks, u, 0) for ks, u in itertools.product(key_splits(prefix, q), unit_sizes(prefix, q))]
        if any(c == 1 for c in q) and any(c > 1 for c in q):
            forced += [(ks, 0, ncu * e // 8) for ks in key_splits(prefix, q) for e in range(2, 8)]
        for ks, u, first in forced:
            mla.debug_set(mla.MLA_DEBUG_CHUNK_KEYS, ks)
            mla.debug_set(mla.MLA_DEBUG_DEC_UNIT, u)
            mla.debug_set(mla.MLA_DEBUG_DEC_FIRST, first)
            try:
                t = timed(db, qq, new, pool, out)
            finally:
                mla.debug_set(mla.MLA_DEBUG_CHUNK_KEYS, 0)
                mla.debug_set(mla.MLA_DEBUG_DEC_UNIT, 0)
                mla.debug_set(mla.MLA_DEBUG_DEC_FIRST, -1)
            if csv:
                csv.write(f"{name},{ks},{u},{t:.2f},{first}\n")
            best = min(best, (t, (ks, u, first)))
        own = min(own, timed(db, qq, new, pool, out))  # timed again after the forced plans
        regret = own / best[0] - 1
        regrets.append(regret)
        rows.append((name, own, best[0], best[1], regret))
        print(f"[plan_sweep] {si + 1}/{len(all_steps)} {name}: planner {own:.1f} us, fastest {best[0]:.1f} us "
              f"(key split {best[1][0]}, unit {best[1][1]}, decode-first {best[1][2]}), regret {100 * regret:.1f} %",
              file=sys.stderr, flush=True)
        del pool, new, qq, out, db, wl, li
        torch.cuda.empty_cache()
    r = np.array(regrets)
    print("| step | planner µs | fastest forced µs | its key split, unit, decode-first | regret |")
    print("|---|---|---|---|---|")
    for name, own, best, (ks, u, first), reg in rows:
        print(f"| {name} | {own:.1f} | {best:.1f} | {ks}, {u or 'planned'}, {first} | {100 * reg:.1f} % |")
    print(f"\nSteps: {len(r)}; regret mean {100 * r.mean():.2f} %, 90th percentile {100 * np.percentile(r, 90):.1f} %, "
          f"max {100 * r.max():.1f} % (negative: the planner's own plan, timed separately, came out faster).")


if __name__ == "__main__":
    main()
