"""Per-item timeline of one mixed step (profiling tool).

Needs the profiling build of the library (`python -m
paper_2607_02043_amd.build --trace` writes libmlastep_trace.so next to the
regular one): its attention kernel records, per work item, the 100 MHz
real-time counter at the item's start and end and at the phase boundaries of
its prologue and epilogue, the item's tile count, the workgroup's hardware
id, and shader-clock stamps at the phase boundaries of the item's third
tile.  This tool runs `mixed_step` on one layer of a benchmark workload (a
few times, the last call kept) and prints a markdown summary:

* the launch span and, per item kind, duration, prologue, epilogue and time
  per tile;
* the phases of a chunk tile in shader clocks (median over the items):
  waiting at the tile barrier, issuing the tile DMA, P*V, scores + softmax;
* per workgroup: busy time and the time its last item ended, and the idle
  share of the launch;
* the longest items (the critical path).

Usage: python -m paper_2607_02043_amd.timeline --config 5 [--chunk C] [--keys KS] [--unit U] [--first D]
[--dump FILE.npy]
(--keys, --unit and --first force the chunk key split, the decode unit size
and the decode-first workgroups, as the MLA_DEBUG_CHUNK_KEYS,
MLA_DEBUG_DEC_UNIT and MLA_DEBUG_DEC_FIRST debug knobs, --first 0 being the
chunk-first schedule; --dump saves the stamps of the last launch, one row
per item.)
"""
import argparse
import ctypes
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import paper_2607_02043_amd as mla  # noqa: E402
from paper_2607_02043_amd import build as _build  # noqa: E402

SLOTS = 16        # stamps per item in the trace buffer
MAX_ITEMS = 1 << 16
TICK_US = 0.01    # the real-time counter runs at 100 MHz


def run(config, chunk=None, keys=0, calls=3, unit=0, first=-1, dump=None):
    import torch

    from paper_2607_02043_amd import workloads as W
    if not os.path.exists(_build.TRACE_LIB):
        raise SystemExit(f"{_build.TRACE_LIB} is missing: build it with python -m paper_2607_02043_amd.build --trace")
    mla.LIB_PATH = _build.TRACE_LIB
    L = mla.lib()
    L.mla_trace_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t]
    L.mla_trace_read.restype = ctypes.c_int
    wl = W.config(config, chunk=chunk) if chunk is not None else W.config(config)
    dev = torch.device("cuda:0")
    b, li = wl.batch, wl.layer(0)

    def up(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev)

    knobs = ((mla.MLA_DEBUG_CHUNK_KEYS, keys), (mla.MLA_DEBUG_DEC_UNIT, unit), (mla.MLA_DEBUG_DEC_FIRST, first))
    for k, v in knobs:
        mla.debug_set(k, v)
    try:
        db = mla.DeviceBatch.from_batch(b, device=dev)
        ws = mla.workspace_for(db, device=dev)
        pool, new, q = up(li.pool), up(li.new_latents), up(li.q)
        out = torch.empty((b.num_rows, 16, 512), dtype=torch.float32, device=dev)
        for _ in range(calls):
            mla.mixed_step(db, q, new, pool, W.SOFTMAX_SCALE, out, None, ws)
        torch.cuda.synchronize()
    finally:
        for k, _ in knobs:
            mla.debug_set(k, -1)  # each knob's default
    buf = np.zeros((MAX_ITEMS, SLOTS), dtype=np.uint64)
    if L.mla_trace_read(buf.ctypes.data, buf.nbytes) != 0:
        raise SystemExit("reading the trace buffer failed")
    if dump:
        np.save(dump, buf[last_launch(buf)])
    return wl, summarize(buf)


def last_launch(buf):
    """Indices of the items of the last launch recorded in `buf` (items whose
    start lies within 3 ms of the latest start; earlier launches of other
    shapes may have left items with higher indices)."""
    valid = buf[:, 0] > 0
    t_last = buf[valid, 0].astype(np.int64).max()
    valid &= buf[:, 0].astype(np.int64) >= t_last - int(3000 / TICK_US)
    return np.where(valid)[0]


def summarize(buf):
    """Figures of the last launch recorded in `buf`."""
    ix = last_launch(buf)
    stamp = lambda k: buf[ix, k].astype(np.int64)
    kind = (buf[ix, 8] // 1000000).astype(np.int64)   # 1: chunk item, 2: decode item
    units = (buf[ix, 8] % 1000000).astype(np.int64)   # tiles (chunk) or units (decode)
    t0 = stamp(0)
    start, end = (t0 - t0.min()) * TICK_US, (stamp(7) - t0.min()) * TICK_US
    res = {"span_us": float(end.max()), "items": int(len(ix)), "kinds": {}}
    for k, name in ((1, "chunk"), (2, "decode")):
        m = kind == k
        if not m.any():
            continue
        dur = end[m] - start[m]
        pro = (stamp(3)[m] - stamp(0)[m]) * TICK_US
        epi = (stamp(7)[m] - stamp(4)[m]) * TICK_US
        per = (dur - pro - epi) / np.maximum(units[m], 1)
        res["kinds"][name] = {"n": int(m.sum()), "dur_mean": float(dur.mean()), "dur_max": float(dur.max()),
                              "prologue": float(np.median(pro)), "epilogue": float(np.median(epi)),
                              "units_mean": float(units[m].mean()), "units_max": int(units[m].max()),
                              "us_per_unit": float(np.median(per))}
    m = (kind == 1) & (buf[ix, 11] > 0) & (buf[ix, 13] > 0)
    if m.any():
        d = lambda a, b: float(np.median(stamp(b)[m] - stamp(a)[m]))
        res["chunk_tile_clocks"] = {"barrier": d(11, 12), "dma_issue": d(12, 14), "pv": d(14, 15),
                                    "scores_softmax": d(15, 13), "total": d(11, 13)}
    hw = buf[ix, 9]
    busy, last = {}, {}
    for i in range(len(ix)):
        w = int(hw[i])
        busy[w] = busy.get(w, 0.0) + end[i] - start[i]
        last[w] = max(last.get(w, 0.0), end[i])
    bv, lv = np.array(list(busy.values())), np.array(list(last.values()))
    res["workgroups"] = {"n": len(busy), "busy_mean": float(bv.mean()), "busy_max": float(bv.max()),
                         "last_end_min": float(lv.min()), "last_end_median": float(np.median(lv)),
                         "idle_share": float(1.0 - bv.sum() / (len(busy) * res["span_us"]))}
    order = np.argsort(-(end - start))[:3]
    res["longest"] = [{"item": int(ix[i]), "kind": int(kind[i]), "units": int(units[i]),
                       "start": float(start[i]), "end": float(end[i])} for i in order]
    return res


def markdown(wl, res, cmd):
    out = [f"Workload: {wl.name} (one layer; the last of three calls).", "", f"Command: `{cmd}`", "",
           f"Launch span {res['span_us']:.1f} us, {res['items']} items.", "",
           "| items | count | duration mean / max us | prologue us | epilogue us | tiles (units) mean / max | us per tile (unit) |",
           "|---|---|---|---|---|---|---|"]
    for name, k in res["kinds"].items():
        out.append(f"| {name} | {k['n']} | {k['dur_mean']:.1f} / {k['dur_max']:.1f} | {k['prologue']:.1f} | "
                   f"{k['epilogue']:.1f} | {k['units_mean']:.1f} / {k['units_max']} | {k['us_per_unit']:.2f} |")
    if "chunk_tile_clocks" in res:
        c = res["chunk_tile_clocks"]
        out += ["", f"Chunk tile (third tile of each item, shader clocks, median, as seen by wave 0): barrier wait "
                    f"{c['barrier']:.0f}, DMA issue {c['dma_issue']:.0f}, P*V {c['pv']:.0f}, scores + softmax "
                    f"{c['scores_softmax']:.0f}, total {c['total']:.0f}."]
    w = res["workgroups"]
    out += ["", f"Workgroups: {w['n']}; busy mean {w['busy_mean']:.1f} us (max {w['busy_max']:.1f}); last item ends "
                f"min {w['last_end_min']:.1f}, median {w['last_end_median']:.1f} us; idle share of the launch "
                f"{w['idle_share']:.3f}.", "", "Longest items:", ""]
    for it in res["longest"]:
        out.append(f"* item {it['item']} ({'chunk' if it['kind'] == 1 else 'decode'}, {it['units']} tiles/units): "
                   f"{it['start']:.1f} → {it['end']:.1f} us")
    return "\n".join(out)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", type=int, default=5)
    ap.add_argument("--chunk", type=int, default=None)
    ap.add_argument("--keys", type=int, default=0)
    ap.add_argument("--unit", type=int, default=0)
    ap.add_argument("--first", type=int, default=-1)
    ap.add_argument("--dump", default=None)
    args = ap.parse_args()
    wl, res = run(args.config, args.chunk, args.keys, unit=args.unit, first=args.first, dump=args.dump)
    cmd = "python -m paper_2607_02043_amd.timeline " + " ".join(sys.argv[1:])
    print(markdown(wl, res, cmd.strip()), flush=True)


if __name__ == "__main__":
    main()
