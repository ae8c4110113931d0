#!/usr/bin/env python3
"""Benchmark of one decode-node mixed step (latent append + mixed-step
attention) on one MI355X, through the C ABI.

Headline (default): the full-depth step, 27 layers back to back on one stream,
each with its own paged latent cache; per layer 64 decode requests (lognormal
contexts, median 4096, sigma 1.0, clipped to 32768) plus the chunks of four
deflected prompts, 1024 tokens each at prefixes 0 / 1024 / 3072 / 8192, page
size 64 (the paper's mixed step: section 2.3, section 4.3.1 Eq. 4; the model of
section 6).  `--config N` picks another workload (1..5; `--chunk C` sets
workload 4's chunk length).

The same JSON line also carries sub-records (unless --no-sub): workload 2
(32 decodes + a 512-token chunk), workload 3 (128 decodes + a 2048-token
chunk over a 6144-token prefix), the step-latency curve over the prefill
chunk length C = 0 .. 4096 at the fixed 256-request decode batch of
workload 4, and plan-inclusive steps (decode lengths grow by one token every
step, so the host plans every step).

Timing: W untimed warm-up steps, then K timed steps bracketed by
torch.cuda.synchronize().  All inputs are resident in HBM before timing
starts.  Unless --no-rotate is given, the step cycles through enough
independent copies of its buffers (pool, queries, new latents, outputs) that
the rotating working set is >= 1 GiB, four times the 256 MB last-level
(Infinity) cache, so bytes really come from HBM.

Printed: one JSON line (metric, value = us/step, roofline of the mixed_step
call from HIP events on its stream, CPU-oracle baseline on rank 0).
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16/fp16 MFMA
ROTATE_TARGET_BYTES = 1 << 30
METRIC = "mixed-step MLA attention µs/step; TB/s & TFLOP/s as % of combined roofline"
DEFAULT_CONFIG = 5
CPU_SAMPLE_PAIRS = 4_000_000  # query-key pairs of the oracle sample (10-30 s of host work in all)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash(root=ROOT):
    """Hash of the attention kernels' sources (kernels, host planner, shared
    header) with comments and blank lines left out, so that a profile taken
    from them stays valid across comment edits and no longer after any code
    change."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in ("mla_kernels.hip", "mla_api.cpp", "mla_kernels.h"):
        with open(os.path.join(root, "paper_2607_02043_amd", "csrc", f)) as fh:
            text = re.sub(r"/\*.*?\*/", "", fh.read(), flags=re.S)
        for line in text.splitlines():
            code = line.split("//", 1)[0].rstrip()
            if code:
                h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def profiled_traffic(config_idx, root=ROOT):
    """HBM bytes per mixed_step call from the committed rocprofv3 counter
    summary, or None if there is none for this workload or the kernels changed
    since it was taken."""
    path = os.path.join(root, "profiles", "mixed_step_config%d.md" % config_idx)
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and line.startswith("    "):
                k, v = line.strip().split(":", 1)
                fields[k.strip()] = v.strip()
    if fields.get("kernel_source_sha256_16") != kernel_source_hash(root):
        return None
    try:
        return int(fields["traffic_bytes_per_call"])
    except (KeyError, ValueError):
        return None


# ---------------------------------------------------------------- work model
def algorithmic_work(batch, out_bytes_per_elem=4):
    """Bytes and flops the method must move / compute for one layer.

    Fused step (append + attention): every cached key read once (1152 B per
    cached latent), every new latent read once and written once into its
    page, queries read once (16 x 576 bf16 per row), outputs written once
    (16 x 512 per row), block-table entries read once, plus the two length
    words of each request.  The attention call alone (append done before)
    reads the new latents from the cache instead: 1152 B per key, cached or
    new, and writes none.  flops: 2 x 16 x (576 + 512) per (query token,
    visible key) pair.  lse and softmax work are not counted.
    """
    p = batch.prefix_lens.astype(np.int64)
    c = batch.q_lens.astype(np.int64)
    T = int(c.sum())
    keys = int((p + c).sum())
    pages = int(np.ceil((p + c) / batch.page_size).sum())
    common = 18432 * T + 16 * 512 * out_bytes_per_elem * T + 4 * pages + 8 * batch.num_reqs
    step_bytes = 1152 * int(p.sum()) + 2 * 1152 * T + common
    attn_bytes = 1152 * keys + common
    pairs = int((c * p + c * (c + 1) // 2).sum())
    flops = 34816 * pairs
    return {"attn_bytes": attn_bytes, "step_bytes": step_bytes, "flops": flops, "pairs": pairs, "rows": T,
            "keys": keys}


def ideal_time_us(step_bytes, step_flops):
    return max(step_bytes / (HBM_PEAK_GBS * 1e9), step_flops / (MFMA_BF16_PEAK_TFLOPS * 1e12)) * 1e6


def bound_of(step_bytes, step_flops):
    return "hbm" if step_bytes / HBM_PEAK_GBS >= step_flops / (MFMA_BF16_PEAK_TFLOPS * 1e3) else "mfma"


def summary(wl, m, two_call=False):
    """Step figures of one measured workload (all layers of a step)."""
    work, L = m["work"], wl.num_layers
    step_bytes = (work["attn_bytes"] if two_call else work["step_bytes"]) * L
    step_flops = work["flops"] * L
    ideal = ideal_time_us(step_bytes, step_flops)
    us = m["us_per_step"]
    return {"workload": wl.name, "us_per_step": round(us, 3), "ideal_us": round(ideal, 3),
            "roofline_frac": round(ideal / us, 4), "bound": bound_of(step_bytes, step_flops),
            "TB_per_s": round(step_bytes / (us * 1e-6) / 1e12, 3),
            "TFLOP_per_s": round(step_flops / (us * 1e-6) / 1e12, 2),
            "call_us": {"mean": round(m["attn_us"], 3), "p10": round(m["p10"], 3), "p50": round(m["p50"], 3),
                        "p90": round(m["p90"], 3)}}


# -------------------------------------------------------------------- bench
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=DEFAULT_CONFIG)
    ap.add_argument("--chunk", type=int, default=2048, help="prefill chunk length of workload 4")
    ap.add_argument("--out-dtype", choices=["f32", "bf16"], default="f32")
    ap.add_argument("--no-rotate", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sub", action="store_true",
                    help="only the selected workload (no sub-records for workloads 2, 3, the workload-4 curve "
                         "and the plan-inclusive steps)")
    ap.add_argument("--two-call", action="store_true",
                    help="time append_latent_kv + mixed_step_attn instead of the fused mixed_step")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one device copy of this many MiB (counter calibration)")
    ap.add_argument("--layer", action="store_true",
                    help="time the whole attention layer (projections + append + attention, mla_attention_layer) "
                         "instead of the mixed step alone")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only (--gpus 1): every decode node of the "
                                   "paper's deployment is an independent one-GPU unit; "
                                   f"--gpus {args.gpus} is not supported"}))
        sys.exit(2)

    import torch

    from paper_2607_02043_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    wl = W.config(args.config, chunk=args.chunk) if args.config == 4 else W.config(args.config)
    if args.layer:
        result = layer_bench(args, wl)
        if not args.no_cpu_baseline:
            result["cpu_baseline"] = cpu_baseline(wl, args.config, layer=True)
        print(json.dumps(result), flush=True)
        return
    m = measure(args, wl, args.steps, args.warmup, calib=args.calib_copy_mib)
    work, b, L = m["work"], wl.batch, wl.num_layers
    out_bf16 = args.out_dtype == "bf16"
    us_per_step, call_us = m["us_per_step"], m["attn_us"]
    head = summary(wl, m, args.two_call)

    # roofline of the timed call (per layer): the fused step (attention_kernel
    # with the append, plus the split merge when the batch has split rows), or
    # the attention call alone
    call_bytes = work["attn_bytes"] if args.two_call else work["step_bytes"]
    bound = bound_of(call_bytes, work["flops"])
    if bound == "hbm":
        ach = call_bytes / (call_us * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4)}
    else:
        ach = work["flops"] / (call_us * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(ach / MFMA_BF16_PEAK_TFLOPS, 4)}
    roof["traffic"] = profiled_traffic(args.config) if not (out_bf16 or args.two_call) else None
    roof["kernel"] = ("mixed_step_attn call (attention_kernel + combine_kernel)" if args.two_call
                      else "mixed_step call (attention_kernel with the fused append, + combine_kernel when rows "
                           "are split)")
    roof["per_launch_us"] = round(call_us, 3)
    roof["launches_per_step"] = L
    roof["algorithmic_bytes"] = call_bytes
    roof["algorithmic_flops"] = work["flops"]

    result = {
        "metric": METRIC,
        "value": round(us_per_step, 3),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(us_per_step / 1e3, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "layers": L, "page_size": b.page_size, "requests": b.num_reqs,
                   "rows": work["rows"], "decode_rows": wl.num_decode, "chunks": [list(x) for x in wl.chunks],
                   "out_dtype": args.out_dtype, "rotating_sets": m["n_rot"], "parallelism": "single GPU",
                   "entry": "append_latent_kv + mixed_step_attn" if args.two_call else "mixed_step"},
        "step": {"ideal_us": head["ideal_us"], "roofline_frac": head["roofline_frac"], "bound": head["bound"],
                 "TB_per_s": head["TB_per_s"], "TFLOP_per_s": head["TFLOP_per_s"],
                 "algorithmic_bytes": call_bytes * L, "algorithmic_flops": work["flops"] * L,
                 "call_us": head["call_us"]},
        "roofline": roof,
    }

    if not args.no_sub:
        sub = {}
        n_sub, w_sub = max(10, args.steps), max(3, args.warmup)
        for idx in (2, 3):
            if idx == args.config:
                continue
            wi = W.config(idx)
            sub[f"workload_{idx}"] = summary(wi, measure(args, wi, n_sub, w_sub))
            del wi
        # step latency vs prefill chunk length at the fixed decode batch of
        # workload 4 (the paper's chi counts decode + prefill tokens: 256 + C)
        curve = []
        for c in W.CHUNK_SWEEP:
            wc = W.config(4, chunk=c)
            s = summary(wc, measure(args, wc, n_sub, w_sub))
            curve.append({"chunk": c, "chi": wc.num_decode + c, "us_per_step": s["us_per_step"],
                          "ideal_us": s["ideal_us"], "roofline_frac": s["roofline_frac"], "bound": s["bound"]})
            log(f"[bench] curve C={c}: {s['us_per_step']:.1f} us/step (ideal {s['ideal_us']:.1f})")
            del wc
        sub["workload_4_curve"] = {"workload": "256 decode (uniform 512..16384) + C-token chunk at prefix 0, "
                                               "page 64", "points": curve}
        sub["plan_inclusive"] = [plan_inclusive(args, W.config(idx), n_sub, w_sub) for idx in (2, args.config)
                                 if idx in (2, 3, 5)]
        # host planning alone for the other workloads (new batch every step)
        plans = {}
        for name, wi in (("workload_3", W.config(3)), ("workload_4_c2048", W.config(4, chunk=2048)),
                         ("workload_4_c4096", W.config(4, chunk=4096))):
            cold, warm = host_plan_times(advancing_batches(wi, 25))
            plans[name] = {"workload": wi.name, "host_plan_us": warm, "host_plan_full_us": cold}
            log(f"[bench] host plan {name}: {warm['median']:.1f} us warm, {cold['median']:.1f} us in full")
        sub["host_plan"] = plans
        result["sub"] = sub

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, args.config)
    print(json.dumps(result), flush=True)


# Projection shapes of one layer (hidden 2048, 16 heads, 128 + 64 query dims,
# 512 + 64 latent dims, 128 value dims per head).
PROJ_FLOPS_PER_ROW = 2 * (2048 * 3648 + 16 * 128 * 512 + 16 * 512 * 128 + 2048 * 2048)
PROJ_WEIGHT_BYTES = 2 * (3648 * 2048 + 512 + 16 * 512 * 128 + 16 * 128 * 512 + 2048 * 2048)


def layer_work(batch):
    """Algorithmic bytes and flops of one attention layer: the mixed step's
    (keys once, block table, new latents written) plus the weights read once,
    the hidden input read and the fp32 output written; the intermediates
    between kernels (queries, attention output) are not counted, a fused
    layer would not move them."""
    a = algorithmic_work(batch)
    T = a["rows"]
    pages = int(np.ceil((batch.prefix_lens.astype(np.int64) + batch.q_lens) / batch.page_size).sum())
    step_bytes = 1152 * a["keys"] + 4 * pages + 1152 * T + PROJ_WEIGHT_BYTES + T * (2048 * 2 + 2048 * 4)
    proj_flops = PROJ_FLOPS_PER_ROW * T
    return {"bytes": step_bytes, "flops": a["flops"] + proj_flops, "attn_flops": a["flops"],
            "proj_flops": proj_flops, "rows": T, "keys": a["keys"], "pairs": a["pairs"]}


def layer_bench(args, wl):
    """Whole attention layers (mla_attention_layer) of the workload: W warm-up
    steps, K timed steps of all layers, then the same steps again with HIP
    events around the three phases (projections before, mixed step, after).
    The phases are those of the absorbed sequence, every row on the absorbed
    kernel; the layer call itself may send long chunk requests to the
    multi-head path instead, so the phases need not add up to the step."""
    import torch

    import paper_2607_02043_amd as mla
    from paper_2607_02043_amd import workloads as W

    dev = torch.device("cuda:0")
    b = wl.batch
    L = wl.num_layers
    work = layer_work(b)
    T = work["rows"]
    log(f"[bench] layer mode: {wl.name}; rows={T} keys={work['keys']}")
    db = mla.DeviceBatch.from_batch(b, device=dev)

    def up(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev)

    t0 = time.time()
    layers = []
    for layer in range(L):
        li = wl.layer(layer)
        layers.append({"pool": up(li.pool), "w": mla.DeviceProjWeights(W.make_proj_weights(wl.seed, layer), dev),
                       "hidden": up(W.random_hidden(T, wl.seed, layer)),
                       "out": torch.empty((T, 2048), dtype=torch.float32, device=dev)})
        del li
    log(f"[bench] inputs generated and uploaded in {time.time() - t0:.1f}s")
    set_bytes = sum(d["pool"].numel() * 2 + d["hidden"].numel() * 2 + T * 2048 * 4 for d in layers) + \
        L * PROJ_WEIGHT_BYTES
    n_rot = 1 if args.no_rotate else max(1, math.ceil(ROTATE_TARGET_BYTES / set_bytes))
    rotations = [layers] + [[{"pool": d["pool"].clone(), "w": d["w"], "hidden": d["hidden"].clone(),
                              "out": torch.empty_like(d["out"])} for d in layers] for _ in range(n_rot - 1)]
    # rotated copies share the weights only when one set already exceeds the rotation target
    if n_rot > 1:
        for k in range(1, n_rot):
            for j, d in enumerate(rotations[k]):
                d["w"] = mla.DeviceProjWeights(W.make_proj_weights(wl.seed, 1000 * k + j), dev)
    log(f"[bench] {n_rot} rotating buffer set(s) of {set_bytes / 2**20:.1f} MiB")
    ws = mla.layer_workspace_for(db, device=dev)
    stream = torch.cuda.current_stream()
    scale = W.SOFTMAX_SCALE

    def step(k):
        for d in rotations[k % n_rot]:
            mla.mla_attention_layer(db, d["hidden"], d["w"], d["pool"], scale, d["out"], ws, stream)

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        step(k)
    torch.cuda.synchronize()
    us_per_step = (time.perf_counter() - t_start) / args.steps * 1e6

    # phases, with HIP events on the stream: the calls mla_attention_layer makes
    # when no request takes the multi-head path
    q = torch.empty((T, 16, 576), dtype=torch.int16, device=dev)
    lat = torch.empty((T, 576), dtype=torch.int16, device=dev)
    o = torch.empty((T, 16, 512), dtype=torch.bfloat16, device=dev)
    pws = torch.empty(mla.mla_proj_workspace_bytes(T), dtype=torch.uint8, device=dev)
    aws = mla.workspace_for(db, device=dev)
    ph = {"pre": [], "attn": [], "post": []}
    n_ev = max(8, min(args.steps, 50))
    for k in range(n_ev):
        for d in rotations[k % n_rot]:
            e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            e[0].record(stream)
            mla.mla_pre_attn(db, d["hidden"], d["w"], q, lat, pws, stream)
            e[1].record(stream)
            mla.mixed_step(db, q, lat, d["pool"], scale, o, None, aws, stream)
            e[2].record(stream)
            mla.mla_post_attn(o, d["w"], d["out"], pws, stream)
            e[3].record(stream)
            ph["pre"].append((e[0], e[1]))
            ph["attn"].append((e[1], e[2]))
            ph["post"].append((e[2], e[3]))
    torch.cuda.synchronize()
    us = {k: float(np.mean([a.elapsed_time(z) for a, z in v])) * 1e3 for k, v in ph.items()}
    log(f"[bench] layer step {us_per_step:.1f} us; phases: pre {us['pre']:.1f}, mixed step {us['attn']:.1f}, "
        f"post {us['post']:.1f} us")

    bytes_all, flops_all = work["bytes"] * L, work["flops"] * L
    ideal = ideal_time_us(bytes_all, flops_all)
    proj_us = us["pre"] + us["post"]
    proj_tflops = work["proj_flops"] / (proj_us * 1e-6) / 1e12
    a = algorithmic_work(b, 2)
    attn_bound_hbm = a["step_bytes"] / HBM_PEAK_GBS >= a["flops"] / (MFMA_BF16_PEAK_TFLOPS * 1e3)
    if attn_bound_hbm:
        ach = a["step_bytes"] / (us["attn"] * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4)}
    else:
        ach = a["flops"] / (us["attn"] * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(ach / MFMA_BF16_PEAK_TFLOPS, 4)}
    roof.update({"traffic": None, "kernel": "mixed_step inside the layer (bf16 attention output)",
                 "per_launch_us": round(us["attn"], 3)})
    return {
        "metric": "MLA attention-layer step µs/step (projections + append + attention); % of combined roofline",
        "value": round(us_per_step, 3), "unit": "us/step", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(us_per_step / 1e3, 6), "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic (random weights)",
        "config": {"workload": wl.name, "layers": L, "rows": T, "page_size": b.page_size,
                   "rotating_sets": n_rot, "parallelism": "single GPU", "entry": "mla_attention_layer",
                   "out_dtype": "f32"},
        "step": {"ideal_us": round(ideal, 3), "roofline_frac": round(ideal / us_per_step, 4),
                 "TB_per_s": round(bytes_all / (us_per_step * 1e-6) / 1e12, 3),
                 "TFLOP_per_s": round(flops_all / (us_per_step * 1e-6) / 1e12, 2),
                 "algorithmic_bytes": bytes_all, "algorithmic_flops": flops_all},
        "phases_us": {k: round(v, 2) for k, v in us.items()},
        "projections": {"flops": work["proj_flops"], "us": round(proj_us, 2), "TFLOP_per_s": round(proj_tflops, 1),
                        "mfma_frac": round(proj_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
                        "weight_bytes": PROJ_WEIGHT_BYTES},
        "roofline": roof,
    }


def measure(args, wl, steps, warmup, calib=0, batches=None):
    """Upload one workload (rotating buffer sets), time `steps` whole steps
    after `warmup` untimed ones, then the same steps again with HIP events
    around each attention call on its stream.  `batches`: one
    DeviceBatch per step (warm-up steps first) instead of the workload's own."""
    import torch

    import paper_2607_02043_amd as mla
    from paper_2607_02043_amd import workloads as W

    dev = torch.device("cuda:0")
    b = wl.batch
    out_bf16 = args.out_dtype == "bf16"
    work = algorithmic_work(b, 2 if out_bf16 else 4)
    L = wl.num_layers
    log(f"[bench] workload: {wl.name}; rows={work['rows']} keys={work['keys']} pairs={work['pairs']}")

    dbs = batches if batches is not None else [mla.DeviceBatch.from_batch(b, device=dev)]
    ws_bytes = max(mla.mixed_step_workspace_bytes(d) for d in dbs)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device=dev) if ws_bytes > 0 else None

    def up(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev)

    # one buffer set per layer; rotation copies for small steps
    layer_sets = []
    t0 = time.time()
    for layer in range(L):
        li = wl.layer(layer)
        layer_sets.append({"pool": up(li.pool), "new": up(li.new_latents), "q": up(li.q)})
        del li
    log(f"[bench] inputs generated and uploaded in {time.time() - t0:.1f}s")
    odt = torch.bfloat16 if out_bf16 else torch.float32
    set_bytes = sum(s["pool"].numel() * 2 + s["new"].numel() * 2 + s["q"].numel() * 2 for s in layer_sets)
    set_bytes += L * work["rows"] * 16 * 512 * (2 if out_bf16 else 4)
    n_rot = 1 if args.no_rotate else max(1, math.ceil(ROTATE_TARGET_BYTES / set_bytes))
    rotations = []
    for k in range(n_rot):
        layers = []
        for s in layer_sets:
            d = {key: (v if k == 0 else v.clone()) for key, v in s.items()}
            d["out"] = torch.empty((work["rows"], 16, 512), dtype=odt, device=dev)
            d["lse"] = torch.empty((work["rows"], 16), dtype=torch.float32, device=dev)
            layers.append(d)
        rotations.append(layers)
    log(f"[bench] {n_rot} rotating buffer set(s) of {set_bytes / 2**20:.1f} MiB")

    stream = torch.cuda.current_stream()
    scale = W.SOFTMAX_SCALE

    def step(k, ev=None):
        db = dbs[k % len(dbs)]
        for j, d in enumerate(rotations[k % n_rot]):
            if args.two_call:
                mla.append_latent_kv(db, d["new"], d["pool"], stream)
            if ev is not None:
                ev[j][0].record(stream)
            if args.two_call:
                mla.mixed_step_attn(db, d["q"], d["pool"], scale, d["out"], d["lse"], ws, stream)
            else:
                mla.mixed_step(db, d["q"], d["new"], d["pool"], scale, d["out"], d["lse"], ws, stream)
            if ev is not None:
                ev[j][1].record(stream)

    for k in range(warmup):
        step(k)
    torch.cuda.synchronize()

    if calib > 0:
        n = calib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {calib} MiB done")
        del src, dst

    # timed region: whole steps
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(warmup, warmup + steps):
        step(k)
    torch.cuda.synchronize()
    t_total = time.perf_counter() - t_start
    us_per_step = t_total / steps * 1e6

    # same steps again with HIP events around the attention call (on its stream)
    evs = [[[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)] for _ in range(L)]
           for _ in range(steps)]
    torch.cuda.synchronize()
    for k in range(steps):
        step(warmup + k, evs[k])
    torch.cuda.synchronize()
    attn_ms = [e0.elapsed_time(e1) for row in evs for e0, e1 in row]
    attn_us = float(np.mean(attn_ms)) * 1e3
    p10, p50, p90 = (float(np.percentile(attn_ms, q)) * 1e3 for q in (10, 50, 90))
    log(f"[bench] step {us_per_step:.2f} us; attention call mean {attn_us:.2f} us (p10 {p10:.2f}, "
        f"p50 {p50:.2f}, p90 {p90:.2f})")
    del rotations, layer_sets
    torch.cuda.empty_cache()
    return {"work": work, "us_per_step": us_per_step, "attn_us": attn_us, "p10": p10, "p50": p50, "p90": p90,
            "n_rot": n_rot}


def advancing_batches(wl, n):
    """n device batches of the workload whose decode lengths grow by one token
    per step: step k uses decode prefixes p - (n - 1) + k (clipped at 0), where
    p are the workload's, so every appended slot lies inside the workload's
    block table and pool."""
    import torch

    import paper_2607_02043_amd as mla

    dev = torch.device("cuda:0")
    b = wl.batch
    dec = b.q_lens == 1
    batches = []
    for k in range(n):
        p = b.prefix_lens.astype(np.int64).copy()
        p[dec] = np.maximum(0, p[dec] - (n - 1) + k)
        batches.append(mla.DeviceBatch(b.q_lens, p.astype(np.int32), b.block_table, b.page_size, b.num_pages,
                                       device=dev))
    return batches


def host_plan_times(batches):
    """Host time of the checks and the planning per new batch (the workspace
    query plans the batch): every batch planned in full, then warm-started from
    the last full plan as a serving loop does.  Median and min over 5 passes."""
    import paper_2607_02043_amd as mla

    def plan_time(warm):
        mla.debug_set(mla.MLA_DEBUG_WARM_PLAN, 1 if warm else 0)
        try:
            reps = []
            for _ in range(5):  # every call meets a new batch: the exact-lengths cache never hits
                t = time.perf_counter()
                for db in batches:
                    mla.mixed_step_workspace_bytes(db)
                reps.append((time.perf_counter() - t) / len(batches) * 1e6)
        finally:
            mla.debug_set(mla.MLA_DEBUG_WARM_PLAN, -1)
        return {"median": round(float(np.median(reps)), 2), "min": round(float(np.min(reps)), 2)}

    return plan_time(False), plan_time(True)


def plan_inclusive(args, wl, steps, warmup):
    """Steps whose decode lengths grow by one token per step, as in serving:
    every step is a new batch, so the host plans every step (a plan is reused
    only across the layers of one step).  Step k of n uses decode prefixes
    p - (n - 1) + k (clipped at 0), where p are the workload's, so every
    appended slot lies inside the workload's block table and pool.  Reported:
    the wall time per step of the whole loop (host checks, planning and
    launches overlap the GPU work of the steps before) and the host time of
    the checks and the planning alone, per new batch: as served (warm-started
    from the last full plan) and with every batch planned in full."""
    batches = advancing_batches(wl, steps + warmup)
    cold, warm = host_plan_times(batches)
    m = measure(args, wl, steps, warmup, batches=batches)
    s = summary(wl, m)
    s["workload"] = wl.name + "; decode lengths +1 per step"
    s["host_plan_us"] = warm
    s["host_plan_full_us"] = cold
    log(f"[bench] plan-inclusive {wl.name[:40]}: {s['us_per_step']:.1f} us/step, host plan "
        f"{warm['median']:.1f} us warm, {cold['median']:.1f} us in full")
    return s


def cpu_baseline(wl, cfg, layer=False):
    """The fp64 oracle as it stands, timed on this host on a bounded sample."""
    import oracle
    from paper_2607_02043_amd import workloads as W
    if layer:
        return cpu_baseline_layer(wl)

    threads = len(os.sched_getaffinity(0))
    b = wl.batch
    li = wl.layer(0)
    work = algorithmic_work(b)
    total_pairs = work["pairs"]
    if total_pairs <= CPU_SAMPLE_PAIRS:
        rows = None
        sample = "one full layer step (append + every row)"
        frac = 1.0
    else:
        # a seeded sample of rows whose pairs add up to about 4M (several seconds of fp64 work per run)
        rng = np.random.default_rng(0)
        order = rng.permutation(b.num_rows)
        cu = b.cu_q
        req_of = np.searchsorted(cu, np.arange(b.num_rows), side="right") - 1
        pairs_of = b.prefix_lens[req_of].astype(np.int64) + (np.arange(b.num_rows) - cu[req_of]) + 1
        csum = np.cumsum(pairs_of[order])
        n = int(np.searchsorted(csum, CPU_SAMPLE_PAIRS)) + 1
        rows = np.sort(order[:n])
        frac = float(pairs_of[rows].sum()) / total_pairs
        sample = f"{len(rows)} seeded random rows ({frac * 100:.2f}% of one layer's query-key pairs), scaled up"
    times = []
    for _ in range(3):
        t = time.perf_counter()
        oracle.step(b, li, W.SOFTMAX_SCALE, rows=rows, threads=threads)
        times.append(time.perf_counter() - t)
    per_layer_s = float(np.median(times)) / frac
    value_us = per_layer_s * wl.num_layers * 1e6
    return {"value": round(value_us, 1), "unit": "us/step", "cores": threads, "kind": "oracle",
            "sample": sample + f"; median of 3; x{wl.num_layers} layer(s)",
            "cpu": _cpu_model()}


def cpu_baseline_layer(wl):
    """The layer oracle (numpy fp64 projections around the C attention
    oracle) on a bounded sample: the projections of a seeded sample of rows
    and the attention of those rows, scaled to the whole step."""
    from oracle import proj_oracle as PO
    from paper_2607_02043_amd import workloads as W

    threads = len(os.sched_getaffinity(0))
    b = wl.batch
    li = wl.layer(0)
    T = b.num_rows
    wo = PO.Weights.from_bits(W.make_proj_weights(wl.seed, 0))
    hidden = W.random_hidden(T, wl.seed, 0)
    rng = np.random.default_rng(0)
    n = min(T, 64)
    rows = np.sort(rng.choice(T, size=n, replace=False))
    pos = PO.positions(b.q_lens, b.prefix_lens)
    import oracle
    t_pre, t_rest = [], []
    for _ in range(3):
        t = time.perf_counter()
        # every row's projections (the attention needs all new latents), the sampled rows' attention and output
        q_abs, lat = PO.pre_attn(pos, PO.bf16_value(hidden), wo, rounded=True)
        t_pre.append(time.perf_counter() - t)
        t = time.perf_counter()
        pool_after = oracle.append(b, lat, li.pool)
        o, _ = oracle.attend(b, q_abs, pool_after, W.SOFTMAX_SCALE, rows=rows, threads=threads)
        PO.post_attn(o, wo, rounded=True)
        t_rest.append(time.perf_counter() - t)
    # projections before attention measured whole; attention + output projection scaled by the sampled pair share
    work = algorithmic_work(b)
    cu = b.cu_q
    req_of = np.searchsorted(cu, rows, side="right") - 1
    pairs = (b.prefix_lens[req_of].astype(np.int64) + (rows - cu[req_of]) + 1).sum()
    frac = min(1.0, float(pairs) / work["pairs"])
    per_layer_s = float(np.median(t_pre)) + float(np.median(t_rest)) / frac
    return {"value": round(per_layer_s * wl.num_layers * 1e6, 1), "unit": "us/step", "cores": threads,
            "kind": "oracle",
            "sample": f"projections of all {T} rows, then attention and output projection of {n} seeded rows "
                      f"({frac * 100:.2f}% of the query-key pairs) scaled by that share; median of 3; "
                      f"x{wl.num_layers} layer(s)",
            "cpu": _cpu_model()}


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


if __name__ == "__main__":
    main()
