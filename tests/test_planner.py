"""The host work planner (host code, no GPU): the real planner source is built
into a small harness and its plans are checked against the kernels' limits and
the mapping the device recomputes.

Checked for random ragged batches: the chunk item count and key split, the
decode unit size against the per-unit segment and page-window limits, the
number of units and items, the merge fan-out, the workspace layout (counter
block, then partial slots that fit every split row), and the planning time."""
import math
import os
import shutil
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "planner", "plan_harness.cpp")

KEYS_PER_TILE, BLOCK_TOKENS, MAX_SEG, PAGE_WINDOW = 32, 8, 64, 256
PARTIAL_FLOATS, PARTIAL_STATS, COUNTER_BYTES = 16 * 512, 16 * 2, 256


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    cxx = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(cxx):
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("planner") / "plan_harness")
    inc = [f"-I{os.path.join(ROOT, 'include')}", f"-I{os.path.join(ROOT, 'paper_2607_02043_amd', 'csrc')}"]
    subprocess.run([cxx, "-O2", "-std=c++17", *inc, SRC, "-o", exe], check=True, capture_output=True)
    return exe


def plan(exe, batches, route=None, chunk_keys=None, dec_unit=None, dec_first=None):
    text = "".join(f"{ncu} {P} {len(q)} " + " ".join(f"{a} {b}" for a, b in zip(q, p)) + "\n"
                   for ncu, P, q, p in batches)
    env = dict(os.environ)
    if route is not None:
        env["PLAN_ROUTE"] = f"{route[0]} {route[1]}"
    if chunk_keys is not None:
        env["PLAN_CHUNK_KEYS"] = str(chunk_keys)
    if dec_unit is not None:
        env["PLAN_DEC_UNIT"] = str(dec_unit)
    if dec_first is not None:
        env["PLAN_DEC_FIRST"] = str(dec_first)
    out = subprocess.run([exe], input=text, capture_output=True, text=True, check=True,
                         env=env).stdout.splitlines()
    assert len(out) == len(batches)
    res = []
    for line in out:
        f = line.split()
        if f[0] == "err":
            res.append(("err", int(f[1]), " ".join(f[2:])))
            continue
        keys = ["ks", "n_chunk_items", "n_dec_items", "U", "dec_total", "grid", "hsplit", "chunk_split",
                "dec_split", "bytes", "off_co", "off_cml", "off_do", "off_dml"]
        d = {k: int(v) for k, v in zip(keys, f[1:15])}
        d["us"], d["est"], d["first"] = float(f[15]), float(f[17]), int(f[18])
        res.append(d)
    return res


def random_batch(rng, ncu):
    P = int(rng.choice([1, 2, 16, 32, 64, 256]))
    n_dec = int(rng.integers(0, 300))
    n_chunk = int(rng.integers(0, 5)) if n_dec else int(rng.integers(1, 5))
    cap = 4096 if P >= 16 else 1024
    q = [1] * n_dec + [int(rng.integers(2, 2049)) for _ in range(n_chunk)]
    p = [int(rng.integers(0, cap)) for _ in range(n_dec)] + [int(rng.integers(0, 8193)) for _ in range(n_chunk)]
    perm = rng.permutation(len(q))
    return ncu, P, [q[i] for i in perm], [p[i] for i in perm]


def unit_limits(dec, U, P):
    """(max segments, max page-window entries) over the units of U tiles of
    the flattened decode tile list (dec: [(first_tile, tiles, p)])."""
    total = sum(t for _, t, _ in dec)
    worst_seg = worst_pages = 0
    for R0 in range(0, total, U):
        R1 = min(R0 + U, total)
        segs = pages = 0
        for first, tiles, p in dec:
            if first + tiles <= R0 or first >= R1:
                continue
            t0, t1 = max(R0 - first, 0), min(R1 - first, tiles)
            k0, klast = t0 * KEYS_PER_TILE, min(t1 * KEYS_PER_TILE, p + 1) - 1
            pages += klast // P - k0 // P + 1
            segs += 1
        worst_seg, worst_pages = max(worst_seg, segs), max(worst_pages, pages)
    return worst_seg, worst_pages


def multi_head(route, p, c):
    """The layer's route of a chunk request (c rows at prefix p) to the
    multi-head path: at least min_rows rows and c (p + c/2) / (p + c) query-key
    pairs per key reaching pair_keys."""
    return route is not None and c >= route[0] and c * (2 * p + c) >= 2 * route[1] * (p + c)


def check_plan(batch, d, route=None):
    ncu, P, q, p = batch
    chunks = [(pi, qi) for qi, pi in zip(q, p) if qi > 1 and not multi_head(route, pi, qi)]
    dec, first = [], 0
    for qi, pi in zip(q, p):
        if qi == 1:
            nt = -(-(pi + 1) // KEYS_PER_TILE)
            dec.append((first, nt, pi))
            first += nt
    ks = d["ks"]
    # chunk items: ceil(c / 8) blocks x ceil((p + c) / ks) key splits per request
    assert d["n_chunk_items"] == sum(-(-c // BLOCK_TOKENS) * -(-(pp + c) // ks) for pp, c in chunks)
    assert d["chunk_split"] == int(any(pp + c > ks for pp, c in chunks))
    if chunks:
        assert ks % 64 == 0 and ks >= 64
        assert ks <= max(64, (PAGE_WINDOW - 1) * P // 64 * 64)  # an item's keys fit the page window
    assert d["dec_total"] == first
    if dec:
        U = d["U"]
        assert 1 <= U <= first
        units = -(-first // U)
        assert d["n_dec_items"] == -(-units // 2)
        seg, pages = unit_limits(dec, U, P)
        assert seg <= MAX_SEG and pages <= PAGE_WINDOW
        parts = max((f + t - 1) // U - f // U + 1 for f, t, _ in dec)
        assert d["dec_split"] == int(parts > 1)
        assert d["hsplit"] == (8 if parts > 16 else 4 if parts > 4 else 1)
    else:
        units = 0
        assert d["n_dec_items"] == 0 and d["dec_split"] == 0
    assert 1 <= d["grid"] <= ncu and d["grid"] <= d["n_chunk_items"] + d["n_dec_items"]
    # decode-first workgroups: only with both kinds of work, at most the launch
    assert 0 <= d["first"] <= d["grid"]
    if d["n_chunk_items"] == 0 or d["n_dec_items"] == 0:
        assert d["first"] == 0
    # workspace: counters, then 256-byte aligned partial slots
    off = COUNTER_BYTES
    align = lambda v: (v + 255) // 256 * 256
    if d["chunk_split"]:
        assert d["off_co"] == off
        off = align(off + d["n_chunk_items"] * BLOCK_TOKENS * PARTIAL_FLOATS * 4)
        assert d["off_cml"] == off
        off = align(off + d["n_chunk_items"] * BLOCK_TOKENS * PARTIAL_STATS * 4)
    if d["dec_split"]:
        assert d["off_do"] == off
        off = align(off + 2 * units * PARTIAL_FLOATS * 4)
        assert d["off_dml"] == off
        off = align(off + 2 * units * PARTIAL_STATS * 4)
    assert d["bytes"] == off


def test_plans_of_random_batches_respect_the_kernel_limits(harness):
    rng = np.random.default_rng(7)
    batches = [random_batch(rng, int(rng.choice([64, 256, 304]))) for _ in range(60)]
    for b, d in zip(batches, plan(harness, batches)):
        assert not isinstance(d, tuple), (b[:2], d)
        check_plan(b, d)


def test_plans_of_the_benchmark_workloads(harness):
    from paper_2607_02043_amd import workloads as W
    wls = [W.config(1), W.config(2), W.config(3), W.config(4, chunk=0), W.config(4, chunk=2048), W.config(5)]
    batches = [(256, w.batch.page_size, [int(x) for x in w.batch.q_lens], [int(x) for x in w.batch.prefix_lens])
               for w in wls]
    reps = 15
    res = plan(harness, [b for b in batches for _ in range(reps)])
    for i, b in enumerate(batches):
        runs = res[i * reps:(i + 1) * reps]
        check_plan(b, runs[0])
        assert all({k: v for k, v in d.items() if k != "us"} == {k: v for k, v in runs[0].items() if k != "us"}
                   for d in runs), "the planner is not deterministic"
        # a full plan (a batch shape not seen before) takes some 5-25 us on
        # one core of a current server CPU; the bound leaves room for a busy
        # or slower host
        us = float(np.median([d["us"] for d in runs]))
        assert us < 150.0, (i, us)
    res = res[::reps]
    # decode-only: one item of two equal units per CU
    assert res[3]["n_chunk_items"] == 0 and res[3]["n_dec_items"] == 256
    # the 2048-token chunk beside 256 long decode rows streams the decode work
    # beside the chunk from the start, one decode item per decode-first
    # workgroup; workload 3 (whose launch its longest chunk item bounds) keeps
    # the chunk-first schedule
    assert res[4]["first"] > 0 and res[4]["n_dec_items"] == res[4]["first"]
    assert res[2]["first"] == 0


@pytest.mark.parametrize("first", [0, 1, 96, 100000])
def test_forced_decode_first_workgroups(harness, first):
    """The debug knob fixes the decode-first workgroups (0: none), capped by
    the launch; without both kinds of work there are none.  The plan still
    respects every limit."""
    rng = np.random.default_rng(first % 1000 + 7)
    batches = [random_batch(rng, 256) for _ in range(40)]
    for batch, d in zip(batches, plan(harness, batches, dec_first=first)):
        check_plan(batch, d)
        if d["n_chunk_items"] > 0 and d["n_dec_items"] > 0:
            assert d["first"] == min(first, d["grid"])


def test_single_request_extremes(harness):
    cases = [(256, 64, [1], [0]), (256, 1, [1], [0]), (256, 64, [2], [0]), (256, 16, [1], [1 << 20]),
             (256, 64, [4096], [1 << 16]), (1, 64, [1, 1, 300], [5, 70, 1000])]
    for b, d in zip(cases, plan(harness, cases)):
        check_plan(b, d)


@pytest.mark.parametrize("route", [(256, 1200), (2, 100), (2, 0)])
def test_plan_leaves_out_routed_chunks(harness, route):
    """Chunk requests that the layer sends to the multi-head path get no work
    items; the rest of the plan is that of the remaining requests."""
    rng = np.random.default_rng(7)
    batches = [random_batch(rng, int(rng.choice([80, 256]))) for _ in range(40)]
    batches.append((256, 64, [1] * 128 + [2048], list(rng.integers(0, 4096, 128)) + [6144]))
    batches.append((256, 64, [1500], [0]))  # the only request leaves: nothing to plan
    res = plan(harness, batches, route)
    for b, d in zip(batches, res):
        assert not isinstance(d, tuple), (b[:2], d)
        ncu, P, q, p = b
        if all(qi > 1 and multi_head(route, pi, qi) for qi, pi in zip(q, p)):
            assert d["n_chunk_items"] == 0 and d["n_dec_items"] == 0 and d["grid"] == 0, d
            continue
        check_plan(b, d, route)
    # the benchmark's 2048-row chunk over 6144 keys leaves on every route here
    assert res[-2]["n_chunk_items"] == 0 and res[-2]["n_dec_items"] > 0


def test_workspace_too_small_is_rejected(harness):
    """The real mixed_step_attn entry point (launches stubbed) rejects a
    workspace below what the batch needs with MLA_ERR_WORKSPACE before
    launching anything, and accepts the exact size."""
    q = [1] * 40 + [700]
    p = [int(x) for x in np.random.default_rng(2).integers(100, 9000, 40)] + [3000]
    line = " ".join(f"{a} {b}" for a, b in zip(q, p))
    out = subprocess.run([harness], input=f"ws 0 64 {len(q)} {line}\n", capture_output=True, text=True,
                         check=True).stdout.split()
    assert out[0] == "rc"
    need = int(out[2])
    assert need > 256
    assert int(out[1]) == -3  # MLA_ERR_WORKSPACE
    text = "".join(f"ws {n} 64 {len(q)} {line}\n" for n in (need - 16, need))
    lines = subprocess.run([harness], input=text, capture_output=True, text=True, check=True).stdout.splitlines()
    small, exact = lines[0].split(), lines[1].split()
    assert int(small[1]) == -3 and "needs" in lines[0]
    assert int(exact[1]) == 0


def test_noalloc_entry_rejects_batches_beyond_its_scratch(harness):
    """mixed_step_noalloc plans like mixed_step; a batch whose workspace
    exceeds the library's fixed scratch (128 MiB) is rejected with
    MLA_ERR_WORKSPACE and a message naming the limit, before any launch."""
    big = "na 0 64 1 8192 57344\n"
    small = "na 0 64 2 1 500 64 0\n"
    lines = subprocess.run([harness], input=big + small, capture_output=True, text=True, check=True).stdout.splitlines()
    b, s = lines[0].split(), lines[1].split()
    assert int(b[2]) > 128 << 20 and int(b[1]) == -3 and "no-allocation" in lines[0]
    assert int(s[2]) <= 128 << 20 and int(s[1]) == 0


@pytest.mark.parametrize("keys", [64, 320, 4096])
def test_forced_chunk_key_split(harness, keys):
    """The debug knob fixes the chunk key split (capped by the page window);
    the plan still respects every kernel limit."""
    rng = np.random.default_rng(keys)
    batches = [random_batch(rng, 256) for _ in range(40)]
    for batch, d in zip(batches, plan(harness, batches, chunk_keys=keys)):
        check_plan(batch, d)
        ncu, P, q, p = batch
        if any(qi > 1 for qi in q):
            assert d["ks"] == min(keys, max(64, (PAGE_WINDOW - 1) * P // 64 * 64))


@pytest.mark.parametrize("unit", [1, 3, 40, 100000])
def test_forced_decode_unit(harness, unit):
    """The debug knob fixes the decode unit size, made smaller only as far as
    the kernel's segment and page-window limits require; the plan still
    respects every limit."""
    rng = np.random.default_rng(unit)
    batches = [random_batch(rng, 256) for _ in range(40)]
    reduced = 0
    for batch, d in zip(batches, plan(harness, batches, dec_unit=unit)):
        check_plan(batch, d)
        if d["dec_total"] > 0:
            assert 1 <= d["U"] <= min(unit, d["dec_total"])
            reduced += d["U"] < min(unit, d["dec_total"])
    if unit <= 3:
        assert reduced == 0  # units this small always fit


def _serving_plans(harness, batches):
    env = dict(os.environ, PLAN_SERVING="1")
    text = "".join(f"256 {P} {len(q)} " + " ".join(f"{a} {b}" for a, b in zip(q, p)) + "\n" for _, P, q, p in batches)
    out = subprocess.run([harness], input=text, capture_output=True, text=True, check=True, env=env).stdout
    res = []
    for line in out.splitlines():
        f = line.split()
        assert f[0] == "ok", line
        keys = ["ks", "n_chunk_items", "n_dec_items", "U", "dec_total", "grid", "hsplit", "chunk_split",
                "dec_split", "bytes", "off_co", "off_cml", "off_do", "off_dml"]
        d = {k: int(v) for k, v in zip(keys, f[1:15])}
        d["us"], d["warm"], d["first"] = float(f[15]), int(f[16]), int(f[18])
        res.append(d)
    assert len(res) == len(batches)
    return res


def test_serving_sequence_plans_warm_and_stays_valid(harness):
    """A decode node's consecutive steps: decode lengths grow by one token,
    a request leaves and one joins now and then, the chunk moves on.  Steps
    close to the last full plan reuse its key split and unit size; every plan
    still respects the kernel limits, and a warm plan costs a few
    microseconds."""
    rng = np.random.default_rng(11)
    dec = list(rng.integers(2000, 12000, 64))
    chunk_p, chunk_c = 8192, 2048
    batches = []
    for step in range(60):
        dec = [d + 1 for d in dec]
        if step % 7 == 6:  # one request finishes, another joins
            dec = dec[1:] + [int(rng.integers(2000, 12000))]
        if step == 40:  # the chunk request moves to its next chunk: more keys
            chunk_p += chunk_c
        q = [1] * len(dec) + [chunk_c]
        p = dec + [chunk_p]
        batches.append((256, 64, q, p))
    batches.append((256, 64, [1] * 8, list(rng.integers(100, 200, 8))))  # a different batch: planned in full
    plans = _serving_plans(harness, batches)
    for batch, d in zip(batches, plans):
        check_plan(batch, d)
    assert plans[0]["warm"] == 0 and plans[-1]["warm"] == 0
    warm = [d for d in plans[1:40] if d["warm"]]
    assert len(warm) >= 30
    anchor = None  # a warm plan keeps the key split, unit size and decode-first workgroups of the last full plan
    for d in plans:
        if d["warm"]:
            assert (d["ks"], d["U"]) == anchor[:2]
            if d["n_chunk_items"] > 0 and d["n_dec_items"] > 0:
                assert d["first"] == min(anchor[2], d["grid"])
        else:
            anchor = (d["ks"], d["U"], d["first"])
    assert float(np.median([d["us"] for d in warm])) < 50.0


@pytest.mark.parametrize("seed", [1, 2])
def test_cost_model_matches_brute_force(harness, seed):
    """The planner's queue model against one-at-a-time scheduling on random
    workgroup loads: the chunk-queue simulation gives the same loads, the
    decode fill the same finishing time, and both of its lower bounds (the
    water level, the per-workgroup bound) stay at or below it."""
    out = subprocess.run([harness], input=f"cm {seed} 1500\n", capture_output=True, text=True,
                         check=True).stdout.split()
    assert out == ["cm", "ok", "1500"], out

