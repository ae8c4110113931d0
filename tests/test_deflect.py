"""Step-latency model, chunk schedule and deflection decision (sections
4.3.1-4.4, Eqs. 1-7, Algorithm 1): the reference in oracle/deflect_oracle.py
pinned by exact-data recovery, hand-checked equations and the greedy rule
checked step by step from its definition; the package's implementation against the reference; the fit against
the measured MI355X steps (held-out MAPE, the paper's bar is < 10 %)."""
import csv
import math
import os
import time

import numpy as np
import pytest

from oracle import deflect_oracle as O
from paper_2607_02043_amd import deflect as D

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
MEASURED = os.path.join(ROOT, "profiles", "step_latency_mi355x.csv")
CANDS = [2048, 1024, 512, 256, 128]


def measured_rows():
    with open(MEASURED) as fh:
        return [(int(r["B"]), int(r["K"]), int(r["c"]), int(r["p"]), float(r["us"])) for r in csv.DictReader(fh)]


def as_oracle(model: D.StepModel):
    return (list(map(float, model.dec)), list(map(float, model.mix)), list(map(float, model.prefill)))


# ------------------------------------------------------------ oracle pins
def test_oracle_fit_recovers_an_exact_linear_model():
    a, b, e = [25.0, 0.1, 3e-4, 0.02], [0.05, 3e-5, -1e-6, -5e-8], [50.0, 4e-3, 3e-5, 1e-5]
    rows = []
    for B in (4, 16, 64):
        for Kr in (500, 4000, 12000, 30000):
            K = B * Kr
            t0 = a[0] + a[1] * B + a[2] * K + a[3] * math.sqrt(K)
            rows.append((B, Kr, 0, 0, t0))
            for c in (100, 500, 1900):
                for p in (0, c, 3 * c):
                    d = b[0] * c + b[1] * c * p + b[2] * c * c + b[3] * c * K
                    if d > 0:  # the fit sees the linear part only where it is not clipped
                        rows.append((B, Kr, c, p, t0 + d))
    for chi in (512, 2048, 8192):
        for i in range(4):
            rows.append((0, 0, chi, chi * i, e[0] + e[1] * chi + e[2] * chi * chi * i + e[3] * chi * chi))
    fa, fb, fe = O.fit(rows)
    for got, want in ((fa, a), (fb, b), (fe, e)):
        for g, w in zip(got, want):
            assert abs(g - w) <= 1e-7 * abs(w), (got, want)


def test_oracle_relative_error_weighting_closed_form():
    # a constant fitted to 1, 2, 4 on relative error: argmin sum((w - y)/y)^2 =
    # sum(1/y) / sum(1/y^2) = 1.75 / 1.3125 = 4/3
    w = O.solve_least_squares([[1.0], [1.0], [1.0]], [1.0, 2.0, 4.0], [1.0, 0.25, 0.0625])
    assert abs(w[0] - 4.0 / 3.0) < 1e-12
    # and a line through three points is exact whatever the weights
    w = O.solve_least_squares([[1.0, 0.0], [1.0, 1.0], [1.0, 2.0]], [1.0, 3.0, 5.0], [1.0, 0.1, 0.01])
    assert abs(w[0] - 1.0) < 1e-12 and abs(w[1] - 2.0) < 1e-12


def test_oracle_step_and_prefill_equations_by_hand():
    model = ([10.0, 1.0, 0.01, 0.5], [2.0, 0.001, 0.0, 0.0], [5.0, 1.0, 0.5, 0.25])
    assert O.t_step(model, 4, 1024, 0, 0) == 10.0 + 4.0 + 10.24 + 16.0
    assert O.t_step(model, 4, 1024, 100, 50) == 40.24 + 100.0 + 5.0
    neg = ([10.0, 0.0, 0.0, 0.0], [-1.0, 0.0, 0.0, 0.0], [0.0] * 4)
    assert O.t_step(neg, 1, 0, 0, 30) == 10.0  # a chunk never shortens a step
    # Eq. 2: 300 queued tokens at chi_p 100 = 3 chunks of T(100, 150)
    assert O.queue_wait(model, [100, 200], 100) == 3 * (5.0 + 100 + 0.5 * 100 * 150 + 0.25 * 100 * 100)
    # Eq. 3: 250 tokens = chunks of 100 (prefix 0), 100 (prefix 100), 50 (prefix 200)
    want = sum(5.0 + c + 0.5 * c * q + 0.25 * c * c for c, q in ((100, 0), (100, 100), (50, 200)))
    assert O.prefill_exec(model, 250, 100) == want


def test_oracle_schedule_is_stepwise_largest_safe():
    """Eq. 5's greedy rule, checked step by step from its definition: every
    step is TBT-safe, no larger candidate was safe at that step, the prompt is
    served exactly; and an infeasible answer comes with a prefix at which no
    candidate is safe."""
    rng = np.random.default_rng(3)
    cands = [40, 24, 16, 10]
    n_ok = n_none = 0
    for _ in range(200):
        model = ([float(rng.uniform(5, 20)), 0.5, 1e-3, 0.01],
                 [float(rng.uniform(0, 0.2)), float(rng.uniform(0, 0.02)), float(rng.uniform(-1e-3, 1e-3)), 0.0],
                 [0.0] * 4)
        B, K = int(rng.integers(2, 8)), int(rng.integers(100, 2000))
        prompt = int(rng.integers(5, 90))
        limit = O.t_step(model, B, K, 0, 0) + float(rng.uniform(0.5, 8))
        s = O.chunk_schedule(model, B, K, prompt, cands, limit)
        served = 0
        steps = zip(s[0], s[1]) if s is not None else []
        for chi, c in steps:
            left = prompt - served
            assert c == min(chi - B, left)
            assert O.t_step(model, B, K, served, c) <= limit
            for big in cands:
                if big > chi and big - B > 0:
                    assert O.t_step(model, B, K, served, min(big - B, left)) > limit
            served += c
        if s is None:
            n_none += 1
            # replay the greedy to the prefix where it stopped: nothing is safe there
            served = 0
            while True:
                left = prompt - served
                safe = [chi for chi in cands
                        if chi - B > 0 and O.t_step(model, B, K, served, min(chi - B, left)) <= limit]
                if not safe:
                    break
                served += min(max(safe) - B, left)
                assert served < prompt
        else:
            n_ok += 1
            assert served == prompt and abs(s[2] - sum(
                O.t_step(model, B, K, sum(s[1][:i]), c) for i, c in enumerate(s[1]))) < 1e-9 * s[2]
    assert n_ok > 20 and n_none > 5


def test_oracle_schedule_by_hand():
    # T0 = 10, dT = 0.01 c p: with limit 20 a chunk of c tokens is safe while c p <= 1000
    model = ([10.0, 0.0, 0.0, 0.0], [0.0, 0.01, 0.0, 0.0], [0.0] * 4)
    s = O.chunk_schedule(model, 0, 0, 100, [50, 20, 10], 20.0)
    # p=0: 50 (0 <= 1000); p=50: 50*50=2500 > 1000, 20*50=1000 ok -> 20; p=70: 20*70 > 1000,
    # 10*70=700 -> 10; p=80: 20 left, 20*80 > 1000, 10*80=800 -> 10; p=90: 10 left, so every
    # candidate carries 10 tokens (900 <= 1000) and the largest, 50, is taken; p=100 done
    assert s[0] == [50, 20, 10, 10, 50] and s[1] == [50, 20, 10, 10, 10]
    assert s[2] == 10.0 + (10 + 0.01 * 20 * 50) + (10 + 0.01 * 10 * 70) + (10 + 0.01 * 10 * 80) + \
        (10 + 0.01 * 10 * 90)


def test_oracle_decision_rules():
    model = ([10.0, 0.0, 0.0, 0.0], [0.01, 0.0, 0.0, 0.0], [1.0, 0.01, 0.0, 0.0])
    # no node can host any chunk: tau below the decode-only step
    assert O.decide(model, 100, [0], 100, [(4, 0)], [64], tau=5.0)[0] is False
    d = O.decide(model, 100, [10000], 100, [(4, 0), (2, 0)], [64, 32], tau=100.0)
    assert d[0] is True and d[1] in (0, 1)
    # the SLO condition of Eq. 7 alone can refuse
    assert O.decide(model, 100, [10000], 100, [(4, 0)], [64], tau=100.0, ttft_slo=1.0)[0] is False


# ----------------------------------------------- package against the oracle
def test_fit_matches_the_oracle_on_the_measured_steps():
    rows = measured_rows()
    m = D.StepModel.fit(rows)
    om = O.fit(rows)
    for B, Kr, c, p, t in rows[::7]:
        if B > 0:
            got, want = float(m.step(B, B * Kr, p, c)), O.t_step(om, B, B * Kr, p, c)
        else:
            got, want = float(m.prefill_step(c, p)), O.t_prefill(om, c, p)
        assert abs(got - want) <= 1e-6 * abs(want), (B, Kr, c, p, got, want)


def random_models(n, seed=5):
    base = D.StepModel.fit(measured_rows())
    rng = np.random.default_rng(seed)
    for _ in range(n):
        yield D.StepModel(base.dec * rng.uniform(0.7, 1.3, 4), base.mix * rng.uniform(0.5, 1.5, 4),
                          base.prefill * rng.uniform(0.7, 1.3, 4))


def test_schedules_and_decisions_match_the_oracle():
    rng = np.random.default_rng(11)
    n_sched = 0
    for model in random_models(40):
        om = as_oracle(model)
        for _ in range(6):
            B = int(rng.integers(1, 200))
            K = B * int(rng.integers(200, 16000))
            prompt = int(rng.integers(1, 40000))
            tau = float(model.t0(B, K)) * float(rng.uniform(0.9, 3.0))
            cands = sorted(set(int(x) for x in rng.choice([64, 128, 256, 384, 512, 1024, 2048, 4096], 4)),
                           reverse=True)
            s = D.chunk_schedule(model, B, K, prompt, cands, tau)
            o = O.chunk_schedule(om, B, K, prompt, cands, tau)
            if o is None:
                assert s is None
                continue
            n_sched += 1
            assert s is not None and s.chunks == o[0] and s.tokens == o[1]
            assert abs(s.ttft - o[2]) <= 1e-9 * o[2]
        nodes = [(int(b), int(b) * int(k)) for b, k in zip(rng.integers(1, 200, 6), rng.integers(200, 16000, 6))]
        queue = [int(x) for x in rng.integers(0, 20000, int(rng.integers(0, 5)))]
        prompt = int(rng.integers(1, 30000))
        tau = float(np.median([float(model.t0(b, k)) for b, k in nodes])) * 1.5
        got = D.decide(model, prompt, queue, 2048, nodes, CANDS, tau)
        want = O.decide(om, prompt, queue, 2048, nodes, CANDS, tau)
        assert (got.deflect, got.node) == (want[0], want[1])
        assert abs(got.ttft_pf - want[3]) <= 1e-9 * want[3]
        if math.isfinite(want[4]):
            assert abs(got.ttft_dec - want[4]) <= 1e-9 * want[4]
        if got.deflect:
            assert got.schedule.chunks == want[2]
    assert n_sched > 100


# ------------------------------------------------------------- measurement
def test_held_out_mape_on_mi355x_steps():
    """Fit on 75 % of the measured steps, predict the rest; and leave one of
    the paper's context lengths out entirely."""
    rows = measured_rows()
    rng = np.random.default_rng(0)
    errs = []
    for rep in range(10):
        idx = rng.permutation(len(rows))
        n = len(rows) // 4
        m = D.StepModel.fit([rows[i] for i in idx[n:]])
        errs.append(D.mape(m, [rows[i] for i in idx[:n] if rows[i][0] > 0]))
    assert float(np.mean(errs)) < 0.10, errs
    # a harder extrapolation: one context length never seen by the fit
    m = D.StepModel.fit([r for r in rows if r[1] != 3569])
    assert D.mape(m, [r for r in rows if r[1] == 3569 and r[0] > 0]) < 0.12


def test_committed_model_is_the_fit_of_the_committed_steps():
    m = D.StepModel.load()
    f = D.StepModel.fit(measured_rows())
    for x, y in ((m.dec, f.dec), (m.mix, f.mix), (m.prefill, f.prefill)):
        assert np.allclose(x, y, rtol=1e-9, atol=0)


def test_decision_time_per_request():
    """Algorithm 1 for one request over 8 decode nodes on one CPU core (the
    paper reports < 1 ms); bounded loosely here, the figure goes to the notes."""
    m = D.StepModel.load()
    rng = np.random.default_rng(2)
    nodes = [(int(b), int(b) * int(k)) for b, k in zip(rng.integers(4, 128, 8), rng.integers(800, 14000, 8))]
    D.decide(m, 8192, [3000, 12000], 2048, nodes, CANDS, tau=600.0)
    t = time.perf_counter()
    for _ in range(50):
        D.decide(m, 8192, [3000, 12000], 2048, nodes, CANDS, tau=600.0)
    per = (time.perf_counter() - t) / 50
    assert per < 5e-3, per
