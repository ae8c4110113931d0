"""Step-latency model, TBT-safe chunk schedule and deflection decision of the
paper, fitted to measured steps of this library.

* Step-latency model (section 4.3.1, Eq. 4; the linear estimators of section
  5.2): T_step = T0(B, K) + dT_pf, where T0 is the decode-only step of B
  decode rows over K cached decode tokens and dT_pf the increase from a
  prefill chunk of c = chi - B tokens whose own cached prefix is p.  Both
  terms are linear regressions on the step's counts:
      T0    = a0 + a1 B + a2 K + a3 sqrt(K)
      dT_pf = b1 c + b2 c p + b3 c^2 + b4 c K        (0 when c = 0)
  fitted by least squares on relative error (so the fit targets MAPE); the
  sqrt(K) term bends T0 from latency-bound small batches to the HBM-bound
  rate of large ones.  A
  chunk never makes a step faster, so dT_pf is taken as max(0, fit).  The
  prefill-node step (Eq. 3) is a third regression of a pure chunk:
      T_pf_step(chi_p, cached) = e0 + e1 chi_p + e2 chi_p cached + e3 chi_p^2.
* Chunk schedule (section 4.3.2, Eqs. 5-6): greedily, at each step the largest
  candidate chi whose predicted step stays within beta * tau given the decode
  node's state and the chunks already served; its TTFT estimate is the sum of
  the predicted steps.
* Deflection decision (section 4.4, Algorithm 1 with Eqs. 1-3 and 7).

Readings (the paper leaves these open):
  * Eq. 5 passes K_n + sum_{j<i} chi^(j) as one "cached tokens" argument;
    here the two parts are kept apart (decode cache K_n; the deflected
    request's own cached chunks p), because on this GPU the first costs HBM
    time per key and the second matrix time per (token, key) pair.
  * A step of chi tokens carries chi - B_n prefill tokens (Eq. 4's text), so
    a chunk advances the served count and p by chi - B_n (Algorithm 1 adds
    chi); the last chunk carries only what is left of the prompt.
  * Eq. 3 sums ceil(l / chi_p) chunk steps, chunk i at prefix chi_p i, the
    last one with the remaining tokens.
  * Times are in the unit of the measurements the model is fitted to (us of
    one layer's attention step here); tau and the TTFT SLO use the same unit.
"""
from __future__ import annotations

import dataclasses
import json
import math
import os
from typing import List, Optional, Sequence, Tuple

import numpy as np

MODEL_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "step_model_mi355x.json")


def _dec_features(B, K):
    B = np.asarray(B, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64) + 0 * B
    return np.stack([np.ones_like(B), B, K, np.sqrt(K)], axis=-1)


def _pf_features(B, K, p, c):
    c = np.asarray(c, dtype=np.float64)
    p = np.asarray(p, dtype=np.float64) + 0 * c
    K = np.asarray(K, dtype=np.float64) + 0 * c
    return np.stack([c, c * p, c * c, c * K], axis=-1)


def _prefill_features(chi, cached):
    chi = np.asarray(chi, dtype=np.float64)
    cached = np.asarray(cached, dtype=np.float64) + 0 * chi
    return np.stack([np.ones_like(chi), chi, chi * cached, chi * chi], axis=-1)


def _fit_relative(X, y):
    """Least squares on relative residuals (rows weighted by 1 / y)."""
    w = 1.0 / y
    coef, *_ = np.linalg.lstsq(X * w[:, None], y * w, rcond=None)
    return coef


@dataclasses.dataclass
class StepModel:
    dec: np.ndarray      # a0, a1, a2, a3
    mix: np.ndarray      # b1, b2, b3, b4
    prefill: np.ndarray  # e0, e1, e2, e3

    # ------------------------------------------------------------- predict
    def t0(self, B, K):
        """Decode-only step: B decode rows over K cached decode tokens."""
        return _dec_features(B, K) @ self.dec

    def step(self, B, K, p, c):
        """Mixed step (Eq. 4): B decode rows over K cached tokens plus a chunk
        of c prefill tokens after p cached tokens of its own."""
        c_arr = np.asarray(c, dtype=np.float64)
        return self.t0(B, K) + np.where(c_arr > 0, np.maximum(0.0, _pf_features(B, K, p, c) @ self.mix), 0.0)

    def prefill_step(self, chi, cached):
        """Prefill-node step of chi tokens after `cached` tokens of the prompt."""
        return _prefill_features(chi, cached) @ self.prefill

    # ----------------------------------------------------------------- fit
    @classmethod
    def fit(cls, rows) -> "StepModel":
        """rows: (B, K_per_request, c, p, us) of measured steps; B = 0 rows are
        prefill-node steps (c tokens after p cached)."""
        r = np.asarray(rows, dtype=np.float64)
        B, Kr, c, p, y = r.T
        K = B * Kr
        dec_rows = (B > 0) & (c == 0)
        mix_rows = (B > 0) & (c > 0)
        pf_rows = B == 0
        a = _fit_relative(_dec_features(B[dec_rows], K[dec_rows]), y[dec_rows])
        resid = y[mix_rows] - _dec_features(B[mix_rows], K[mix_rows]) @ a
        Xm = _pf_features(B[mix_rows], K[mix_rows], p[mix_rows], c[mix_rows])
        wm = 1.0 / y[mix_rows]
        b, *_ = np.linalg.lstsq(Xm * wm[:, None], resid * wm, rcond=None)
        e = _fit_relative(_prefill_features(c[pf_rows], p[pf_rows]), y[pf_rows]) if pf_rows.any() \
            else np.zeros(4)
        return cls(a, b, e)

    def to_json(self) -> str:
        return json.dumps({"dec": list(map(float, self.dec)), "mix": list(map(float, self.mix)),
                           "prefill": list(map(float, self.prefill))}, indent=1)

    @classmethod
    def from_json(cls, text: str) -> "StepModel":
        d = json.loads(text)
        return cls(np.array(d["dec"]), np.array(d["mix"]), np.array(d["prefill"]))

    @classmethod
    def load(cls, path: str = MODEL_PATH) -> "StepModel":
        with open(path) as fh:
            return cls.from_json(fh.read())


def mape(model: StepModel, rows) -> float:
    """Mean absolute percentage error of the model over measured rows."""
    r = np.asarray(rows, dtype=np.float64)
    B, Kr, c, p, y = r.T
    pred = np.where(B > 0, model.step(B, B * Kr, p, c), model.prefill_step(c, p))
    return float(np.mean(np.abs(pred - y) / y))


# ------------------------------------------------------------ chunk schedule
@dataclasses.dataclass
class Schedule:
    chunks: List[int]       # chi of each step
    tokens: List[int]       # prefill tokens each step carries
    ttft: float             # Eq. 6: sum of the predicted steps


class _Node:
    """A decode node's fixed part of every step's prediction: for candidate
    chi (c = chi - B prefill tokens) the step after p cached prompt tokens is
    t0 + max(0, u_c + v_c p) with v_c = b2 c >= 0, so each candidate is safe
    exactly up to a prefix bound."""

    def __init__(self, model: StepModel, B: int, K: int, cands: Sequence[int], limit: float):
        self.model, self.B, self.K = model, B, K
        self.t0 = float(model.t0(B, K))
        b1, b2, b3, b4 = (float(x) for x in model.mix)
        self.b = (b1, b2, b3, b4)
        self.cands = []  # (chi, c, u, v, max safe prefix), chi descending
        for chi in sorted(set(int(x) for x in cands), reverse=True):
            c = chi - B
            if c <= 0:
                continue
            u = b1 * c + b3 * c * c + b4 * c * K
            v = b2 * c
            room = limit - self.t0
            if room < 0:
                pmax = -1.0
            elif v > 0:
                pmax = (room - u) / v
            else:
                pmax = math.inf if u <= room else -1.0
            self.cands.append((chi, c, u, v, pmax))

    def step(self, c: int, p: int) -> float:
        b1, b2, b3, b4 = self.b
        return self.t0 + max(0.0, b1 * c + b2 * c * p + b3 * c * c + b4 * c * self.K)


def largest_safe(model: StepModel, B: int, K: int, p: int, cands: Sequence[int], limit: float) -> int:
    """LargestSafe: the largest chi in cands whose step (chi - B prefill tokens
    after p cached ones) is predicted within `limit`; 0 if none is."""
    for chi, c, u, v, pmax in _Node(model, B, K, cands, limit).cands:
        if p <= pmax:
            return chi
    return 0


def chunk_schedule(model: StepModel, B: int, K: int, prompt: int, cands: Sequence[int], tau: float,
                   beta: float = 1.0) -> Optional[Schedule]:
    """Greedy TBT-safe schedule for a prompt of `prompt` tokens on a decode
    node with B decode rows over K cached tokens (Eq. 5); None if infeasible.

    A step of candidate chi carries min(chi - B, tokens left) prompt tokens;
    the largest candidate whose step is predicted safe is taken.  Runs of
    equal full chunks are taken at once: a full candidate is safe exactly up
    to its prefix bound, and a larger candidate cannot turn safe while it is
    still full (its bound was already passed), so a run ends at the bound or
    when the largest candidate would no longer be full."""
    limit = beta * tau
    node = _Node(model, B, K, cands, limit)
    if not node.cands:
        return None
    c_top = node.cands[0][1]
    served, ttft = 0, 0.0
    chunks: List[int] = []
    tokens: List[int] = []
    while served < prompt:
        left = prompt - served
        pick = None
        for chi, c, u, v, pmax in node.cands:
            if c >= left:  # carries what is left: evaluate that step
                if node.step(left, served) <= limit:
                    pick = (chi, left, None)
                    break
            elif served <= pmax:
                pick = (chi, c, (u, v, pmax))
                break
        if pick is None:
            return None
        chi, c, full = pick
        if full is None:  # last step
            chunks.append(chi)
            tokens.append(c)
            ttft += node.step(c, served)
            break
        u, v, pmax = full
        n = left // c if math.isinf(pmax) else min(math.floor((pmax - served) / c) + 1, left // c)
        if c < c_top:  # every larger candidate must stay full (left >= its chunk) for the whole run
            n = min(n, max(1, (left - c_top) // c + 1))
        n = max(int(n), 1)
        ps = served + c * np.arange(n, dtype=np.float64)
        ttft += float(np.sum(node.t0 + np.maximum(0.0, u + v * ps)))
        chunks += [chi] * n
        tokens += [c] * n
        served += n * c
    return Schedule(chunks, tokens, ttft)


# ---------------------------------------------------------------- decision
def prefill_ttft(model: StepModel, queue: Sequence[int], chi_p: int, prompt: int) -> Tuple[float, float]:
    """(W_queue, T_pf) on the prefill node (Eqs. 2 and 3)."""
    q = float(sum(queue))
    wait = (q / chi_p) * float(model.prefill_step(chi_p, q / 2.0)) if q > 0 else 0.0
    n = math.ceil(prompt / chi_p)
    sizes = np.minimum(chi_p, prompt - chi_p * np.arange(n))
    t_pf = float(np.sum(model.prefill_step(sizes, chi_p * np.arange(n))))
    return wait, t_pf


@dataclasses.dataclass
class Decision:
    deflect: bool
    node: int                     # -1 when kept on the prefill node
    schedule: Optional[Schedule]
    ttft_pf: float
    ttft_dec: float               # inf when no node is feasible


def decide(model: StepModel, prompt: int, queue: Sequence[int], chi_p: int, nodes: Sequence[Tuple[int, int]],
           cands: Sequence[int], tau: float, beta: float = 1.0, alpha: float = 1.3,
           ttft_slo: float = float("inf")) -> Decision:
    """Algorithm 1 for one request: nodes are (B_n, K_n) of each decode node."""
    wait, t_pf = prefill_ttft(model, queue, chi_p, prompt)
    ttft_pf = wait + t_pf
    best, best_node = None, -1
    for n, (B, K) in enumerate(nodes):
        s = chunk_schedule(model, B, K, prompt, cands, tau, beta)
        if s is not None and (best is None or s.ttft < best.ttft):
            best, best_node = s, n
    if best is None:
        return Decision(False, -1, None, ttft_pf, float("inf"))
    ok = best.ttft <= alpha * ttft_pf and best.ttft <= ttft_slo  # Eq. 7
    return Decision(ok, best_node if ok else -1, best if ok else None, ttft_pf, best.ttft)


def main(argv=None):
    import argparse
    import csv
    ap = argparse.ArgumentParser(description="fit the step-latency model to measured steps (CSV B,K,c,p,us)")
    ap.add_argument("csv")
    ap.add_argument("--out", default=MODEL_PATH)
    args = ap.parse_args(argv)
    with open(args.csv) as fh:
        rows = [(int(r["B"]), int(r["K"]), int(r["c"]), int(r["p"]), float(r["us"])) for r in csv.DictReader(fh)]
    model = StepModel.fit(rows)
    with open(args.out, "w") as fh:
        fh.write(model.to_json() + "\n")
    dec = [r for r in rows if r[0] > 0]
    pf = [r for r in rows if r[0] == 0]
    print(f"fitted {len(rows)} steps: MAPE decode-node {mape(model, dec):.3f}, prefill-node "
          f"{mape(model, pf) if pf else float('nan'):.3f}; wrote {args.out}")


if __name__ == "__main__":
    main()
