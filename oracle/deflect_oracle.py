"""Plain reference of the step-latency model, the TBT-safe chunk schedule and
the deflection decision (sections 4.3.1-4.4 of the paper; Eqs. 1-7 and
Algorithm 1).

TEST INFRASTRUCTURE ONLY: imported by tests/, never by the product path.  It
shares no code with the package: every formula is written out here from the
paper's definitions, with scalar Python floats, one step at a time, in the
order the paper states them.

Model (the reading shared with the package, stated once here):
  T_step(B, K, p, c) = T0(B, K) + max(0, dT_pf)          (Eq. 4)
  T0    = a0 + a1 B + a2 K + a3 sqrt(K)
  dT_pf = b1 c + b2 c p + b3 c^2 + b4 c K                (only when c > 0)
  T_prefill(chi, cached) = e0 + e1 chi + e2 chi cached + e3 chi^2
B decode rows over K cached decode tokens; a chunk of c prompt tokens after
p cached tokens of its own prompt.  A step of chi tokens carries chi - B
prompt tokens (the last one what is left of the prompt).
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence, Tuple


# --------------------------------------------------------------- regression
def solve_least_squares(rows: Sequence[Sequence[float]], y: Sequence[float],
                        weights: Optional[Sequence[float]] = None) -> List[float]:
    """Weighted least squares through the normal equations (X^T W X) w =
    X^T W y, solved by Gaussian elimination with partial pivoting."""
    n = len(rows[0])
    if weights is None:
        weights = [1.0] * len(rows)
    A = [[0.0] * n for _ in range(n)]
    b = [0.0] * n
    for x, t, wt in zip(rows, y, weights):
        for i in range(n):
            b[i] += wt * x[i] * t
            for j in range(n):
                A[i][j] += wt * x[i] * x[j]
    # column scaling by powers of two (exact) keeps the elimination well scaled
    scale = [2.0 ** -round(math.log2(math.sqrt(A[i][i]))) if A[i][i] > 0 else 1.0 for i in range(n)]
    A = [[A[i][j] * scale[i] * scale[j] for j in range(n)] for i in range(n)]
    b = [b[i] * scale[i] for i in range(n)]
    for col in range(n):
        piv = max(range(col, n), key=lambda r: abs(A[r][col]))
        A[col], A[piv] = A[piv], A[col]
        b[col], b[piv] = b[piv], b[col]
        for r in range(col + 1, n):
            f = A[r][col] / A[col][col]
            for j in range(col, n):
                A[r][j] -= f * A[col][j]
            b[r] -= f * b[col]
    w = [0.0] * n
    for i in reversed(range(n)):
        s = b[i] - sum(A[i][j] * w[j] for j in range(i + 1, n))
        w[i] = s / A[i][i]
    return [w[i] * scale[i] for i in range(n)]


def fit(measured: Sequence[Tuple[int, int, int, int, float]]):
    """Fit (a, b, e) from measured steps (B, K per decode request, c, p, t):
    T0 on decode-only steps, dT_pf on the residual of mixed steps, the
    prefill model on steps without decode rows; every fit minimises relative
    error (weights 1 / t^2 on squared residuals)."""
    dec = [(B, B * Kr, c, p, t) for B, Kr, c, p, t in measured if B > 0 and c == 0]
    mix = [(B, B * Kr, c, p, t) for B, Kr, c, p, t in measured if B > 0 and c > 0]
    pre = [(c, p, t) for B, Kr, c, p, t in measured if B == 0]
    a = solve_least_squares([[1.0, B, K, math.sqrt(K)] for B, K, c, p, t in dec], [t for *_, t in dec],
                            [1.0 / (t * t) for *_, t in dec])
    resid = [t - (a[0] + a[1] * B + a[2] * K + a[3] * math.sqrt(K)) for B, K, c, p, t in mix]
    b = solve_least_squares([[c, c * p, c * c, c * K] for B, K, c, p, t in mix], resid,
                            [1.0 / (t * t) for *_, t in mix])
    e = solve_least_squares([[1.0, c, c * p, c * c] for c, p, t in pre], [t for *_, t in pre],
                            [1.0 / (t * t) for *_, t in pre]) if pre else [0.0] * 4
    return a, b, e


# -------------------------------------------------------------------- model
def t_step(model, B: int, K: int, p: int, c: int) -> float:
    """Eq. 4 for B decode rows over K cached tokens plus c prompt tokens after p."""
    a, b, _ = model
    t0 = a[0] + a[1] * B + a[2] * K + a[3] * math.sqrt(K)
    if c <= 0:
        return t0
    d = b[0] * c + b[1] * c * p + b[2] * c * c + b[3] * c * K
    return t0 + max(0.0, d)


def t_prefill(model, chi: int, cached: float) -> float:
    _, _, e = model
    return e[0] + e[1] * chi + e[2] * chi * cached + e[3] * chi * chi


# ------------------------------------------------------------ chunk schedule
def largest_safe(model, B: int, K: int, served: int, left: int, cands: Sequence[int], limit: float) -> int:
    """The first chi of the candidates, largest first, whose step is TBT-safe (Eq. 5)."""
    for chi in sorted(cands, reverse=True):
        c = min(chi - B, left)
        if c > 0 and t_step(model, B, K, served, c) <= limit:
            return chi
    return 0


def chunk_schedule(model, B: int, K: int, prompt: int, cands: Sequence[int], tau: float, beta: float = 1.0):
    """Algorithm 1's inner loop for one decode node: (chis, tokens, ttft) or None."""
    chis, toks = [], []
    ttft = 0.0
    served = 0
    while served < prompt:
        left = prompt - served
        chi = largest_safe(model, B, K, served, left, cands, beta * tau)
        if chi == 0:
            return None
        c = min(chi - B, left)
        ttft += t_step(model, B, K, served, c)  # Eq. 6
        chis.append(chi)
        toks.append(c)
        served += c
    return chis, toks, ttft


# ----------------------------------------------------------------- decision
def queue_wait(model, queue: Sequence[int], chi_p: int) -> float:
    """Eq. 2."""
    q = sum(queue)
    if q == 0:
        return 0.0
    return (q / chi_p) * t_prefill(model, chi_p, q / 2.0)


def prefill_exec(model, prompt: int, chi_p: int) -> float:
    """Eq. 3: chunk i of the prompt at prefix chi_p * i."""
    total = 0.0
    i = 0
    while chi_p * i < prompt:
        total += t_prefill(model, min(chi_p, prompt - chi_p * i), chi_p * i)
        i += 1
    return total


def decide(model, prompt: int, queue: Sequence[int], chi_p: int, nodes: Sequence[Tuple[int, int]],
           cands: Sequence[int], tau: float, beta: float = 1.0, alpha: float = 1.3, ttft_slo: float = math.inf):
    """Algorithm 1: (deflect, node, chis, ttft_pf, ttft_dec)."""
    ttft_pf = queue_wait(model, queue, chi_p) + prefill_exec(model, prompt, chi_p)  # Eq. 1
    best = None
    for n, (B, K) in enumerate(nodes):
        s = chunk_schedule(model, B, K, prompt, cands, tau, beta)
        if s is not None and (best is None or s[2] < best[1][2]):
            best = (n, s)
    if best is None:
        return False, -1, None, ttft_pf, math.inf
    n, (chis, toks, ttft_dec) = best
    if ttft_dec <= alpha * ttft_pf and ttft_dec <= ttft_slo:  # Eq. 7
        return True, n, chis, ttft_pf, ttft_dec
    return False, -1, None, ttft_pf, ttft_dec
