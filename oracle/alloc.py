"""Rank / bit-width allocator of KV-COBRA (C1, C2, exact DP), written plainly (oracle).

Test infrastructure only: nothing in the product path may import this module.

Passages followed
-----------------
* Head distortion D(r, b) = sum_{i>r} w_i + q(b) sum_{i<=r} w_i:
  Eq. (eq:drb-preview), Lemma lem:head-dist (Appendix A).
* Global problem min sum D s.t. sum r b <= B_tot, B_tot = L H d bpd: Eq. (eq:global).
* Weights: w_i = lambda_i (MSE objective) or w_i = sigma_Q,i^2 lambda_i
  (attention-KL objective, Proposition prop:kl-bound); the basis is reordered
  by w descending before C1/C2 (Section 4, "Reordering and plug-in"; table step 2).
* C1: enumerate the even rank grid, b from the budget, argmin D
  (Section 3.2; Proposition thm:c1-kkt and the Solver paragraph, Appendix B).
* C2: damped proportional update with eta = 0.3, clamp at B_min, then
  renormalise to B_tot; five rounds (Section 3.3; Eq. eq:c2-update, Appendix C;
  table steps 3-4).
* Exact DP over integer per-head budgets (Appendix D, "Alternative solver").
* V side in joint K+V mode: uniform per-head budget, C1 only (Appendix F).
* Exact DP over measured distortion tables (Appendix D, "Exact DP over
  measured distortion"): the same knapsack with the per-head optimum taken
  over a table of measured D(r, b) (measured.py) instead of the model.

Readings (paper silent or inconsistent)
---------------------------------------
* C1 takes b = min(b_max, floor(B / r)), not round(B / r): rounding can break
  the constraint r b <= B that the problem states; the floor keeps every
  candidate feasible. Candidates r = r_min, r_min + r_step, ... up to
  min(d, floor(B / b_min)); ties keep the smallest r. If no candidate is
  feasible the head gets (r_min, b_min).
* B_min = r_min * b_min, B_max = d * b_max. A final C1 runs after the last
  C2 update. The damped update clamps, then renormalises (paper order).
* fp64 evaluation order (both sides of the parity check use it):
  head sums S_r accumulate w_1..w_r left to right; tail sums accumulate from
  w_d down to w_{r+1}; D = tail + q(b) * head. C2 sums run over heads in
  index order.
* DP: integer budgets beta_h in [ceil(B_min), floor(B_max)], sum <= floor(B_tot),
  D*_h(beta) = C1(beta). Heads are processed in index order; for each total the
  smallest beta_h attaining the minimum is kept (strict comparison).
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from .quant import q_model

SOLVER_DAMPED = 0
SOLVER_DP = 1
SOLVER_C1_ONLY = 2


@dataclass
class AllocOpts:
    d: int = 128
    r_min: int = 2
    r_step: int = 2
    b_min: int = 1
    b_max: int = 8
    solver: int = SOLVER_DAMPED
    rounds: int = 5
    reorder: bool = True
    bpd: float = 2.0
    eta: float = 0.3
    B_min: float | None = None   # default r_min * b_min
    B_max: float | None = None   # default d * b_max

    def bmin(self) -> float:
        return float(self.r_min * self.b_min) if self.B_min is None else float(self.B_min)

    def bmax(self) -> float:
        return float(self.d * self.b_max) if self.B_max is None else float(self.B_max)


def kl_weights(lam, sigma2_q):
    """w_i = sigma_Q,i^2 * lambda_i (Proposition prop:kl-bound)."""
    return [float(s) * float(l) for s, l in zip(sigma2_q, lam)]


def importance_order(w) -> list[int]:
    """Eigen indices sorted by w descending; equal weights keep eigen order."""
    idx = list(range(len(w)))
    return sorted(idx, key=lambda i: (-float(w[i]), i))


def head_sum(w, r: int) -> float:
    s = 0.0
    for i in range(r):
        s = s + float(w[i])
    return s


def tail_sum(w, r: int) -> float:
    s = 0.0
    for i in range(len(w) - 1, r - 1, -1):
        s = s + float(w[i])
    return s


def distortion(w, r: int, b: int) -> float:
    """D(r, b) = sum_{i>r} w_i + q(b) sum_{i<=r} w_i for w in importance order."""
    return tail_sum(w, r) + q_model(b) * head_sum(w, r)


class HeadSums:
    """All head sums S[r] and tail sums T[r] of one head, built with the same
    additions, in the same order, as head_sum / tail_sum."""

    def __init__(self, w):
        d = len(w)
        self.S = [0.0] * (d + 1)
        self.T = [0.0] * (d + 1)
        for k in range(d):
            self.S[k + 1] = self.S[k] + float(w[k])
        for k in range(d - 1, -1, -1):
            self.T[k] = self.T[k + 1] + float(w[k])
        self.d = d

    def __len__(self):
        return self.d

    def distortion(self, r: int, b: int) -> float:
        return self.T[r] + q_model(b) * self.S[r]


def c1(w, B: float, o: AllocOpts):
    """Per-head optimum (r, b, D) at real budget B (w: weights or their HeadSums)."""
    hs = w if isinstance(w, HeadSums) else HeadSums(w)
    d = len(hs)
    r_hi = min(d, math.floor(B / o.b_min))
    best = None
    r = o.r_min
    while r <= r_hi:
        b = min(o.b_max, math.floor(B / r))
        D = hs.distortion(r, b)
        if best is None or D < best[2]:
            best = (r, b, D)
        r += o.r_step
    if best is None:
        best = (o.r_min, o.b_min, hs.distortion(o.r_min, o.b_min))
    return best


def brute_force_head(w, B: float, o: AllocOpts):
    """Minimum of D(r, b) over every grid pair with r * b <= B (exhaustive)."""
    d = len(w)
    best = None
    for r in range(o.r_min, d + 1, o.r_step):
        for b in range(o.b_min, o.b_max + 1):
            if r * b <= B:
                D = distortion(w, r, b)
                if best is None or D < best[2]:
                    best = (r, b, D)
    return best


def c2_damped(W, o: AllocOpts):
    """Table steps 3-4 with the damped update of Eq. (eq:c2-update); returns (budgets, allocs)."""
    N = len(W)
    d = o.d
    B_tot = o.bpd * float(N * d)
    B_bar = B_tot / N
    step = o.eta * B_bar
    W = [HeadSums(w) for w in W]
    B = [o.bpd * float(d) for _ in range(N)]
    for _ in range(o.rounds):
        allocs = [c1(W[h], B[h], o) for h in range(N)]
        D_sum = 0.0
        for a in allocs:
            D_sum = D_sum + a[2]
        D_bar = D_sum / N
        if not D_bar > 0.0:
            break
        Bp = [max(o.bmin(), B[h] + step * (math.sqrt(allocs[h][2] / D_bar) - 1.0)) for h in range(N)]
        S = 0.0
        for v in Bp:
            S = S + v
        f = B_tot / S
        B = [v * f for v in Bp]
    allocs = [c1(W[h], B[h], o) for h in range(N)]
    return B, allocs


def dp_exact(W, o: AllocOpts):
    """Exact separable knapsack over integer budgets (Appendix D), full enumeration."""
    W = [HeadSums(w) for w in W]
    return _dp(len(W), lambda h, beta: c1(W[h], float(beta), o), o)


def _dp(N, head_opt, o: AllocOpts):
    """The knapsack of dp_exact over integer budgets with the per-head optimum head_opt(h, beta)."""
    B_tot = o.bpd * float(N * o.d)
    cap = math.floor(B_tot)
    lo = math.ceil(o.bmin())
    hi = math.floor(o.bmax())
    dstar = [[None] * (hi + 1) for _ in range(N)]
    for h in range(N):
        for beta in range(lo, hi + 1):
            dstar[h][beta] = head_opt(h, beta)
    INF = math.inf
    prev = [0.0] * (cap + 1)
    choice = []
    for h in range(N):
        cur = [INF] * (cap + 1)
        ch = [-1] * (cap + 1)
        for tot in range(cap + 1):
            best = INF
            arg = -1
            for beta in range(lo, min(hi, tot) + 1):
                base = prev[tot - beta]
                if base == INF:
                    continue
                v = base + dstar[h][beta][2]
                if v < best:
                    best, arg = v, beta
            cur[tot] = best
            ch[tot] = arg
        choice.append(ch)
        prev = cur
    if prev[cap] == INF:
        raise ValueError("budget below N * B_min")
    budgets = [0] * N
    tot = cap
    for h in range(N - 1, -1, -1):
        budgets[h] = choice[h][tot]
        tot -= budgets[h]
    allocs = [dstar[h][budgets[h]] for h in range(N)]
    return [float(x) for x in budgets], allocs, prev[cap]


def c1_table(Dt, B: float, o: AllocOpts):
    """Per-head optimum over a distortion table Dt[ri][bi] (r = r_min + ri r_step, b = b_min + bi): the
    smallest D over every grid pair with r b <= B (ties: smallest r, then smallest b), as (r, b, D).
    Below the smallest pair the head gets (r_min, b_min)."""
    best = None
    for ri in range(len(Dt)):
        r = o.r_min + ri * o.r_step
        for bi in range(len(Dt[ri])):
            b = o.b_min + bi
            if r * b <= B and (best is None or Dt[ri][bi] < best[2]):
                best = (r, b, float(Dt[ri][bi]))
    if best is None:
        best = (o.r_min, o.b_min, float(Dt[0][0]))
    return best


def dp_tables(tables, o: AllocOpts):
    """Exact DP (Appendix D) with D*_h(beta) = c1_table(tables[h], beta): the measured-distortion solver."""
    return _dp(len(tables), lambda h, beta: c1_table(tables[h], float(beta), o), o)


def brute_force_tables(tables, o: AllocOpts) -> float:
    """min sum_h tables[h][r_h][b_h] s.t. sum r_h b_h <= floor(B_tot), every pair enumerated (tiny only)."""
    N = len(tables)
    cap = math.floor(o.bpd * float(N * o.d))
    best = math.inf

    def rec(h, used, acc):
        nonlocal best
        if h == N:
            best = min(best, acc)
            return
        for ri in range(len(tables[h])):
            r = o.r_min + ri * o.r_step
            for bi in range(len(tables[h][ri])):
                b = o.b_min + bi
                if used + r * b <= cap:
                    rec(h + 1, used + r * b, acc + tables[h][ri][bi])

    rec(0, 0, 0.0)
    return best


def brute_force_global(W, o: AllocOpts) -> float:
    """min sum_h D_h(r_h, b_h) s.t. sum r_h b_h <= floor(B_tot), every pair enumerated (tiny only)."""
    N = len(W)
    cap = math.floor(o.bpd * float(N * o.d))
    pairs = []
    for h in range(N):
        ph = []
        for r in range(o.r_min, len(W[h]) + 1, o.r_step):
            for b in range(o.b_min, o.b_max + 1):
                ph.append((r * b, distortion(W[h], r, b)))
        pairs.append(ph)
    best = math.inf

    def rec(h, used, acc):
        nonlocal best
        if h == N:
            best = min(best, acc)
            return
        for cost, D in pairs[h]:
            if used + cost <= cap:
                rec(h + 1, used + cost, acc + D)

    rec(0, 0, 0.0)
    return best


def allocate(lam, sigma2_q, o: AllocOpts):
    """kvc_allocate semantics: weights, importance reorder, solver; returns dict of arrays.

    lam[h], sigma2_q[h] are indexed by eigen index (descending lambda). With
    sigma2_q None the MSE weights w = lambda are used.
    """
    N = len(lam)
    W, orders = [], []
    for h in range(N):
        w = [float(v) for v in lam[h]] if sigma2_q is None else kl_weights(lam[h], sigma2_q[h])
        order = importance_order(w) if o.reorder else list(range(len(w)))
        W.append([w[i] for i in order])
        orders.append(order)
    if o.solver == SOLVER_C1_ONLY:
        B = [o.bpd * float(o.d) for _ in range(N)]
        allocs = [c1(HeadSums(W[h]), B[h], o) for h in range(N)]
    elif o.solver == SOLVER_DAMPED:
        B, allocs = c2_damped(W, o)
    elif o.solver == SOLVER_DP:
        B, allocs, _ = dp_exact(W, o)
    else:
        raise ValueError("unknown solver")
    return {
        "r": np.array([a[0] for a in allocs], dtype=np.int32),
        "b": np.array([a[1] for a in allocs], dtype=np.int32),
        "B": np.array(B, dtype=np.float64),
        "D": np.array([a[2] for a in allocs], dtype=np.float64),
        "order": np.array(orders, dtype=np.int32),
        "w_sorted": W,
    }
