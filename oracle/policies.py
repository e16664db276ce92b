"""Oracle of the reservation-policy comparison (TEST INFRASTRUCTURE ONLY).

Plain definitions of the policies the paper prices against each other
(Sec. 5.1 baselines; Sec. 5.4 length-prediction baselines; Table 2 and
Table 5) and their average stochastic cost on held-out samples (Sec. 3.3):

  DRO(eps)   the grid reservation of least worst-case cost (App. A; Prop. 4.2
             on the grid), one per radius row
  SAA        eps = 0: the critical-fractile quantile (Prop. 4.2)
  P90/P99    the ceil(qN)-th smallest training sample
  P95        the same at q = 0.95, rounded up to a multiple of 16 tokens
             (block alignment of the KV cache)
  Mean       the smallest integer >= the training mean
  Max        L
  LP+k sigma the smallest integer >= mean + k * (population standard
             deviation), at most L, for k = 1, 2

Quantile ranks, means and spreads are exact rationals here (Fractions), an
implementation independent of the library's integer arithmetic.
"""
from __future__ import annotations

import math
from fractions import Fraction as F

import numpy as np

import oracle

BLOCK = 16
BASELINES = ("SAA", "P90", "P95", "P99", "Mean", "Max", "LP+1sigma", "LP+2sigma")


def policy_names(eps_fracs) -> list[str]:
    return [f"DRO(eps={f:g}*mean)" for f in eps_fracs] + list(BASELINES)


def _order_stat(xs_sorted, q: F) -> int:
    n = len(xs_sorted)
    j = math.ceil(q * n)            # rank, 1-based
    return int(xs_sorted[max(1, min(n, j)) - 1])


def _mean_plus(xs, k: int, L: int) -> int:
    n = len(xs)
    s = sum(int(v) for v in xs)
    ss = sum(int(v) * int(v) for v in xs)
    mean = F(s, n)
    var = F(ss, n) - mean * mean
    r = math.floor(float(mean) + k * math.sqrt(float(var))) - 2
    while True:                     # smallest r with r >= mean + k sqrt(var)
        d = r - mean
        if d >= 0 and d * d >= k * k * var:
            break
        r += 1
    return min(r, L)


def reservations(w_train, eps_fracs) -> np.ndarray:
    """[R, C] reservations of every policy for every training class."""
    sol = oracle.solve(w_train, grouped=True)
    dro = np.stack([w_train.eta[sol["k_star"][e]] for e in range(len(eps_fracs))])
    rows = [r for r in dro]
    C = w_train.C
    qv, _ = oracle.quantile(w_train)
    per = {"SAA": qv}
    for name in ("P90", "P95", "P99", "Mean", "Max", "LP+1sigma", "LP+2sigma"):
        per[name] = np.empty(C, np.int64)
    for c in range(C):
        xs = np.sort(w_train.samples_of(c))
        L = int(w_train.L[c])
        per["P90"][c] = _order_stat(xs, F(90, 100))
        p95 = _order_stat(xs, F(95, 100))
        per["P95"][c] = -(-p95 // BLOCK) * BLOCK
        per["P99"][c] = _order_stat(xs, F(99, 100))
        per["Mean"][c] = math.ceil(F(sum(int(v) for v in xs), len(xs)))
        per["Max"][c] = L
        per["LP+1sigma"][c] = _mean_plus(xs, 1, L)
        per["LP+2sigma"][c] = _mean_plus(xs, 2, L)
    rows += [per[n] for n in BASELINES]
    return np.stack(rows).astype(np.int32)


def price(w_eval, eta_train: np.ndarray):
    """Cost and cover of each training-class reservation on every shifted set.

    Evaluation class s * C + i is segment (shift) s priced with the costs of
    training class i; returns cost [R, S, C] and cover [R, S, C].
    """
    R, C = eta_train.shape
    S = w_eval.C // C
    eta_r = np.tile(eta_train, (1, S))
    cost, cover, _ = oracle.reservation_cost(w_eval, eta_r)
    return cost.reshape(R, S, C), cover.reshape(R, S, C)


def table(w_train, w_eval, eps_fracs) -> dict:
    eta = reservations(w_train, eps_fracs)
    cost, cover = price(w_eval, eta)
    c_in, cov_in, _ = oracle.reservation_cost(w_train, eta)
    return dict(names=policy_names(eps_fracs), eta=eta, cost=cost, cover=cover,
                cost_train=c_in, cover_train=cov_in)
