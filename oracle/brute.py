"""Brute-force routines that pin the oracle to something other than itself.

TEST INFRASTRUCTURE ONLY.  Everything here works on tiny inputs, in exact
rational arithmetic (fractions.Fraction) or with a general-purpose LP solver,
and is written directly from the definitions, not from the closed forms the
oracle uses:

  * `sup_brute`       the pointwise supremum of Step 4 (Appendix A) by
                      scanning the support [0, L] on a fine rational grid
                      plus the kinks of the objective;
  * `worst_case_lp`   the primal worst-case expectation over the Wasserstein
                      ball (Appendix A, Step 1: the ball and its W1 distance), as a
                      transport-plan linear program solved with HiGHS;
  * `dual_exact`      min over gamma >= 0 of the Kantorovich dual (App. A, Step 3),
                      evaluated exactly at every breakpoint of the convex
                      piecewise-linear objective;
  * `saa_exact`       the empirical mean of the stochastic cost (Sec. 3.3).
"""
from __future__ import annotations

import math
from fractions import Fraction as F
from itertools import product

import numpy as np


def Q(eta, x, cp, cw):
    """Stochastic cost c_p (x - eta)^+ + c_w (eta - x)^+ (Sec. 3.3, L_in folded into eta)."""
    return F(cp) * max(F(x) - F(eta), 0) + F(cw) * max(F(eta) - F(x), 0)


def sup_brute(eta, xh, L, cp, cw, lam, steps: int = 64):
    """sup over xi in [0, L] of Q(eta, xi) - lam |xi - xh|, by exhaustive scan.

    The objective is piecewise linear with kinks at eta and xh, so the scan
    over a fine grid plus those kinks attains the supremum exactly.
    """
    pts = {F(0), F(L), F(eta), F(xh)}
    pts |= {F(L) * i / steps for i in range(steps + 1)}
    best = None
    for p in pts:
        if p < 0 or p > L:
            continue
        v = Q(eta, p, cp, cw) - F(lam) * abs(p - F(xh))
        best = v if best is None or v > best else best
    return best


def saa_exact(eta, xs, cp, cw):
    """(1/N) sum_n Q(eta, x_n) as an exact rational."""
    return sum((Q(eta, x, cp, cw) for x in xs), F(0)) / len(xs)


def _phi_max3(eta, x, L, cp, cw, g):
    cand = (F(cw) * F(eta) - g * F(x), Q(eta, x, cp, cw), F(cp) * (F(L) - F(eta)) - g * (F(L) - F(x)))
    return max(cand)


def dual_exact(eta, xs, L, cp, cw, eps):
    """min over gamma >= 0 of the Kantorovich dual (App. A, Step 3), exactly.

    Each per-sample supremum is a max of lines in gamma, so the objective is
    convex piecewise linear in gamma; its minimum sits at gamma = 0 or at a
    point where two of the lines cross.  All such points are enumerated.
    Returns (value, gamma_at_min) with the smallest minimising gamma.
    """
    cands = {F(0), F(cp), F(cw)}
    for x in set(xs):
        # line in gamma of each candidate point: a - b*gamma
        lines = [(F(cw) * F(eta), F(x)), (Q(eta, x, cp, cw), F(0)),
                 (F(cp) * (F(L) - F(eta)), F(L) - F(x))]
        for (a1, b1), (a2, b2) in product(lines, lines):
            if b1 != b2:
                gam = (a1 - a2) / (b1 - b2)
                if gam >= 0:
                    cands.add(gam)
    best = None
    for g in sorted(cands):
        v = g * F(eps) + sum((_phi_max3(eta, x, L, cp, cw, g) for x in xs), F(0)) / len(xs)
        if best is None or v < best[0]:
            best = (v, g)
    return best


def worst_case_lp(eta, xs, L, cp, cw, eps, support=None):
    """sup over P with W1(P, P_N) <= eps of E_P[Q] as a transport-plan LP.

    Variables pi[n, v] >= 0 move the mass 1/N of sample n to support point v;
    sum_v pi[n, v] = 1/N, sum pi[n, v] |v - x_n| <= eps.  The default support
    is every integer and half-integer in [0, L].
    """
    from scipy.optimize import linprog

    if support is None:
        support = np.arange(0, 2 * L + 1) / 2.0
    N, V = len(xs), len(support)
    cost = np.array([float(Q(eta, v, cp, cw)) for v in support])
    c = -np.tile(cost, N) / 1.0
    A_eq = np.zeros((N, N * V))
    for n in range(N):
        A_eq[n, n * V:(n + 1) * V] = 1.0
    b_eq = np.full(N, 1.0 / N)
    A_ub = np.concatenate([np.abs(support - x) for x in xs])[None, :]
    b_ub = np.array([float(eps)])
    res = linprog(c, A_ub=A_ub, b_ub=b_ub, A_eq=A_eq, b_eq=b_eq, bounds=(0, None), method="highs")
    if res.status != 0:
        raise RuntimeError(res.message)
    return -res.fun


def rank_exact(cp, cw, N):
    """ceil(c_p N / (c_p + c_w)) in rationals, clamped to [1, N]."""
    q = F(cp) / (F(cp) + F(cw))
    return min(max(math.ceil(q * N), 1), N)
