"""Oracle of the rest of Alg. 1: routing (LP1), prefix caching (Block 2) and
configuration search (Block 3), around the reservation update (LP2).

TEST INFRASTRUCTURE ONLY: called by the tests and by the golden-file script.

Definitions (Sec. 3.1-3.4, Prop. 4.1 and Alg. 1), with the readings of what
the paper leaves open marked "reading":

  T[c,g]   = pp_g alpha Lin_c / Cc_g + beta E[xi_c] / Bc_g + NL tau_g t_ar      service time
  ET2[c,g] = A^2 + 2 A B E[xi_c] + B^2 E[xi_c^2] with A = pp_g alpha Lin_c / Cc_g
             + NL tau_g t_ar and B = beta / Bc_g: second moment of the service
             time over the samples (reading: the paper takes the variability of
             the service time from the training samples)
  conc[c,g] = lam_c T_cg pi_cg / z_g                 concurrent requests (Little's law)
  mem[g]   = (1 + kappa) (sum_c lam_c T_cg pi_cg (Lin_c + eta_c - delta_cg Lpre_c)) / z_g
             + sum_c delta_cg Lpre_c                 KV tokens in use (Sec. 3.4)
  util[g]  = mem_g / Mcap_g  (reading: the memory utilisation, at which the
             paper's simulator evaluates the queue; with the compute utilisation
             sum_c conc_cg, which the queue needs below 1, no concurrency could
             exceed 1 and Block 2 would never cache)
  Wq[g]    = util (1 + Cs2) / (2 (1 - util)) Tbar   Pollaczek-Khinchin, where with
             X = sum_c lam_c pi_cg > 0: Tbar = sum_c lam_c pi_cg T_cg / X and
             Cs2 = (sum_c lam_c pi_cg ET2_cg / X) / Tbar^2 - 1 (no traffic: Wq = 0)
  objective = sum_c lam_c (a_c W_c + sum_g pi_cg c_gpu tau_g pp_g T_cg + c_slo s_c
                           + (1 - a_c) c_rej),  a_c = sum_g pi_cg,
             s_c = max(0, sum_g pi_cg (Wq_g + T_cg) - a_c D_c),
             W_c = the exact worst-case cost of class c at its grid reservation
  feasible = sum_g z_g tau_g pp_g <= J; pi_cg > 0 only where z_g >= 1;
             mem_g <= u_max Mcap_g where z_g >= 1 (reading: the capacity of
             Sec. 3.4 with a margin that keeps the waiting time finite), checked
             with a relative slack of 1e-9 so that a routing the LP leaves
             exactly at the bound counts as feasible
  LP1      = min over pi >= 0 (and s >= 0) of the objective with eta, z, delta
             fixed and Wq frozen (reading: the queue is linearised at the state
             entering Block 1 and held while LP1 and LP2 alternate, so that the
             alternation is between two LPs with fixed data), subject to
             sum_g pi_cg <= 1, the slack rows and the memory rows
  LP2      = the block step's reservation sweep with conc_cg and the capacity
             left after the prefixes and the input tokens
  Block 2  : delta_cg = 1[conc_cg > 1]
  Block 3  : over every feasible z in Z (r, pi, delta fixed) the first minimiser in
             lexicographic order of (z_0, ..., z_{G-1}); the current z is kept
             when it attains the minimum (reading: a block moves only on a strict
             improvement, as in the monotone-descent argument of Prop. 4.3)

Every double expression is written in a fixed order, one rounding per
operation, as the library evaluates it.

Pins (tests/test_oracle_pins.py): the P-K wait reduces to the M/M/1 wait,
caching saves memory exactly when the concurrency exceeds the margin, the LP1
optimum (HiGHS) beats sampled feasible routings, the configuration scan equals
brute force, and the LP2 sweep equals the pinned block step (P20-P24); the
service-time moments, concurrencies, memory, waiting times and objective equal
their formulas evaluated in exact rationals in another algebraic form (per
sample value; E[S^2] / (2 E[S]) for the wait) (P25-P28).  What stays unpinned
is the model itself: it follows readings of a model whose constants the paper
does not print.
"""
from __future__ import annotations

import itertools
import math

import numpy as np

import oracle

PI_TOL = 1e-9     # routing change below which Block 1 counts as converged
MEM_SLACK = 1.0 + 1e-9   # relative slack of the memory check of a configuration
ETA_SLACK = 1e-6         # tokens of slack of the reservation bound of the sweep


def service_times(svc, w):
    """T[c,g] and ET2[c,g] from the exact per-class moments."""
    mo = oracle.moments(w)
    C, G = w.C, svc.G
    T = np.empty((C, G))
    ET2 = np.empty((C, G))
    for c in range(C):
        n = float(int(mo["count"][c]))
        mean = float(int(mo["sum"][c])) / n          # RN(RN(sum) / N)
        ex2 = float(int(mo["sumsq"][c])) / n         # RN(RN(sum of squares) / N)
        for g in range(G):
            A = float(svc.pp[g]) * float(svc.alpha) * float(svc.Lin[c]) / float(svc.Cc[g])
            A = A + float(svc.NL) * float(svc.tau[g]) * float(svc.t_ar)
            B = float(svc.beta) / float(svc.Bc[g])
            T[c, g] = A + B * mean
            ET2[c, g] = A * A + 2.0 * A * B * mean + B * B * ex2
    return T, ET2


def concurrency(svc, T, pi, z):
    """conc[c,g] = (lam_c T_cg pi_cg) / z_g (0 where z_g = 0)."""
    C, G = T.shape
    conc = np.zeros((C, G))
    for c in range(C):
        for g in range(G):
            if z[g] > 0:
                conc[c, g] = float(svc.lam[c]) * T[c, g] * pi[c, g] / float(z[g])
    return conc


def memory(svc, T, pi, z, eta_c, delta):
    """KV tokens in use per group: (1 + kappa) (sum_c lam_c T_cg pi_cg rt_cg) / z_g
    + sum_c delta_cg Lpre_c with rt_cg = Lin_c + eta_c - delta_cg Lpre_c
    (0 where z_g = 0)."""
    C, G = T.shape
    mem = np.zeros(G)
    for g in range(G):
        if z[g] <= 0:
            continue
        used = 0.0
        pre = 0.0
        for c in range(C):
            rt = float(int(svc.Lin[c]) + int(eta_c[c]) - int(delta[c, g]) * int(svc.Lpre[c]))
            used = used + float(svc.lam[c]) * T[c, g] * pi[c, g] * rt
            pre = pre + float(int(delta[c, g]) * int(svc.Lpre[c]))
        mem[g] = (1.0 + float(svc.kappa)) * (used / float(z[g])) + pre
    return mem


def queue(svc, T, ET2, pi, z, mem):
    """Waiting time Wq[g] at memory use mem[g]."""
    C, G = T.shape
    Wq = np.zeros(G)
    for g in range(G):
        if z[g] <= 0:
            continue
        load = 0.0
        X = 0.0
        m2 = 0.0
        for c in range(C):
            wgt = float(svc.lam[c]) * pi[c, g]
            load = load + wgt * T[c, g]
            X = X + wgt
            m2 = m2 + wgt * ET2[c, g]
        if X > 0.0:
            u = mem[g] / float(svc.Mcap[g])
            tb = load / X
            cs2 = (m2 / X) / (tb * tb) - 1.0
            Wq[g] = u * (1.0 + cs2) / (2.0 * (1.0 - u)) * tb if u < 1.0 else math.inf
    return Wq


def objective(svc, Wc, T, Wq, pi):
    C, G = T.shape
    obj = 0.0
    for c in range(C):
        a = 0.0
        gpu = 0.0
        resp = 0.0
        for g in range(G):
            p = pi[c, g]
            a = a + p
            gpu = gpu + p * (float(svc.c_gpu) * float(int(svc.tau[g]) * int(svc.pp[g])) * T[c, g])
            resp = resp + p * (Wq[g] + T[c, g])
        s = resp - a * float(svc.D[c])
        if s < 0.0:
            s = 0.0
        term = a * Wc[c] + gpu + float(svc.c_slo) * s + (1.0 - a) * float(svc.c_rej)
        obj = obj + float(svc.lam[c]) * term
    return obj


def feasible(svc, T, pi, z, eta_c, delta):
    G = svc.G
    if sum(int(z[g]) * int(svc.tau[g]) * int(svc.pp[g]) for g in range(G)) > svc.J:
        return False
    for g in range(G):
        if z[g] <= 0 and np.any(pi[:, g] > 0.0):
            return False
    mem = memory(svc, T, pi, z, eta_c, delta)
    return all(mem[g] <= float(svc.u_max) * float(svc.Mcap[g]) * MEM_SLACK
               for g in range(G) if z[g] > 0)


def state_objective(svc, Wc, T, ET2, pi, z, eta_c, delta):
    mem = memory(svc, T, pi, z, eta_c, delta)
    return objective(svc, Wc, T, queue(svc, T, ET2, pi, z, mem), pi)


def routing_lp(svc, Wc, T, Wq, z, eta_c, delta):
    """LP1 with scipy's HiGHS: returns (pi [C, G], optimal objective)."""
    from scipy.optimize import linprog
    C, G = T.shape
    nv = C * G + C                     # pi (row-major c, g), then s_c
    cost = np.zeros(nv)
    lam = svc.lam.astype(np.float64)
    for c in range(C):
        for g in range(G):
            cost[c * G + g] = lam[c] * (Wc[c] + float(svc.c_gpu)
                                        * float(int(svc.tau[g]) * int(svc.pp[g])) * T[c, g]
                                        - float(svc.c_rej))
        cost[C * G + c] = lam[c] * float(svc.c_slo)
    A, b = [], []
    for c in range(C):                 # sum_g pi_cg <= 1
        row = np.zeros(nv)
        row[c * G:(c + 1) * G] = 1.0
        A.append(row)
        b.append(1.0)
    for c in range(C):                 # sum_g pi_cg (Wq_g + T_cg - D_c) - s_c <= 0
        row = np.zeros(nv)
        for g in range(G):
            if z[g] > 0:
                row[c * G + g] = Wq[g] + T[c, g] - float(svc.D[c])
        row[C * G + c] = -1.0
        A.append(row)
        b.append(0.0)
    kap = 1.0 + float(svc.kappa)
    for g in range(G):                 # memory: mem_g <= u_max Mcap_g
        if z[g] <= 0:
            continue
        row = np.zeros(nv)
        pre = 0.0
        for c in range(C):
            rt = float(int(svc.Lin[c]) + int(eta_c[c]) - int(delta[c, g]) * int(svc.Lpre[c]))
            row[c * G + g] = kap * (lam[c] * T[c, g] / float(z[g])) * rt
            pre += float(int(delta[c, g]) * int(svc.Lpre[c]))
        A.append(row)
        b.append(float(svc.u_max) * float(svc.Mcap[g]) - pre)
    bounds = [(0.0, 0.0 if z[g] <= 0 else None) for c in range(C) for g in range(G)]
    bounds += [(0.0, None)] * C
    r = linprog(cost, A_ub=np.array(A), b_ub=np.array(b), bounds=bounds, method="highs")
    if r.status != 0:
        raise RuntimeError(f"LP1: {r.message}")
    pi = np.maximum(r.x[:C * G].reshape(C, G), 0.0)
    return pi, float(r.fun) + float(np.sum(lam * float(svc.c_rej)))


def lp2_inputs(svc, T, pi, z, delta):
    """conc_cg and the memory left for the reservations:
    cap_g = u_max Mcap_g - sum_c delta_cg Lpre_c
            - (1 + kappa) (sum_c lam_c T_cg pi_cg (Lin_c - delta_cg Lpre_c)) / z_g."""
    C, G = T.shape
    conc = concurrency(svc, T, pi, z)
    cap = np.full(G, math.inf)
    kap = 1.0 + float(svc.kappa)
    for g in range(G):
        if z[g] <= 0:
            continue
        fixed = 0.0
        pre = 0.0
        for c in range(C):
            rt = float(int(svc.Lin[c]) - int(delta[c, g]) * int(svc.Lpre[c]))
            fixed = fixed + float(svc.lam[c]) * T[c, g] * pi[c, g] * rt
            pre = pre + float(int(delta[c, g]) * int(svc.Lpre[c]))
        cap[g] = float(svc.u_max) * float(svc.Mcap[g]) - pre - kap * (fixed / float(z[g]))
    return conc, cap


def sweep(W, eta, conc, cap_eff, kappa, k_prev):
    """LP2 on the grid: one Gauss-Seidel sweep over the classes.  For class c,
    bound_g = (cap_eff_g - (1+kappa) sum_{c' != c} conc_c'g eta_k(c')) /
    ((1+kappa) conc_cg) over the g with conc_cg > 0, kmax = the largest k with
    eta_k <= min_g bound_g + 1e-6 (the slack keeps a reservation at which the
    routing LP left the memory exactly full; none: k = 0, infeasible), k = the
    lowest argmin of W[c, :kmax+1]."""
    C, K = W.shape
    G = conc.shape[1]
    k = np.array(k_prev, dtype=np.int64)
    ok = np.ones(C, bool)
    onek = 1.0 + float(kappa)
    for c in range(C):
        bound = math.inf
        for g in range(G):
            if not (conc[c, g] > 0.0):
                continue
            other = 0.0
            for c2 in range(C):
                if c2 != c:
                    other = other + conc[c2, g] * float(eta[k[c2]])
            b = (cap_eff[g] - onek * other) / (onek * conc[c, g])
            if b < bound:
                bound = b
        kmax = -1
        for kk in range(K):
            if float(eta[kk]) <= bound + ETA_SLACK:
                kmax = kk
        ok[c] = kmax >= 0
        kmax = max(kmax, 0)
        best = 0
        for kk in range(1, kmax + 1):
            if W[c, kk] < W[c, best]:
                best = kk
        k[c] = best
    return k, ok


def prefix_cache(svc, T, pi, z):
    """Block 2: delta_cg = 1[conc_cg > 1]."""
    return (concurrency(svc, T, pi, z) > 1.0).astype(np.uint8)


def config_space(svc):
    """Every z in Z in lexicographic order."""
    G = svc.G
    cost = [int(svc.tau[g]) * int(svc.pp[g]) for g in range(G)]
    ranges = [range(svc.J // cost[g] + 1) for g in range(G)]
    for z in itertools.product(*ranges):
        if sum(z[g] * cost[g] for g in range(G)) <= svc.J:
            yield np.array(z, np.int64)


def config_search(svc, Wc, T, ET2, pi, eta_c, delta):
    """Block 3 scan: (first minimising z, its objective, its rank, feasible count)."""
    best, best_obj, best_rank, nfeas = None, math.inf, -1, 0
    for rank, z in enumerate(config_space(svc)):
        if not feasible(svc, T, pi, z, eta_c, delta):
            continue
        nfeas += 1
        o = state_objective(svc, Wc, T, ET2, pi, z, eta_c, delta)
        if o < best_obj:
            best, best_obj, best_rank = z, o, rank
    return best, best_obj, best_rank, nfeas


def solve(w, svc, max_outer: int = 10, max_inner: int = 10) -> dict:
    """Alg. 1 with the reservation on the grid (radius row 0 of w.eps).

    Start: z = svc.z0, delta = 0, pi = 0, r0 = L_in + E[xi] on the grid.
    Block 1 takes Wq at its entering state and alternates LP1 and LP2 until the
    reservations repeat and the
    routing moves by at most PI_TOL (or max_inner rounds); Block 2 sets delta;
    Block 3 picks z; the loop stops when z and delta repeat (or after
    max_outer iterations).
    """
    S = oracle.S_exact(w)
    W1 = oracle.W_table(w, S)[0][0]                   # [C, K], radius row 0
    T, ET2 = service_times(svc, w)
    C, G = w.C, svc.G
    z = np.array(svc.z0, np.int64)
    delta = np.zeros((C, G), np.uint8)
    k = oracle.bcd_init(w).astype(np.int64)
    pi = np.zeros((C, G))
    outer = inner = 0

    def wc(kk):
        return np.array([W1[c, kk[c]] for c in range(C)])

    for _ in range(max_outer):
        outer += 1
        # the wait is linearised once per Block 1, at the state entering it
        Wq = queue(svc, T, ET2, pi, z, memory(svc, T, pi, z, w.eta[k], delta))
        for _ in range(max_inner):
            inner += 1
            pi_new, _ = routing_lp(svc, wc(k), T, Wq, z, w.eta[k], delta)
            conc, cap = lp2_inputs(svc, T, pi_new, z, delta)
            k_new, _ = sweep(W1, w.eta, conc, cap, svc.kappa, k)
            done = np.array_equal(k_new, k) and float(np.max(np.abs(pi_new - pi))) <= PI_TOL
            pi, k = pi_new, k_new
            if done:
                break
        d_new = prefix_cache(svc, T, pi, z)
        z_new, best, _, _ = config_search_vec(svc, wc(k), T, ET2, pi, w.eta[k], d_new)
        if z_new is None:
            z_new = z
        elif feasible(svc, T, pi, z, w.eta[k], d_new):
            if state_objective(svc, wc(k), T, ET2, pi, z, w.eta[k], d_new) == best:
                z_new = z
        stop = np.array_equal(z_new, z) and np.array_equal(d_new, delta)
        z, delta = z_new, d_new
        if stop:
            break
    return dict(z=z, k=k, pi=pi, delta=delta,
                objective=state_objective(svc, wc(k), T, ET2, pi, z, w.eta[k], delta),
                outer=outer, inner=inner, W1=W1, T=T, ET2=ET2)


def config_space_array(svc) -> np.ndarray:
    """Every z in Z as the rows of an int64 array, in lexicographic order
    (the same order as config_space)."""
    G = svc.G
    cost = [int(svc.tau[g]) * int(svc.pp[g]) for g in range(G)]
    out = np.zeros((1, 0), np.int64)      # prefixes (z_0, .., z_{g-1})
    used = np.zeros(1, np.int64)          # their GPU counts
    for g in range(G):
        idx, val = [], []
        for v in range(svc.J // cost[g] + 1):
            i = np.nonzero(used + v * cost[g] <= svc.J)[0]
            idx.append(i)
            val.append(np.full(i.size, v, np.int64))
        idx, val = np.concatenate(idx), np.concatenate(val)
        order = np.lexsort((val, idx))    # each prefix in order, then its z_g ascending
        idx, val = idx[order], val[order]
        out = np.concatenate([out[idx], val[:, None]], axis=1)
        used = used[idx] + val * cost[g]
    return out


def config_search_vec(svc, Wc, T, ET2, pi, eta_c, delta):
    """config_search over every z at once (numpy over z, the same operations
    in the same order per z, so the objectives are bit-identical)."""
    with np.errstate(divide="ignore", invalid="ignore"):
        return _config_search_vec(svc, Wc, T, ET2, pi, eta_c, delta)


def _config_search_vec(svc, Wc, T, ET2, pi, eta_c, delta):
    Z = config_space_array(svc)
    C, G = T.shape
    nz = Z.shape[0]
    kap = 1.0 + float(svc.kappa)
    lam = [float(svc.lam[c]) for c in range(C)]
    # z-independent sums
    used = np.zeros(G)
    pre = np.zeros(G)
    load = np.zeros(G)
    X = np.zeros(G)
    m2 = np.zeros(G)
    route = np.zeros(G, bool)
    for g in range(G):
        u_, p_, l_, x_, m_ = 0.0, 0.0, 0.0, 0.0, 0.0
        for c in range(C):
            rt = float(int(svc.Lin[c]) + int(eta_c[c]) - int(delta[c, g]) * int(svc.Lpre[c]))
            u_ = u_ + lam[c] * T[c, g] * pi[c, g] * rt
            p_ = p_ + float(int(delta[c, g]) * int(svc.Lpre[c]))
            wgt = lam[c] * pi[c, g]
            l_ = l_ + wgt * T[c, g]
            x_ = x_ + wgt
            m_ = m_ + wgt * ET2[c, g]
            route[g] |= pi[c, g] > 0.0
        used[g], pre[g], load[g], X[g], m2[g] = u_, p_, l_, x_, m_
    feas = np.ones(nz, bool)
    Wq = np.zeros((nz, G))
    for g in range(G):
        zg = Z[:, g].astype(np.float64)
        on = Z[:, g] > 0
        if route[g]:
            feas &= on
        mem = kap * (used[g] / zg) + pre[g]
        feas &= ~on | (mem <= float(svc.u_max) * float(svc.Mcap[g]) * MEM_SLACK)
        if X[g] > 0.0:
            u = mem / float(svc.Mcap[g])
            tb = load[g] / X[g]
            cs2 = (m2[g] / X[g]) / (tb * tb) - 1.0
            w = u * (1.0 + cs2) / (2.0 * (1.0 - u)) * tb
            w = np.where(u < 1.0, w, np.inf)
            Wq[:, g] = np.where(on, w, 0.0)
    obj = np.zeros(nz)
    for c in range(C):
        a = 0.0
        gpu = 0.0
        for g in range(G):
            p = pi[c, g]
            a = a + p
            gpu = gpu + p * (float(svc.c_gpu) * float(int(svc.tau[g]) * int(svc.pp[g])) * T[c, g])
        resp = np.zeros(nz)
        for g in range(G):
            resp = resp + pi[c, g] * (Wq[:, g] + T[c, g])
        s = resp - a * float(svc.D[c])
        s = np.where(s < 0.0, 0.0, s)
        term = a * Wc[c] + gpu + float(svc.c_slo) * s + (1.0 - a) * float(svc.c_rej)
        obj = obj + lam[c] * term
    obj = np.where(feas, obj, np.inf)
    nfeas = int(feas.sum())
    if nfeas == 0:
        return None, math.inf, -1, 0
    best = float(obj.min())
    rank = int(np.nonzero(obj == best)[0][0])
    return Z[rank].copy(), best, rank, nfeas
