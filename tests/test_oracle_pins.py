"""Pins of the CPU oracle against the paper and the mathematics (CPU only).

Each test checks the oracle against something that is not the oracle: a
brute-force scan or LP (oracle/brute.py), a closed form the paper states, an
invariance of the definition, or a textbook routine.  The pins are chosen so
that a dropped term, a wrong sign or index, or a transposed operand in
dro_oracle.c fails at least one of them.
"""
import itertools
import math
from fractions import Fraction as F

import numpy as np
import pytest

import oracle
from oracle import brute
from workloads import make_workload, random_workload, lam_grid, eta_grid
from workloads.configs import Workload


def _tiny(seed, C=2, N=(6, 9), L=40, K=9, M=7, E=3, **kw):
    return random_workload(seed=seed, C=C, N=N, L=L, K=K, M=M, E=E, **kw)


# ---------------------------------------------------------------- P1 -------
# Step 4 of Appendix A: the supremum over [0, L] sits at 0, at the sample or
# at L.  The closed form must equal an exhaustive scan of the support.

@pytest.mark.parametrize("seed", range(6))
def test_P1_phi_closed_form_equals_scanned_supremum(seed):
    rng = np.random.default_rng(100 + seed)
    L = int(rng.integers(1, 64))
    for _ in range(60):
        eta = int(rng.integers(0, L + 1))
        x = int(rng.integers(0, L + 1))
        cp = float(np.float32(rng.choice([0.5, 1, 2, 3.25, 8, 17.5, 64.0])))
        cw = float(np.float32(rng.choice([0.25, 0.5, 1, 1.5, 4.0])))
        lam = float(np.float32(rng.choice([0.001, 0.3, 1.0, 2.5, 7.75, 33.0, 100.0])))
        want = brute.sup_brute(eta, x, L, cp, cw, lam, steps=2 * L)
        got_fix = oracle.phi_fix(eta, x, L, cp, cw, lam)
        assert F(got_fix, 1 << 33) == want, (eta, x, L, cp, cw, lam)
        got64 = oracle.phi(eta, x, L, cp, cw, lam)
        assert abs(got64 - float(want)) <= 1e-12 * max(1.0, abs(float(want)))


def test_P1_edges():
    # eta at 0 and at L, samples at 0 and at L, and a multiplier above and below both costs
    L = 10
    for eta in (0, L):
        for x in (0, L, 3):
            for lam in (float(np.float32(v)) for v in (0.001, 1.0, 100.0)):
                want = brute.sup_brute(eta, x, L, 4.0, 1.0, lam, steps=40)
                assert F(oracle.phi_fix(eta, x, L, 4.0, 1.0, lam), 1 << 33) == want


# ---------------------------------------------------------------- P2 -------
# Strong duality (App. A, Step 2) and the LP of App. A, Step 5: the
# transport-plan primal equals the continuous-gamma dual; the grid dual
# (what the path computes) is an upper bound, tight when the grid holds the
# minimising gamma.

@pytest.mark.parametrize("seed", range(5))
def test_P2_primal_lp_equals_dual(seed):
    rng = np.random.default_rng(200 + seed)
    L = int(rng.integers(4, 12))
    N = int(rng.integers(1, 5))
    xs = [int(v) for v in rng.integers(0, L + 1, N)]
    eta = int(rng.integers(0, L + 1))
    cp = float(rng.choice([1.0, 2.0, 5.0, 8.0]))
    cw = float(rng.choice([0.5, 1.0, 2.0]))
    eps = float(rng.choice([0.0, 0.25, 1.0, 2.5]))
    lp = brute.worst_case_lp(eta, xs, L, cp, cw, eps)
    dv, _ = brute.dual_exact(eta, xs, L, cp, cw, eps)
    assert abs(lp - float(dv)) <= 1e-9 * max(1.0, abs(lp))


@pytest.mark.parametrize("seed", range(6))
def test_P2_grid_dual_upper_bound_and_tight_on_breakpoint(seed):
    rng = np.random.default_rng(300 + seed)
    L, N = 24, 5
    xs = np.sort(rng.integers(0, L + 1, N)).astype(np.int32)
    cp, cw = np.float32(rng.choice([2.0, 4.0, 8.0])), np.float32(rng.choice([0.5, 1.0]))
    eps = np.float32(rng.choice([0.5, 2.0, 6.0]))
    eta = eta_grid(7, L)
    lam = lam_grid(9)
    for k in range(eta.size):
        dv, gstar = brute.dual_exact(int(eta[k]), xs.tolist(), L, float(cp), float(cw), float(eps))
        # grid that holds the minimiser (a binary32 value whenever gstar is exact in binary32)
        grids = [lam]
        if gstar > 0 and F(float(np.float32(float(gstar)))) == gstar:
            grids.append(np.unique(np.append(lam, np.float32(float(gstar)))).astype(np.float32))
        for g in grids:
            w = Workload("t", 1, np.array([0, N], np.int64), None, xs, np.array([L], np.int32),
                         eta, g, np.array([cp], np.float32), np.array([cw], np.float32), 1,
                         np.array([eps], np.float32))
            W, _ = oracle.W_table(w, oracle.S_exact(w, grouped=False))
            assert W[0, 0, k] >= float(dv) * (1 - 1e-15)
            if g is not lam:
                assert abs(W[0, 0, k] - float(dv)) <= 1e-13 * max(1.0, float(dv))


# ---------------------------------------------------------------- P3/P4 ----
# Prop. 4.2 at eps = 0: the worst case is the empirical distribution, so the
# cost is the SAA cost and the optimal reservation is the empirical quantile
# at the critical fractile c_p / (c_p + c_w).

@pytest.mark.parametrize("seed", range(4))
def test_P3_eps0_equals_saa(seed):
    w = _tiny(seed, E=1)
    w.eps[:] = 0
    W, _ = oracle.W_table(w, oracle.S_exact(w))
    for c in range(w.C):
        xs = w.samples_of(c).tolist()
        for k in range(w.K):
            want = brute.saa_exact(int(w.eta[k]), xs, float(w.c_p[c]), float(w.c_w[c]))
            # J = RN(RN(S) / N) with S exact: compare against the exact rational
            assert abs(W[0, c, k] - float(want)) <= 2.3e-16 * float(want) + 1e-300


@pytest.mark.parametrize("name", ["lognormal-1x1k", "lognormal-4x100k"])
def test_P4_critical_fractile_brackets_argmin(name):
    w = make_workload(name)
    w.eps[:] = 0
    r = oracle.solve(w)
    for c in range(w.C):
        q = int(r["q_value"][c])
        lo = int(np.searchsorted(w.eta, q, side="right") - 1)   # largest eta <= q
        hi = int(np.searchsorted(w.eta, q, side="left"))        # smallest eta >= q
        assert int(r["k_star"][0, c]) in {lo, hi}


def test_P4_quantile_minimises_saa_on_random_data():
    for seed in range(5):
        w = _tiny(seed, L=60, K=61, E=1)       # grid = every integer: the quantile is a grid point
        w.eps[:] = 0
        r = oracle.solve(w)
        for c in range(w.C):
            assert w.eta[r["k_star"][0, c]] == r["q_value"][c]


# ---------------------------------------------------------------- P5/P6 ----
# Appendix structure: for gamma >= max(c_p, c_w) every sample keeps its own
# point, so S equals the SAA sum; when eps <= D(eta) the continuous dual is
# max(c_p, c_w) eps + SAA.

@pytest.mark.parametrize("seed", range(4))
def test_P5_large_multiplier_gives_saa_sum(seed):
    w = _tiny(seed, E=1)
    S = oracle.S_exact(w)
    for c in range(w.C):
        xs = w.samples_of(c).tolist()
        top = max(float(w.c_p[c]), float(w.c_w[c]))
        for k in range(w.K):
            saa_sum = brute.saa_exact(int(w.eta[k]), xs, float(w.c_p[c]), float(w.c_w[c])) * len(xs)
            for m in range(w.M):
                if float(w.lam[m]) >= top:
                    assert F(S.as_int((c, k, m)), 1 << 33) == saa_sum


def _D(eta, xs, L, cp, cw):
    if cp >= cw:
        return sum((F(L - x) for x in xs if eta <= x < L), F(0)) / len(xs)
    return sum((F(x) for x in xs if 0 < x <= eta), F(0)) / len(xs)


@pytest.mark.parametrize("seed", range(4))
def test_P5_small_radius_identity(seed):
    rng = np.random.default_rng(500 + seed)
    L = 30
    xs = [int(v) for v in rng.integers(0, L + 1, 6)]
    cp, cw = float(rng.choice([2.0, 4.0, 0.5])), float(rng.choice([1.0, 0.25]))
    for eta in range(0, L + 1, 5):
        D = _D(eta, xs, L, cp, cw)
        for eps in (F(0), D / 3, D):
            dv, _ = brute.dual_exact(eta, xs, L, cp, cw, eps)
            assert dv == max(F(cp), F(cw)) * eps + brute.saa_exact(eta, xs, cp, cw)


@pytest.mark.parametrize("seed", range(4))
def test_P6_bounds(seed):
    w = _tiny(seed)
    r = oracle.solve(w)
    W = r["W"]
    for e in range(w.E):
        for c in range(w.C):
            xs = w.samples_of(c).tolist()
            eps = float(w.eps[e * w.C + c])
            for k in range(w.K):
                eta = int(w.eta[k])
                saa = float(brute.saa_exact(eta, xs, float(w.c_p[c]), float(w.c_w[c])))
                tol = 1e-12 * max(1.0, saa)
                assert W[e, c, k] >= saa - tol
                assert W[e, c, k] <= float(w.lam[-1]) * eps + saa + tol
                hi2 = float(w.lam[0]) * eps + max(float(w.c_w[c]) * eta,
                                                  float(w.c_p[c]) * (int(w.L[c]) - eta))
                assert W[e, c, k] <= hi2 + tol


# ---------------------------------------------------------------- P7 -------
# W is non-decreasing and concave in eps (a min over m of lines in eps with
# slopes lam_m >= 0); with J = RN(lam*eps) + fixed RN(S/N) the monotonicity
# holds bit for bit.

def test_P7_monotone_concave_in_radius():
    w = _tiny(11, E=1, N=(40, 25))
    S = oracle.S_exact(w)
    radii = np.linspace(0, 12, 25).astype(np.float32)
    rows = []
    for r in radii:
        Wr, _ = oracle.W_table(w, S, eps=np.full(w.C, r, np.float32), E=1)
        rows.append(Wr[0])
    rows = np.array(rows)                       # [R, C, K]
    assert np.all(np.diff(rows, axis=0) >= 0)
    second = rows[2:] - 2 * rows[1:-1] + rows[:-2]
    assert np.all(second <= 1e-9 * np.abs(rows[1:-1]).max())


# ---------------------------------------------------------------- P8-P10 ---

def test_P8_power_of_two_scaling_is_exact():
    w = _tiny(21, lam_lo=0.01)          # keeps lam * 2^-3 inside the exact range
    base = oracle.solve(w)
    for s in (-3, 2):
        f = np.float32(2.0 ** s)
        w2 = _tiny(21, lam_lo=0.01)
        w2.c_p = (w.c_p * f).astype(np.float32)
        w2.c_w = (w.c_w * f).astype(np.float32)
        w2.lam = (w.lam * f).astype(np.float32)
        r2 = oracle.solve(w2)
        assert np.array_equal(r2["W"], base["W"] * float(f))
        assert np.array_equal(r2["k_star"], base["k_star"])
        assert np.array_equal(r2["m_star"], base["m_star"])
        assert np.array_equal(r2["q_value"], base["q_value"])


def test_P9_permutation_invariance():
    w = _tiny(31, N=(30, 17))
    base = oracle.solve(w)
    rng = np.random.default_rng(0)
    w2 = _tiny(31, N=(30, 17))
    for c in range(w2.C):
        a, b = w2.offsets[c], w2.offsets[c + 1]
        w2.xi[a:b] = rng.permutation(w2.xi[a:b])
    r2 = oracle.solve(w2, grouped=False)
    for key in ("W", "k_star", "m_star", "W_star", "q_value", "q_rank"):
        assert np.array_equal(r2[key], base[key]), key


def test_P10_segment_reorder_and_alias():
    w = _tiny(41, C=3, N=(12, 20, 7))
    base = oracle.solve(w)
    # reorder segments in memory and alias two extra classes onto existing segments
    order = [2, 0, 1]
    parts = [w.samples_of(c) for c in order]
    off = np.zeros(4, np.int64)
    off[1:] = np.cumsum([len(p) for p in parts])
    seg = np.array([order.index(c) for c in range(3)] + [order.index(1), order.index(0)], np.int32)
    ext = [0, 1, 2, 1, 0]
    w2 = Workload("alias", 5, off, seg, np.concatenate(parts).astype(np.int32),
                  np.full(5, w.L[0], np.int32), w.eta, w.lam,
                  w.c_p[ext].astype(np.float32), w.c_w[ext].astype(np.float32), w.E,
                  np.concatenate([w.eps[e * 3:(e + 1) * 3][ext] for e in range(w.E)]).astype(np.float32))
    r2 = oracle.solve(w2)
    for e in range(w.E):
        for c2, c in enumerate(ext):
            assert np.array_equal(r2["W"][e, c2], base["W"][e, c])
            assert r2["k_star"][e, c2] == base["k_star"][e, c]
    assert np.array_equal(r2["q_value"], base["q_value"][ext])


# ---------------------------------------------------------------- P11 ------
# Generalized inverse of the empirical CDF: the ceil(qN)-th order statistic.

def test_P11_rank_is_exact():
    rng = np.random.default_rng(7)
    for _ in range(400):
        cp = np.float32(np.exp(rng.uniform(-6, 4.8)))
        cw = np.float32(np.exp(rng.uniform(-6, 4.8)))
        N = int(rng.integers(1, 1 << 26))
        assert oracle.rank(cp, cw, N) == brute.rank_exact(float(cp), float(cw), N)
    # q N an integer: rho = 4 with N = 100000 gives j = 80000 exactly
    assert oracle.rank(4.0, 1.0, 100000) == 80000
    assert oracle.rank(8.0, 1.0, 9) == 8


@pytest.mark.parametrize("name", ["lognormal-1x1k", "lognormal-4x100k"])
def test_P11_quantile_matches_partition(name):
    w = make_workload(name)
    qv, qr = oracle.quantile(w)
    for c in range(w.C):
        x = w.samples_of(c)
        j = brute.rank_exact(float(w.c_p[c]), float(w.c_w[c]), len(x))
        assert qr[c] == j
        assert qv[c] == np.partition(x, j - 1)[j - 1]


# ---------------------------------------------------------------- P12 ------
# Two independent summations: dense fp64 in sample order vs exact integers.

def test_P12_dense_f64_matches_exact():
    for w in (make_workload("lognormal-1x1k"), _tiny(51, N=(300, 41), L=900, K=33, M=17)):
        d = oracle.S_f64(w)
        x = oracle.S_exact(w).to_double()
        assert np.max(np.abs(d - x) / np.maximum(x, 1e-300)) <= 1e-12


def test_P12_grouped_equals_per_sample():
    w = _tiny(61, N=(80, 33))
    a, b = oracle.S_exact(w, grouped=True), oracle.S_exact(w, grouped=False)
    assert np.array_equal(a.hi, b.hi) and np.array_equal(a.lo, b.lo)


def test_P12_exact_at_equals_the_full_exact_sums():
    """oracle_S_exact_at (the reference of every full-size spot check of S)
    against the full per-sample and value-grouped sums at 300 random
    (c, k, m): aliased segments, a segment of one sample, K, M > 1."""
    w = random_workload(seed=71, C=7, N=(1, 250, 37, 900), alias=True, L=3000, K=41, M=23, E=1)
    assert w.seg is not None and min(np.diff(w.offsets)) == 1
    full = oracle.S_exact(w, grouped=False)
    grouped = oracle.S_exact(w, grouped=True)
    rng = np.random.default_rng(0)
    cs, ks, ms = rng.integers(0, w.C, 300), rng.integers(0, w.K, 300), rng.integers(0, w.M, 300)
    cs[:4] = [c for c in range(w.C) if w.seg[c] == 0][:1] * 4     # the one-sample segment
    at = oracle.S_exact_at(w, cs, ks, ms)
    for i, (c, k, m) in enumerate(zip(cs, ks, ms)):
        assert at.as_int(i) == full.as_int((c, k, m)) == grouped.as_int((c, k, m)), (c, k, m)


def test_P12_exact_at_equals_the_scanned_supremum_summed_in_rationals():
    """oracle_S_exact_at against the sum over the samples of the supremum of
    Step 4 found by scanning the support (brute.sup_brute), in rationals."""
    w = _tiny(72, C=3, N=(5, 1, 8), L=60, K=7, M=5)
    rng = np.random.default_rng(1)
    cs, ks, ms = rng.integers(0, w.C, 24), rng.integers(0, w.K, 24), rng.integers(0, w.M, 24)
    at = oracle.S_exact_at(w, cs, ks, ms)
    for i, (c, k, m) in enumerate(zip(cs, ks, ms)):
        xs = w.samples_of(int(c))
        want = sum((brute.sup_brute(int(w.eta[k]), int(x), int(w.L[c]), float(w.c_p[c]),
                                    float(w.c_w[c]), float(w.lam[m])) for x in xs), F(0))
        assert F(at.as_int(i), 1 << 33) == want, (c, k, m)


def test_fix_to_double_array_equals_the_scalar():
    rng = np.random.default_rng(4)
    hi = rng.integers(0, 1 << 20, 500).astype(np.int64)
    lo = rng.integers(0, 1 << 63, 500, dtype=np.uint64) * np.uint64(2) + np.uint64(1)
    got = oracle.ExactS(hi, lo).to_double()
    for i in range(500):
        assert got[i] == oracle._load().oracle_fix_to_double(int(hi[i]), int(lo[i]))


def test_fix_to_double_is_correctly_rounded():
    rng = np.random.default_rng(3)
    for _ in range(2000):
        bits = int(rng.integers(1, 82))
        v = int(rng.integers(0, 1 << 62)) << max(0, bits - 62) | int(rng.integers(0, 1 << 20))
        v &= (1 << bits) - 1
        hi, lo = v >> 64, v & ((1 << 64) - 1)
        want = float(F(v, 1 << 33))        # Python rounds rationals to nearest, ties to even
        assert oracle._load().oracle_fix_to_double(hi, lo) == want
    # a tie exactly halfway between two doubles rounds to even
    v = (1 << 60) + (1 << 7)               # 2^60 + 2^7: halfway at 53-bit precision
    assert oracle._load().oracle_fix_to_double(v >> 64, v & ((1 << 64) - 1)) == float(F(v, 1 << 33))


# ---------------------------------------------------------------- P13 ------
# The block step: each class takes the exact best grid point that keeps every
# group it is routed to within capacity (the memory-capacity constraint of Sec. 3.4), given the others;
# the sweep never increases the summed cost from a feasible start.

def _feasible_kmax_exact(w, c, kcur):
    g = w.groups
    G = g.G
    one_k = 1 + F(float(np.float32(g.kappa)))
    best = None
    for gg in range(G):
        u = F(float(g.conc[c * G + gg]))
        if u <= 0:
            continue
        other = one_k * sum((F(float(g.conc[c2 * G + gg])) * int(w.eta[kcur[c2]])
                             for c2 in range(w.C) if c2 != c), F(0))
        b = (F(float(g.cap[gg])) - other) / (one_k * u)
        best = b if best is None or b < best else best
    ks = [k for k in range(w.K) if best is None or w.eta[k] <= best]
    return (max(ks), True) if ks else (0, False)


@pytest.mark.parametrize("seed", range(6))
def test_P13_block_step_is_exact_coordinate_minimisation(seed):
    w = random_workload(seed=700 + seed, C=3, N=(20, 9, 14), L=50, K=8, M=9, E=1,
                        with_groups=True, G=2)
    S = oracle.S_exact(w)
    W, _ = oracle.W_table(w, S)
    k0 = oracle.bcd_init(w)
    for c in range(w.C):
        mean = F(int(w.samples_of(c).astype(np.int64).sum()), w.n_of(c))
        assert w.eta[k0[c]] <= mean and (k0[c] == w.K - 1 or w.eta[k0[c] + 1] > mean)
    out = oracle.bcd_step(w, W[0], k0)
    kcur = list(k0)
    for c in range(w.C):
        kmax, feas = _feasible_kmax_exact(w, c, kcur)
        assert bool(out["feasible"][c]) == feas
        want = min(range(kmax + 1), key=lambda k: (W[0, c, k], k))
        assert out["k_next"][c] == want
        kcur[c] = want
    # monotone decrease within a sweep from a feasible start
    if all(out["feasible"]):
        out2 = oracle.bcd_step(w, W[0], out["k_next"])
        s1 = sum(W[0, c, out["k_next"][c]] for c in range(w.C))
        s2 = sum(W[0, c, out2["k_next"][c]] for c in range(w.C))
        assert s2 <= s1 + 1e-12 * abs(s1)
    G = w.groups.G
    for gg in range(G):
        u = (1 + float(np.float32(w.groups.kappa))) * sum(
            float(w.groups.conc[c * G + gg]) * int(w.eta[out["k_next"][c]]) for c in range(w.C))
        assert abs(out["usage"][gg] - u) <= 1e-12 * max(1.0, u)


# ---------------------------------------------------------------- P14 ------
# Printed consequences of Prop. 4.2 (Sec. 5): rho = 10 reserves at about the
# 91st percentile; rho = 20 at the 95th (Table 2: DRO equals P95 at rho = 20).

def test_P14_paper_fractiles():
    import json, os
    path = os.path.join(os.path.dirname(__file__), "golden", "critical_fractile.json")
    data = json.load(open(path))
    N = 100_000
    for row in data["rows"]:
        rho = row["rho"]
        j = oracle.rank(np.float32(rho), np.float32(1.0), N)
        q = j / N
        assert abs(q - row["q_star"]) <= 1.0 / N
        if "printed_percentile" in row:
            assert round(100 * q) == row["printed_percentile"]


# ---------------------------------------------------------------- ties -----
# Ties go to the lowest index.  Exact ties are structural: at eps = 0 every
# multiplier at or above max(c_p, c_w) gives the SAA cost, and when q N is an
# integer the SAA cost is flat between two order statistics.

def test_ties_lowest_reservation_on_flat_saa():
    xs = np.array([3, 9, 14, 20, 26, 31, 37, 44, 52, 60], np.int32)   # q = 4/5, q N = 8
    L = 64
    w = Workload("tie", 1, np.array([0, xs.size], np.int64), None, xs, np.array([L], np.int32),
                 eta_grid(L + 1, L), lam_grid(9), np.array([4.0], np.float32),
                 np.array([1.0], np.float32), 1, np.array([0.0], np.float32))
    r = oracle.solve(w)
    saa = [brute.saa_exact(int(e), xs.tolist(), 4.0, 1.0) for e in w.eta]
    best = min(saa)
    flat = [k for k, v in enumerate(saa) if v == best]
    assert len(flat) > 1                                   # the flat stretch [x_(8), x_(9)]
    assert r["k_star"][0, 0] == flat[0] == 44
    assert r["q_value"][0] == 44 and r["q_rank"][0] == 8


def test_ties_lowest_multiplier():
    w = _tiny(81, E=1, N=(25, 12))
    w.eps[:] = 0
    r = oracle.solve(w)
    S = r["S"]
    for c in range(w.C):
        xs = w.samples_of(c).tolist()
        for k in range(w.K):
            target = brute.saa_exact(int(w.eta[k]), xs, float(w.c_p[c]), float(w.c_w[c])) * len(xs)
            first = next(m for m in range(w.M) if F(S.as_int((c, k, m)), 1 << 33) == target)
            assert r["m_star"][0, c, k] == first


# --------------------------------------------------------------- P15-P17 ---
# Reservation cost (the per-arrival cost of Sec. 3.3 averaged over samples)
# and per-class moments, used to price reservation policies against each other.

@pytest.mark.parametrize("seed", range(5))
def test_P15_reservation_cost_equals_rational_average(seed):
    w = _tiny(200 + seed, C=3, N=(7, 1, 12), L=50)
    rng = np.random.default_rng(seed)
    eta = rng.integers(-5, 60, size=(6, w.C)).astype(np.int32)   # also below 0 and above L
    cost, cover, S = oracle.reservation_cost(w, eta)
    for r in range(eta.shape[0]):
        for c in range(w.C):
            xs = [int(v) for v in w.samples_of(c)]
            cp, cw = float(w.c_p[c]), float(w.c_w[c])
            want = brute.saa_exact(int(eta[r, c]), xs, cp, cw)
            assert S.as_int((r, c)) == want * len(xs) * (1 << 33)
            assert cost[r, c] == float(want * len(xs)) / len(xs)   # RN(RN(S) / N)
            assert cover[r, c] == sum(1 for x in xs if x <= eta[r, c])


def test_P15_closed_forms_at_the_ends():
    w = _tiny(210, C=2, N=(40, 25), L=200)
    m = oracle.moments(w)
    top = int(w.L.max()) + 7
    cost, cover, S = oracle.reservation_cost(w, np.array([[0, 0], [top, top]], np.int32))
    for c in range(w.C):
        n, s = int(m["count"][c]), int(m["sum"][c])
        cp, cw = F(float(w.c_p[c])), F(float(w.c_w[c]))
        assert F(S.as_int((0, c)), 1 << 33) == cp * s            # nothing reserved: all preempted
        assert F(S.as_int((1, c)), 1 << 33) == cw * (top * n - s)  # above every sample: all waste
        assert cover[0, c] == sum(1 for x in w.samples_of(c) if x <= 0) and cover[1, c] == n


@pytest.mark.parametrize("seed", range(4))
def test_P16_quantile_is_the_smallest_cost_minimiser(seed):
    # Prop. 4.2 at eps = 0: the generalized-inverse quantile at c_p/(c_p+c_w)
    # is the smallest integer reservation of least average cost.
    w = _tiny(220 + seed, C=3, N=(31, 9, 57), L=90)
    qv, _ = oracle.quantile(w)
    L = int(w.L.max())
    eta = np.repeat(np.arange(0, L + 1, dtype=np.int32)[:, None], w.C, axis=1)
    _, _, S = oracle.reservation_cost(w, eta)
    for c in range(w.C):
        vals = [S.as_int((r, c)) for r in range(L + 1)]
        best = min(vals)
        assert vals.index(best) == qv[c]


def test_P17_cost_slope_is_the_coverage_balance():
    # S(eta + 1) - S(eta) = c_w #{x <= eta} - c_p #{x > eta}: ties the cost to cover.
    w = _tiny(230, C=2, N=(33, 18), L=70)
    eta = np.repeat(np.arange(-2, 74, dtype=np.int32)[:, None], w.C, axis=1)
    _, cover, S = oracle.reservation_cost(w, eta)
    for c in range(w.C):
        n = w.n_of(c)
        CP, CW = F(float(w.c_p[c])) * (1 << 33), F(float(w.c_w[c])) * (1 << 33)
        for r in range(eta.shape[0] - 1):
            d = S.as_int((r + 1, c)) - S.as_int((r, c))
            assert d == CW * int(cover[r, c]) - CP * (n - int(cover[r, c]))


def test_P17_moments_match_numpy():
    w = random_workload(seed=240, C=3, N=(50, 1, 77), L=32768)
    m = oracle.moments(w)
    for c in range(w.C):
        x = w.samples_of(c).astype(np.int64)
        assert m["count"][c] == x.size and m["sum"][c] == x.sum()
        assert m["sumsq"][c] == (x * x).sum() and m["xmax"][c] == x.max()


# --------------------------------------------------------------- P18-P19 ---
# The policy comparison (Sec. 5.1-5.4): baseline reservations by their plain
# definitions, and the structure Prop. 4.2 puts on the table.

def _policy_tiny(seed=0):
    from workloads import policy_workloads
    return policy_workloads(n_train=3000, n_eval=2000, rhos=(2, 10, 100), shifts=(1.0, 2.0),
                            eps_fracs=(0.0, 0.15), L=600, K=601, M=48, seed=seed)


def test_P18_baseline_reservations_by_definition():
    from oracle import policies
    tr, _ = _policy_tiny(1)
    eta = policies.reservations(tr, (0.0, 0.15))
    names = policies.policy_names((0.0, 0.15))
    x = np.sort(tr.samples_of(0).astype(np.int64))
    n = x.size
    row = {nm: eta[i] for i, nm in enumerate(names)}
    assert np.all(row["P90"] == x[(9 * n + 9) // 10 - 1])          # rank ceil(0.9 n)
    assert np.all(row["P99"] == x[(99 * n + 99) // 100 - 1])
    p95 = x[(19 * n + 19) // 20 - 1]
    assert np.all(row["P95"] == ((p95 + 15) // 16) * 16)
    assert np.all(row["Mean"] == -(-x.sum() // n))
    assert np.all(row["Max"] == 600)
    mu = x.mean()
    sd = x.std()          # population standard deviation
    for k in (1, 2):
        r = row[f"LP+{k}sigma"][0]
        assert r - 1 < mu + k * sd + 1e-9 and r >= mu + k * sd - 1e-9
    # SAA is the critical-fractile quantile at rho/(rho+1) (Prop. 4.2)
    for c, rho in enumerate((2, 10, 100)):
        assert row["SAA"][c] == x[-(-rho * n // (rho + 1)) - 1]


def test_P19_table_structure():
    from oracle import policies
    tr, ev = _policy_tiny(2)
    t = policies.table(tr, ev, (0.0, 0.15))
    names = t["names"]
    i_dro0, i_saa, i_max = names.index("DRO(eps=0*mean)"), names.index("SAA"), names.index("Max")
    # on an every-integer grid the eps = 0 DRO reservation is the SAA quantile
    assert np.array_equal(t["eta"][i_dro0], t["eta"][i_saa])
    # in sample, SAA has the least cost of all policies (Prop. 4.2)
    assert np.all(t["cost_train"][i_saa][None, :] <= t["cost_train"])
    # reserving L costs exactly c_w (L - mean) on every shifted set
    for s in range(ev.C // tr.C):
        xs = ev.samples_of(s * tr.C).astype(np.int64)
        assert t["cost"][i_max, s, 0] == float(F(600 * xs.size - int(xs.sum()), xs.size))
        assert np.all(t["cover"][i_max, s] == xs.size)


# --------------------------------------------------------------- P20-P24 ---
# The serving-model oracle (oracle/serving.py) of the rest of Alg. 1.

def _serving_tiny(seed, C=3, J=8, configs=((1, 1), (2, 1), (2, 2))):
    from workloads.configs import serving_workload
    return serving_workload(C=C, N=400, J=J, L=600, K=61, M=12, seed=seed, configs=list(configs))


def test_P20_waiting_time_reduces_to_mm1():
    # Pollaczek-Khinchin with exponential service (second moment 2 T^2, Cs2 = 1)
    # is the M/M/1 wait u T / (1 - u).
    from oracle import serving as osv
    w, svc = _serving_tiny(1)
    T, _ = osv.service_times(svc, w)
    ET2 = 2.0 * T * T
    pi = np.zeros((w.C, svc.G))
    pi[0, :] = 0.3                     # one class per group: a single exponential
    z = np.ones(svc.G, np.int64)
    mem = np.array([0.3, 0.6, 0.9]) * svc.Mcap.astype(np.float64)
    Wq = osv.queue(svc, T, ET2, pi, z, mem)
    for g in range(svc.G):
        lam = svc.lam.astype(np.float64)
        tb = float((lam * pi[:, g] * T[:, g]).sum() / (lam * pi[:, g]).sum())
        u = mem[g] / float(svc.Mcap[g])
        assert Wq[g] == pytest.approx(u * tb / (1.0 - u), rel=1e-12)


def test_P21_prefix_caching_saves_memory_exactly_when_concurrency_exceeds_the_margin():
    # Caching class c's prefix on g changes mem_g by Lpre (1 - (1 + kappa) conc_cg):
    # it saves memory iff (1 + kappa) conc_cg > 1 (Block 2 caches at conc > 1).
    from oracle import serving as osv
    w, svc = _serving_tiny(2)
    T, _ = osv.service_times(svc, w)
    rng = np.random.default_rng(2)
    pi = rng.uniform(0.0, 0.5, (w.C, svc.G))
    z = np.array([1, 2, 1], np.int64)
    eta_c = rng.integers(0, 300, w.C)
    d0 = np.zeros((w.C, svc.G), np.uint8)
    conc = osv.concurrency(svc, T, pi, z)
    for c in range(w.C):
        for g in range(svc.G):
            d1 = d0.copy()
            d1[c, g] = 1
            diff = osv.memory(svc, T, pi, z, eta_c, d1)[g] - osv.memory(svc, T, pi, z, eta_c, d0)[g]
            want = float(svc.Lpre[c]) * (1.0 - (1.0 + float(svc.kappa)) * conc[c, g])
            assert diff == pytest.approx(want, rel=1e-9, abs=1e-9)


def test_P22_routing_lp_beats_every_sampled_feasible_routing():
    from oracle import serving as osv
    w, svc = _serving_tiny(3)
    T, ET2 = osv.service_times(svc, w)
    z = np.array([2, 1, 1], np.int64)
    eta_c = np.array([50, 120, 300])
    delta = np.zeros((w.C, svc.G), np.uint8)
    Wq = np.array([0.2, 0.5, 1.0])
    Wc = np.array([300.0, 900.0, 2500.0])
    pi, obj = osv.routing_lp(svc, Wc, T, Wq, z, eta_c, delta)

    def lp_obj(p):
        tot = 0.0
        for c in range(w.C):
            lin = sum(p[c, g] * (Wc[c] + float(svc.c_gpu) * float(svc.tau[g] * svc.pp[g]) * T[c, g]
                                 - float(svc.c_rej)) for g in range(svc.G))
            h = sum(p[c, g] * (Wq[g] + T[c, g] - float(svc.D[c])) for g in range(svc.G))
            tot += float(svc.lam[c]) * (lin + float(svc.c_slo) * max(h, 0.0) + float(svc.c_rej))
        return tot

    assert lp_obj(pi) == pytest.approx(obj, rel=1e-9)
    assert np.all(pi.sum(axis=1) <= 1 + 1e-9)
    assert np.all(osv.memory(svc, T, pi, z, eta_c, delta) <= float(svc.u_max) * svc.Mcap * (1 + 1e-9))
    rng = np.random.default_rng(3)
    lim = float(svc.u_max) * svc.Mcap.astype(np.float64)
    for _ in range(400):
        p = rng.dirichlet(np.ones(svc.G + 1), w.C)[:, :svc.G]
        mem = osv.memory(svc, T, p, z, eta_c, delta)
        if np.all(mem <= lim):
            assert obj <= lp_obj(p) + 1e-9 * abs(obj)


@pytest.mark.parametrize("seed", range(3))
def test_P23_configuration_search_equals_brute_force(seed):
    # the vectorised scan (numpy over z) against the plain loop over
    # itertools.product: the same minimiser, objective bits, rank and count
    from oracle import serving as osv
    w, svc = _serving_tiny(10 + seed, C=4, J=12)
    T, ET2 = osv.service_times(svc, w)
    rng = np.random.default_rng(seed)
    pi = rng.dirichlet(np.ones(svc.G + 1), w.C)[:, :svc.G] * 0.4
    delta = (rng.random((w.C, svc.G)) < 0.3).astype(np.uint8)
    eta_c = rng.integers(0, 200, w.C)
    Wc = rng.uniform(50, 2000, w.C)
    a = osv.config_search(svc, Wc, T, ET2, pi, eta_c, delta)
    b = osv.config_search_vec(svc, Wc, T, ET2, pi, eta_c, delta)
    assert np.array_equal(a[0], b[0]) and a[1] == b[1] and a[2] == b[2] and a[3] == b[3]
    # the count of Z is the number of z with sum z_g tau_g pp_g <= J
    n = sum(1 for _ in itertools.product(*[range(svc.J // int(svc.tau[g] * svc.pp[g]) + 1)
                                         for g in range(svc.G)])
            if sum(zz * int(svc.tau[g] * svc.pp[g]) for g, zz in enumerate(_)) <= svc.J)
    assert osv.config_space_array(svc).shape[0] == n


@pytest.mark.parametrize("seed", range(3))
def test_P24_sweep_agrees_with_the_block_step(seed):
    # the fp64 sweep of LP2 and the oracle's block step (pinned by P13) on the
    # same float32-representable capacities and concurrencies
    from oracle import serving as osv
    from workloads.configs import Groups
    w = _tiny(900 + seed, C=4, N=(60, 31, 90, 77), L=600, K=33, M=9, E=1, with_groups=True, G=3)
    S = oracle.S_exact(w)
    W = oracle.W_table(w, S)[0][0]
    k_prev = oracle.bcd_init(w)
    o = oracle.bcd_step(w, W, k_prev)
    conc = w.groups.conc.astype(np.float64).reshape(w.C, -1)
    k, ok = osv.sweep(W, w.eta, conc, w.groups.cap.astype(np.float64), w.groups.kappa, k_prev)
    assert np.array_equal(k, o["k_next"]) and np.array_equal(ok, o["feasible"].astype(bool))


@pytest.mark.parametrize("seed", [6, 7])
def test_P24_alg1_ends_blockwise_optimal(seed):
    # Prop. 4.3: at termination no block improves on its own: Block 3 keeps z,
    # Block 2 reproduces delta, and the reservations are a fixed point of LP2.
    from oracle import serving as osv
    from workloads.configs import serving_workload
    w, svc = serving_workload(C=4, N=2000, J=12, K=129, M=16, seed=seed,
                              configs=[(1, 1), (2, 1), (4, 1), (2, 2)])
    r = osv.solve(w, svc, max_outer=20)
    if r["outer"] >= 20:
        pytest.skip("the loop did not terminate on this instance")
    T, ET2 = r["T"], r["ET2"]
    Wc = np.array([r["W1"][c, r["k"][c]] for c in range(w.C)])
    eta_c = w.eta[r["k"]]
    assert np.array_equal(osv.prefix_cache(svc, T, r["pi"], r["z"]), r["delta"])
    zb, best, _, _ = osv.config_search_vec(svc, Wc, T, ET2, r["pi"], eta_c, r["delta"])
    assert osv.state_objective(svc, Wc, T, ET2, r["pi"], r["z"], eta_c, r["delta"]) == best
    conc, cap = osv.lp2_inputs(svc, T, r["pi"], r["z"], r["delta"])
    k2, _ = osv.sweep(r["W1"], w.eta, conc, cap, svc.kappa, r["k"])
    assert np.array_equal(k2, r["k"])


def test_P24_sweep_takes_the_lowest_minimiser_on_ties():
    # a flat table: every grid point is a minimiser, the lowest one is taken
    # (the tie rule of the reservation argmin), and a binding bound caps it
    from oracle import serving as osv
    W = np.zeros((2, 9))
    eta = np.arange(0, 90, 10)
    conc = np.array([[1.0], [0.0]])
    k, ok = osv.sweep(W, eta, conc, np.array([1000.0]), 0.0, np.array([8, 8]))
    assert k.tolist() == [0, 0] and ok.all()
    W[0, :] = [5, 5, 3, 3, 3, 4, 1, 1, 2]
    k, ok = osv.sweep(W, eta, conc, np.array([1000.0]), 0.0, np.array([0, 0]))
    assert k[0] == 6                                   # lowest of the tied minima
    k, ok = osv.sweep(W, eta, conc, np.array([45.0]), 0.0, np.array([0, 0]))
    assert k[0] == 2                                   # eta <= 45: grid points 0..4


def test_P21_block2_caches_exactly_where_caching_saves_memory_at_zero_margin():
    # with kappa = 0, caching the prefix of (c, g) lowers the memory of g iff
    # conc_cg > 1, which is Block 2's rule
    from dataclasses import replace
    from oracle import serving as osv
    w, svc = _serving_tiny(5)
    svc = replace(svc, kappa=0.0)
    T, _ = osv.service_times(svc, w)
    z = np.array([1, 1, 2], np.int64)
    # routings that give the concurrencies 0.3 .. 2.5 (some just below and above 1)
    target = np.array([0.3, 0.6, 0.9, 0.99, 1.01, 1.2, 1.6, 2.0, 2.5]).reshape(w.C, svc.G)
    pi = target * z[None, :] / (svc.lam.astype(np.float64)[:, None] * T)
    eta_c = np.zeros(w.C, np.int64)
    d0 = np.zeros((w.C, svc.G), np.uint8)
    delta = osv.prefix_cache(svc, T, pi, z)
    for c in range(w.C):
        for g in range(svc.G):
            d1 = d0.copy()
            d1[c, g] = 1
            saves = osv.memory(svc, T, pi, z, eta_c, d1)[g] < osv.memory(svc, T, pi, z, eta_c, d0)[g]
            assert bool(delta[c, g]) == saves, (c, g)
    assert 0 < delta.sum() < delta.size


def test_P18_mean_plus_spread_on_a_hand_worked_sample():
    # samples 1, 2, 3, 10: mean 4, population variance 12.5, sigma 3.5355...:
    # LP+1sigma = ceil(7.5355) = 8, LP+2sigma = ceil(11.071) = 12, Mean = 4
    from oracle import policies
    from workloads.configs import Workload
    xs = np.array([1, 2, 3, 10], np.int32)
    w = Workload("hand", 1, np.array([0, 4], np.int64), None, xs, np.array([20], np.int32),
                 np.arange(21, dtype=np.int32), np.array([1.0], np.float32),
                 np.array([10.0], np.float32), np.array([1.0], np.float32), 1,
                 np.array([0.0], np.float32))
    eta = policies.reservations(w, (0.0,))
    row = dict(zip(policies.policy_names((0.0,)), eta[:, 0]))
    assert row["Mean"] == 4 and row["LP+1sigma"] == 8 and row["LP+2sigma"] == 12
    assert row["P90"] == 10 and row["Max"] == 20     # ceil(0.9 * 4) = 4th smallest


# ---- P25-P28: the serving oracle's arithmetic against its formulas in exact
# rationals, written in a different algebraic form (per sample value instead of
# expanded moments, the textbook E[S^2] / (2 E[S]) form of the P-K wait), so a
# dropped term, a wrong sign or divisor, or a swapped index fails whatever the
# operation order of the fp64 code.

def _q(v):
    return F(float(v))


def _close(a, b, rel):
    a, b = F(float(a)), F(b)
    return abs(a - b) <= F(rel) * max(abs(b), F(1, 10 ** 30))


@pytest.mark.parametrize("seed", [31, 32])
def test_P25_service_time_moments_in_rationals(seed):
    # Sec. 3.1: on configuration g a request of class c with output length x
    # takes A + B x, A = pp alpha Lin / Cc + NL tau t_ar, B = beta / Bc; T and ET2
    # are its mean and second moment over the class's samples
    from oracle import serving as osv
    w, svc = _serving_tiny(seed)
    T, ET2 = osv.service_times(svc, w)
    for c in range(w.C):
        vals, cnt = np.unique(w.samples_of(c), return_counts=True)
        n = int(cnt.sum())
        for g in range(svc.G):
            A = (_q(svc.pp[g]) * _q(svc.alpha) * _q(svc.Lin[c]) / _q(svc.Cc[g])
                 + _q(svc.NL) * _q(svc.tau[g]) * _q(svc.t_ar))
            B = _q(svc.beta) / _q(svc.Bc[g])
            t = sum(int(m) * (A + B * int(v)) for v, m in zip(vals, cnt)) / n
            t2 = sum(int(m) * (A + B * int(v)) ** 2 for v, m in zip(vals, cnt)) / n
            assert _close(T[c, g], t, 1e-14), (c, g)
            assert _close(ET2[c, g], t2, 1e-14), (c, g)


def test_P26_concurrency_and_memory_in_rationals():
    # Little's law conc = lam T pi / z, and the KV tokens of Sec. 3.4:
    # mem = (1 + kappa) sum_c conc_cg (Lin_c + eta_c - delta_cg Lpre_c) + sum_c delta_cg Lpre_c
    from oracle import serving as osv
    w, svc = _serving_tiny(33)
    T, _ = osv.service_times(svc, w)
    rng = np.random.default_rng(33)
    pi = rng.uniform(0.0, 0.5, (w.C, svc.G))
    z = np.array([1, 3, 2], np.int64)
    eta_c = rng.integers(0, 600, w.C)
    delta = (rng.random((w.C, svc.G)) < 0.5).astype(np.uint8)
    conc = osv.concurrency(svc, T, pi, z)
    mem = osv.memory(svc, T, pi, z, eta_c, delta)
    for g in range(svc.G):
        tot = F(0)
        for c in range(w.C):
            q = _q(svc.lam[c]) * _q(T[c, g]) * _q(pi[c, g]) / int(z[g])
            assert _close(conc[c, g], q, 1e-15)
            tot += (1 + _q(svc.kappa)) * q * (int(svc.Lin[c]) + int(eta_c[c])
                                              - int(delta[c, g]) * int(svc.Lpre[c]))
            tot += int(delta[c, g]) * int(svc.Lpre[c])
        assert _close(mem[g], tot, 1e-13), g


def test_P27_waiting_time_in_the_textbook_form():
    # Pollaczek-Khinchin: Wq = u E[S^2] / (2 (1 - u) E[S]) with the service-time
    # moments mixed by the routed arrival rates, u = mem / Mcap
    from oracle import serving as osv
    w, svc = _serving_tiny(34)
    T, ET2 = osv.service_times(svc, w)
    rng = np.random.default_rng(34)
    pi = rng.uniform(0.05, 0.5, (w.C, svc.G))
    z = np.array([2, 1, 1], np.int64)
    mem = rng.uniform(0.1, 0.9, svc.G) * svc.Mcap.astype(np.float64)
    Wq = osv.queue(svc, T, ET2, pi, z, mem)
    for g in range(svc.G):
        X = sum(_q(svc.lam[c]) * _q(pi[c, g]) for c in range(w.C))
        es = sum(_q(svc.lam[c]) * _q(pi[c, g]) * _q(T[c, g]) for c in range(w.C)) / X
        es2 = sum(_q(svc.lam[c]) * _q(pi[c, g]) * _q(ET2[c, g]) for c in range(w.C)) / X
        u = _q(mem[g]) / _q(svc.Mcap[g])
        assert _close(Wq[g], u * es2 / (2 * (1 - u) * es), 1e-12), g


def test_P28_objective_in_rationals():
    # the per-class cost of Sec. 3.3-3.4 summed with the arrival rates:
    # lam (a W + sum_g pi c_gpu tau pp T + c_slo max(0, sum_g pi (Wq + T) - a D)
    #      + (1 - a) c_rej), a = sum_g pi
    from oracle import serving as osv
    w, svc = _serving_tiny(35)
    T, _ = osv.service_times(svc, w)
    rng = np.random.default_rng(35)
    Wc = rng.uniform(10.0, 3000.0, w.C)
    for trial in range(4):
        pi = rng.dirichlet(np.ones(svc.G + 1), w.C)[:, :svc.G]
        Wq = rng.uniform(0.0, 30.0 if trial % 2 else 0.5, svc.G)
        obj = osv.objective(svc, Wc, T, Wq, pi)
        tot = F(0)
        for c in range(w.C):
            a = sum(_q(pi[c, g]) for g in range(svc.G))
            gpu = sum(_q(pi[c, g]) * _q(svc.c_gpu) * int(svc.tau[g]) * int(svc.pp[g]) * _q(T[c, g])
                      for g in range(svc.G))
            slack = sum(_q(pi[c, g]) * (_q(Wq[g]) + _q(T[c, g])) for g in range(svc.G)) - a * _q(svc.D[c])
            tot += _q(svc.lam[c]) * (a * _q(Wc[c]) + gpu + _q(svc.c_slo) * max(slack, F(0))
                                     + (1 - a) * _q(svc.c_rej))
        assert _close(obj, tot, 1e-12), trial
