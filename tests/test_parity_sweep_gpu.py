"""Randomized parity sweep: many small problems across the shape space.

Sixty-four seeded cases drawn over the sizes where the kernels change behaviour:
one or several classes, aliased segments, segments of 1 to 20,000 samples,
supports L from 1 to 2^15, grids of 1 to 129 reservations and 1 to 300
multipliers (on both sides of a 32-pair tile and of a 256-multiplier chunk),
1 to 65 radii (one lane group per radius up to 64, then a second pass), cost
ratios up to 2^17 either way, constant, uniform and lognormal samples, and a
capacity bound k_max on about a third of them.  Every case runs the whole
path (dro_cost_eval, dro_argmin_reservation with k_max, class_quantile) and
the exact table (dro_exact_table), and is compared bit for bit with the
oracle's exact definitions (App. A, Steps 3-5; Prop. 4.2): S, W, m_star, k*,
W*, m at k*, the quantile and its rank.  The cases run one after another on
one context, so its workspace and staged offsets are reused across problems
of changing size.
"""
import numpy as np
import pytest

from workloads import random_workload

N_CASES = 64
L_CHOICES = [1, 2, 3, 50, 300, 4096, 32768]
N_CHOICES = [1, 2, 3, 5, 17, 63, 64, 65, 255, 256, 1000, 4097, 20000]
K_CHOICES = [1, 2, 3, 31, 32, 33, 64, 65, 129]
M_CHOICES = [1, 2, 3, 31, 32, 33, 64, 65, 256, 257, 300]
E_CHOICES = [1, 2, 3, 8, 16, 33, 64, 65]
EXTREME_COSTS = [(2.0 ** 7, 2.0 ** -10), (2.0 ** -10, 2.0 ** 7), (1.0, 1.0), (3.0, 0.5),
                 (0.25, 8.0)]


def sweep_case(i: int):
    """The i-th case: keyword arguments of random_workload and an optional k_max."""
    rng = np.random.default_rng(1000 + i)
    pick = lambda xs: xs[int(rng.integers(len(xs)))]
    C = int(rng.integers(1, 7))
    alias = C > 1 and rng.random() < 0.3
    S = int(rng.integers(1, C + 1)) if alias else C
    L = pick(L_CHOICES)
    K = min(pick(K_CHOICES), L + 1)
    kw = dict(seed=2000 + i, C=C, N=tuple(pick(N_CHOICES) for _ in range(S)), L=L, K=K,
              M=pick(M_CHOICES), E=pick(E_CHOICES), alias=alias,
              dist=pick(["lognormal", "lognormal", "uniform", "constant"]),
              lam_lo=pick([1e-3, 1e-2, 0.5]), lam_hi=pick([1.0, 10.0, 100.0, 128.0]))
    if rng.random() < 0.5:
        kw["cost_choices"] = EXTREME_COSTS
    kmax = rng.integers(0, K, C).astype(np.int32) if rng.random() < 0.3 else None
    return kw, kmax


CASES = [sweep_case(i) for i in range(N_CASES)]


def test_sweep_cases_are_valid_problems():
    """Every case stays inside what the library accepts (CPU check of the generator)."""
    for kw, kmax in CASES:
        w = random_workload(**kw)
        assert 1 <= w.L.max() <= 1 << 15
        assert w.eta.min() >= 0 and w.eta.max() <= w.L.min()
        assert np.all(np.diff(w.eta.astype(np.int64)) > 0)
        assert np.all(np.diff(w.lam.astype(np.float64)) > 0)
        for v in (w.lam, w.c_p, w.c_w):
            assert v.min() >= 2.0 ** -10 and v.max() <= 2.0 ** 7
        assert np.all(w.eps >= 0) and w.eps.size == w.E * w.C
        assert np.all(np.diff(w.offsets) >= 1)
        if kmax is not None:
            assert kmax.min() >= 0 and kmax.max() < w.K


@pytest.fixture(scope="module")
def ctx(dev):
    import paper_2607_16892_amd as dro
    c = dro.Context(dev.index or 0)
    yield c
    c.close()


@pytest.mark.gpu
@pytest.mark.parametrize("i", range(N_CASES))
def test_sweep_case_against_oracle(ctx, dev, i):
    import torch
    import oracle
    import paper_2607_16892_amd as dro
    kw, kmax = CASES[i]
    w = random_workload(**kw)
    print(f"[gpu] sweep {i}: C={w.C} S={len(w.offsets) - 1} N={w.offsets[-1]} L={int(w.L[0])} "
          f"K={w.K} M={w.M} E={w.E} kmax={'yes' if kmax is not None else 'no'}", flush=True)
    prob = dro.Problem.from_workload(w, dev)
    eps = torch.from_numpy(w.eps).to(dev)
    km = None if kmax is None else torch.from_numpy(kmax).to(dev)
    r = dro.dro_cost_eval(ctx, prob, eps)
    a = dro.dro_argmin_reservation(ctx, prob, eps, r["S"], k_max=km)
    q = dro.class_quantile(ctx, prob)
    x = dro.dro_exact_table(ctx, prob, eps, k_max=km)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for d in (r, a, q) for k, v in d.items() if v is not None}
    gx = {k: v.cpu().numpy() for k, v in x.items() if v is not None}
    ref = oracle.solve(w, grouped=True, kmax=kmax)
    bits = lambda v: np.ascontiguousarray(v).view(np.uint64)
    Sx = ref["S"].to_double()
    bad = np.argwhere(bits(g["S"]) != bits(Sx))
    assert bad.size == 0, f"S differs at {len(bad)} of {Sx.size} entries, first {tuple(bad[0])}"
    for name, got in (("dense path", g), ("exact table", gx)):
        assert np.array_equal(bits(got["W"]), bits(ref["W"])), f"{name}: W"
        assert np.array_equal(got["m_star"], ref["m_star"]), f"{name}: m_star"
        assert np.array_equal(got["k_star"], ref["k_star"]), f"{name}: k_star"
        assert np.array_equal(bits(got["W_star"]), bits(ref["W_star"])), f"{name}: W_star"
        assert np.array_equal(got["m_at_star"], ref["m_at_star"]), f"{name}: m_at_star"
    assert np.array_equal(g["q_value"], ref["q_value"])
    assert np.array_equal(g["q_rank"], ref["q_rank"])
