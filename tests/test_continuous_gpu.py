"""The continuous-multiplier dual (dro_continuous_dual) against exact rationals.

The reference is oracle/brute.dual_exact: the Kantorovich dual of
App. A, Step 3, minimised over continuous gamma >= 0 by evaluating it,
in fractions, at every breakpoint (itself pinned to the HiGHS transport LP on
the CPU).  At full size the checks are the grid bound (the grid dual can only
be larger) and the SAA bound.
"""
from fractions import Fraction as F

import numpy as np
import pytest

import oracle
from oracle import brute
from workloads import make_workload, random_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx(dev):
    import paper_2607_16892_amd as dro
    c = dro.Context(dev.index or 0)
    yield c
    c.close()


def run_cont(ctx, w, dev):
    import torch
    import paper_2607_16892_amd as dro
    print(f"[gpu] continuous dual {w.name} C={w.C} K={w.K} E={w.E}", flush=True)
    prob = dro.Problem.from_workload(w, dev)
    eps = torch.from_numpy(w.eps).to(dev)
    r = dro.dro_continuous_dual(ctx, prob, eps)
    torch.cuda.synchronize()
    return r["W"].cpu().numpy(), r["gamma"].cpu().numpy()


@pytest.mark.parametrize("seed", range(4))
def test_matches_exact_rational_dual(ctx, dev, seed):
    w = random_workload(seed=400 + seed, C=2, N=(7, 5), L=36, K=10, M=5, E=2)
    W, g = run_cont(ctx, w, dev)
    worst = 0.0
    for e in range(w.E):
        for c in range(w.C):
            xs = w.samples_of(c).tolist()
            for k in range(w.K):
                dv, _ = brute.dual_exact(int(w.eta[k]), xs, int(w.L[c]), float(w.c_p[c]),
                                         float(w.c_w[c]), float(w.eps[e * w.C + c]))
                rel = abs(W[e, c, k] - float(dv)) / max(float(dv), 1e-300)
                worst = max(worst, rel)
                # the returned gamma attains the minimum
                gam = F(float(g[e, c, k]))
                at = gam * F(float(w.eps[e * w.C + c])) + sum(
                    (brute._phi_max3(int(w.eta[k]), x, int(w.L[c]), float(w.c_p[c]),
                                     float(w.c_w[c]), gam) for x in xs), F(0)) / len(xs)
                assert abs(float(at) - float(dv)) <= 1e-9 * max(float(dv), 1.0)
                assert 0.0 <= g[e, c, k] <= max(float(w.c_p[c]), float(w.c_w[c]))
    print(f"  max rel err vs exact dual {worst:.2e}", flush=True)
    assert worst <= 1e-10


def test_grid_and_saa_bounds_lognormal_4x100k(ctx, dev):
    import torch
    import paper_2607_16892_amd as dro
    w = make_workload("lognormal-4x100k")
    W, g = run_cont(ctx, w, dev)
    prob = dro.Problem.from_workload(w, dev)
    ex = dro.dro_exact_table(ctx, prob, torch.from_numpy(w.eps).to(dev), want_argmin=False)
    Wg = ex["W"].cpu().numpy()
    assert np.all(W <= Wg * (1 + 1e-12)), "continuous dual above the grid dual"
    # the grid is dense near gamma*: the two agree to a few 1e-3 at most
    assert np.max((Wg - W) / Wg) < 0.05
    # SAA lower bound, from the oracle with eps = 0 (the exact SAA table)
    w0 = make_workload("lognormal-4x100k")
    w0.eps[:] = 0
    saa, _ = oracle.W_table(w0, oracle.S_exact(w0))
    assert np.all(W >= saa * (1 - 1e-12))
