"""The dense sums do not depend on how the launch schedules its work.

A problem large enough for the persistent grid that claims sample slices
(at least 65,536 (tile, sample) terms per resident block), with ragged
segments (2e6 samples, one sample, 3e5 uniform samples), classes aliasing
segments, costs on both sides of c_w = c_p (both kink orientations), and more
resident blocks than tiles, so that most blocks start by taking slices of
tiles they do not own and slices of the one-sample segment are empty.  Bars,
bit for bit against the oracle's exact definitions (App. A, Steps 3-5): every
S[c,k,m], W[e,c,k], m_star, the optimum and the quantiles; and two runs give
the same bytes.
"""
import numpy as np
import pytest

import oracle
from workloads.configs import Workload, _csr, _f32, eta_grid, lam_grid

pytestmark = pytest.mark.gpu


def _workload():
    rng = np.random.default_rng(21)
    L = 32768
    parts = [np.clip(np.rint(rng.lognormal(5.5, 1.3, 2_000_000)), 1, L).astype(np.int32),
             np.array([L], np.int32),
             rng.integers(0, L + 1, 300_000).astype(np.int32)]
    offsets, xi = _csr(parts)
    seg = np.array([0, 1, 2, 0, 2], np.int32)
    C, E = 5, 2
    c_p = _f32([8.0, 0.5, 2.0, 0.25, 96.0])
    c_w = _f32([1.0, 4.0, 2.0, 3.0, 0.125])
    eps = _f32(rng.uniform(0.0, 400.0, E * C))
    eps[:C] = 0.0
    return Workload("schedule", C, offsets, seg, xi, np.full(C, L, np.int32), eta_grid(512, L),
                    lam_grid(128), c_p, c_w, E, eps)


def _run(ctx, dev, w):
    import torch
    import paper_2607_16892_amd as dro
    prob = dro.Problem.from_workload(w, dev)
    eps = torch.from_numpy(w.eps).to(dev)
    r = dro.dro_cost_eval(ctx, prob, eps)
    a = dro.dro_argmin_reservation(ctx, prob, eps, r["S"])
    q = dro.class_quantile(ctx, prob)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for d in (r, a, q) for k, v in d.items() if v is not None}


def test_claimed_slices_give_the_exact_table(dev):
    import paper_2607_16892_amd as dro
    w = _workload()
    # 5 classes x 8 tiles (K = 512, M = 128) x 2e6 samples: past the direct-mode bound
    assert 5 * 8 * 2_000_000 >= 65536 * 1024
    print(f"[gpu] {w.name}: C={w.C} K={w.K} M={w.M} E={w.E} N={int(w.offsets[-1])}", flush=True)
    with dro.Context(dev.index or 0) as ctx:
        g1 = _run(ctx, dev, w)
        g2 = _run(ctx, dev, w)
    for k in g1:
        assert g1[k].tobytes() == g2[k].tobytes(), f"{k} differs between two runs"
    ref = oracle.solve(w, grouped=True)
    Sx = ref["S"].to_double()
    bad = np.argwhere(g1["S"].view(np.uint64) != Sx.view(np.uint64))
    assert bad.size == 0, f"S differs at {len(bad)} of {Sx.size} entries, first {tuple(bad[0])}"
    assert np.array_equal(g1["W"].view(np.uint64), ref["W"].view(np.uint64))
    assert np.array_equal(g1["m_star"], ref["m_star"])
    assert np.array_equal(g1["k_star"], ref["k_star"])
    assert np.array_equal(g1["W_star"].view(np.uint64), ref["W_star"].view(np.uint64))
    assert np.array_equal(g1["q_value"], ref["q_value"])
    assert np.array_equal(g1["q_rank"], ref["q_rank"])
