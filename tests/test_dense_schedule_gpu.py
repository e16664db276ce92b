"""The dense sums do not depend on how the launch schedules its work.

Problems large enough for the persistent grid that claims sample slices (at
least 65,536 (tile, sample) terms per resident block, 1,024 resident blocks),
each bit for bit against the oracle's exact definitions (App. A, Steps 3-5):
every S[c,k,m], W[e,c,k], m_star, the optimum and the quantiles; and two runs
give the same bytes.

- A: ragged segments (2e6 samples, one sample, 3e5 uniform samples), classes
  aliasing segments, costs on both sides of c_w = c_p (both kink
  orientations), whole tiles (K = 512, M = 128), and more resident blocks
  than tiles, so that most blocks start by taking slices of tiles they do not
  own and slices of the one-sample segment are empty.
- B: partial tiles in both directions (K = 300 over tiles of 128 grid
  points, M = 50 of a 64-multiplier tile), 9 tiles in all, one segment of
  1.2e7 samples and one of 5, so nearly every slice of the short segment's
  tiles is empty.
- C: more tiles than resident blocks (1,152), so every block starts with more
  than one tile of its own: 128 classes on 4 aliased segments of 1e5 samples,
  K = 1025 (the last k-tile holds one grid point), M = 33 (half a tile),
  cost ratios up to 2^17 either way.
"""
import numpy as np
import pytest

import oracle
from workloads.configs import Workload, _csr, _f32, eta_grid, lam_grid

pytestmark = pytest.mark.gpu

RESIDENT = 1024   # resident blocks of the dense launch (256 compute units x 4)
DIRECT_TERMS = 65536


def tiles_per_class(K, M, threads=256, tm=32):
    """Tiles of one class as the dense launch forms them: lanes_m, a power of
    two, covers M in groups of tm multipliers; the remaining lanes take grid
    points."""
    lanes_m = 1
    while lanes_m < -(-M // tm) and lanes_m < threads:
        lanes_m *= 2
    lanes_k = threads // lanes_m
    return -(-K // lanes_k) * -(-M // (tm * lanes_m))


def _case_a():
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
    return Workload("schedule-a", C, offsets, seg, xi, np.full(C, L, np.int32), eta_grid(512, L),
                    lam_grid(128), c_p, c_w, E, eps)


def _case_b():
    rng = np.random.default_rng(22)
    L = 4096
    parts = [np.clip(np.rint(rng.lognormal(5.0, 1.0, 12_000_000)), 0, L).astype(np.int32),
             np.array([0, 7, L, 7, 3000], np.int32)]
    offsets, xi = _csr(parts)
    seg = np.array([0, 1, 0], np.int32)
    C, E = 3, 3
    c_p = _f32([4.0, 0.75, 0.5])
    c_w = _f32([1.0, 0.75, 6.0])
    eps = _f32(rng.uniform(0.0, 60.0, E * C))
    eps[:C] = 0.0
    return Workload("schedule-b", C, offsets, seg, xi, np.full(C, L, np.int32), eta_grid(300, L),
                    lam_grid(50, 2.0 ** -10, 2.0 ** 7), c_p, c_w, E, eps)


def _case_c():
    rng = np.random.default_rng(23)
    L, S, C, E = 8192, 4, 128, 2
    parts = [np.clip(np.rint(rng.lognormal(4.0 + s, 0.9, 100_000)), 0, L).astype(np.int32)
             for s in range(S)]
    offsets, xi = _csr(parts)
    seg = (np.arange(C) % S).astype(np.int32)
    choices = [(2.0 ** 7, 2.0 ** -10), (2.0 ** -10, 2.0 ** 7), (8.0, 1.0), (1.0, 1.0), (0.5, 3.0)]
    pick = rng.integers(len(choices), size=C)
    c_p = _f32([choices[i][0] for i in pick])
    c_w = _f32([choices[i][1] for i in pick])
    eps = _f32(rng.uniform(0.0, 200.0, E * C))
    eps[:C] = 0.0
    return Workload("schedule-c", C, offsets, seg, xi, np.full(C, L, np.int32), eta_grid(1025, L),
                    lam_grid(33, 0.01, 100.0), c_p, c_w, E, eps)


CASES = {"a": _case_a, "b": _case_b, "c": _case_c}


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


@pytest.mark.parametrize("case", sorted(CASES))
def test_claimed_slices_give_the_exact_table(dev, case):
    import paper_2607_16892_amd as dro
    w = CASES[case]()
    T = w.C * tiles_per_class(w.K, w.M)
    max_n = int(np.diff(w.offsets).max())
    assert T * max_n >= DIRECT_TERMS * RESIDENT  # past the one-block-per-slice bound
    if case == "c":
        assert T > RESIDENT
    print(f"[gpu] {w.name}: C={w.C} K={w.K} M={w.M} E={w.E} N={int(w.offsets[-1])} tiles={T}",
          flush=True)
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
