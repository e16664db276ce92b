"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Bars:
  * integer results (k_star, m_at_star, q_value, q_rank) are bit-exact;
  * W_star, the exact optimum, is bit-exact (same fp64 expression of the same
    exact sum);
  * the dense sums S and the table W are within 1e-5 relative, plus
    1e-9 (c_p + c_w) absolute for values at or near zero.
"""
import json
import os

import numpy as np
import pytest

import oracle
from workloads import make_workload, random_workload

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
REL = 1e-5


@pytest.fixture(scope="module")
def ctx(dev):
    import paper_2607_16892_amd as dro
    c = dro.Context(dev.index or 0)
    yield c
    c.close()


def run_gpu(ctx, w, dev, k_max=None):
    import torch
    import paper_2607_16892_amd as dro
    print(f"[gpu] {w.name} C={w.C} K={w.K} M={w.M} E={w.E} N={w.offsets[-1]}", flush=True)
    prob = dro.Problem.from_workload(w, dev)
    eps = torch.from_numpy(w.eps).to(dev)
    dro.dro_validate(ctx, prob, eps)
    km = None if k_max is None else torch.from_numpy(np.asarray(k_max, np.int32)).to(dev)
    r = dro.dro_cost_eval(ctx, prob, eps)
    a = dro.dro_argmin_reservation(ctx, prob, eps, r["S"], k_max=km)
    q = dro.class_quantile(ctx, prob)
    torch.cuda.synchronize()
    flags = ctx.take_flags()
    out = {k: v.cpu().numpy() for d in (r, a, q) for k, v in d.items() if v is not None}
    out["flags"] = flags
    return out


def check_against_oracle(w, g, kmax=None):
    ref = oracle.solve(w, grouped=True, kmax=kmax)
    Sx = ref["S"].to_double()
    scale = (w.c_p + w.c_w).astype(np.float64)
    tolS = REL * Sx + 1e-9 * scale[:, None, None] * np.array([w.n_of(c) for c in range(w.C)])[:, None, None]
    errS = np.abs(g["S"] - Sx)
    assert np.all(errS <= tolS), f"S max rel err {np.max(errS / np.maximum(Sx, 1e-300)):.3e}"
    tolW = REL * np.abs(ref["W"]) + 1e-9 * scale[None, :, None]
    errW = np.abs(g["W"] - ref["W"])
    assert np.all(errW <= tolW), f"W max rel err {np.max(errW / np.maximum(ref['W'], 1e-300)):.3e}"
    assert np.array_equal(g["k_star"], ref["k_star"])
    assert np.array_equal(g["W_star"].view(np.uint64), ref["W_star"].view(np.uint64))
    assert np.array_equal(g["m_at_star"], ref["m_at_star"])
    assert np.array_equal(g["q_value"], ref["q_value"])
    assert np.array_equal(g["q_rank"], ref["q_rank"])
    assert g["flags"] == 0
    relS = errS / np.maximum(Sx, 1e-300)
    worst = np.unravel_index(np.argmax(relS), relS.shape)
    print(f"  S rel err {relS.max():.2e} at (c,k,m)={tuple(int(v) for v in worst)}  "
          f"W rel err {np.max(errW / np.maximum(ref['W'], 1e-300)):.2e}", flush=True)


@pytest.mark.parametrize("name", ["lognormal-1x1k", "lognormal-4x100k"])
def test_full_config_against_oracle(ctx, dev, name):
    w = make_workload(name)
    check_against_oracle(w, run_gpu(ctx, w, dev))


RANDOM_CASES = [
    dict(seed=1),
    dict(seed=2, C=4, N=(1, 2, 3, 1000), L=500, K=40, M=20, E=2),            # ragged, N = 1
    dict(seed=3, C=5, N=(60, 9), alias=True, L=200, K=25, M=11, E=3),       # aliased segments
    dict(seed=4, C=2, N=(3000, 257), L=32768, K=129, M=33, E=2),            # largest support
    dict(seed=5, C=3, N=(40, 40, 40), dist="constant", L=100, K=101, M=9),  # all samples equal
    dict(seed=6, C=2, N=(500, 77), dist="uniform", L=1000, K=1, M=7),       # one grid point
    dict(seed=7, C=2, N=(123, 45), L=300, K=31, M=1, E=2),                  # one multiplier
    dict(seed=8, C=3, N=(2049, 1025, 4097), L=4096, K=513, M=70, E=1,
         cost_choices=[(4.0, 1.0), (8.0, 1.0), (2.0, 2.0)]),               # q N integer: ties
    dict(seed=10, C=6, N=(700, 33, 1500), alias=True, L=2000, K=97, M=40, E=19),  # 19 radii
    dict(seed=11, C=4, N=(256, 511, 512, 16385), L=3000, K=33, M=40, E=2),  # slice-floor sizes
    dict(seed=12, C=3, N=(300, 41, 2000), L=1500, K=77, M=3, E=8),         # 8 radii, 3 multipliers
    dict(seed=13, C=2, N=(500, 60), L=700, K=50, M=2, E=3),                 # 2 multipliers
]


@pytest.mark.parametrize("case", RANDOM_CASES, ids=lambda c: f"seed{c['seed']}")
def test_random_workloads_against_oracle(ctx, dev, case):
    w = random_workload(**case)
    check_against_oracle(w, run_gpu(ctx, w, dev))


def test_capacity_limited_argmin(ctx, dev):
    w = random_workload(seed=9, C=3, N=(300, 200, 100), L=800, K=65, M=17, E=2)
    kmax = np.array([5, 64, 0], np.int32)
    check_against_oracle(w, run_gpu(ctx, w, dev, k_max=kmax), kmax=kmax)


def test_deterministic_run_to_run(ctx, dev):
    w = make_workload("lognormal-4x100k")
    a, b = run_gpu(ctx, w, dev), run_gpu(ctx, w, dev)
    for k in ("S", "W", "m_star", "k_star", "W_star", "m_at_star", "q_value", "q_rank"):
        assert a[k].tobytes() == b[k].tobytes(), k


def _golden(name):
    path = os.path.join(HERE, "golden", f"{name}.json")
    if not os.path.exists(path):
        pytest.skip(f"no stored oracle results for {name}")
    return json.load(open(path))


@pytest.mark.parametrize("name", ["mixture-16x1M", "ratios-8x250k"])
def test_large_config_against_stored_oracle(ctx, dev, name):
    gold = _golden(name)
    w = make_workload(name)
    assert w.checksum() == gold["checksum"], "generated inputs differ from the stored ones"
    g = run_gpu(ctx, w, dev)
    assert g["flags"] == 0
    assert np.array_equal(g["k_star"], np.array(gold["k_star"]))
    ws = np.array([[float.fromhex(v) for v in row] for row in gold["W_star"]])
    assert np.array_equal(g["W_star"].view(np.uint64), ws.view(np.uint64))
    assert np.array_equal(g["m_at_star"], np.array(gold["m_at_star"]))
    assert np.array_equal(g["q_value"], np.array(gold["q_value"]))
    assert np.array_equal(g["q_rank"], np.array(gold["q_rank"]))
    for c, row in gold["W_rows"].items():
        ref = np.array([float.fromhex(v) for v in row])
        got = g["W"][0, int(c)]
        assert np.all(np.abs(got - ref) <= REL * ref), f"class {c}"
    # sampled dense sums, computed one by one by the oracle at full size
    rng = np.random.default_rng(0)
    P = 24
    cs = rng.integers(0, w.C, P)
    ks = rng.integers(0, w.K, P)
    ms = rng.integers(0, w.M, P)
    ex = oracle.S_exact_at(w, cs, ks, ms)
    for i in range(P):
        ref = oracle._load().oracle_fix_to_double(int(ex.hi[i]), int(ex.lo[i]))
        got = g["S"][cs[i], ks[i], ms[i]]
        assert abs(got - ref) <= REL * ref, (cs[i], ks[i], ms[i], got, ref)


def _kink_workload():
    """Every sample sits just above the crossing point x0 of the two lines of phi.

    With c_w = c_p = 1.00055 lam_37 and eta = 30000 the crossing point is
    x0 = 30007.49 while phi there is only about 6.5.  A kink rounded to fp32 in
    absolute terms (error up to 2^-10 tokens at this size) would move S by
    about 2e-4 relative; measured from eta it is exact to ~1e-7.
    """
    from workloads import eta_grid, lam_grid
    from workloads.configs import Workload
    L, K, M = 32768, 2049, 64
    lam = lam_grid(M)
    c = np.float32(lam[37] * np.float32(1.00055))
    xs = np.full(2000, 30008, np.int32)
    return Workload("kink", 1, np.array([0, xs.size], np.int64), None, xs,
                    np.array([L], np.int32), eta_grid(K, L), lam, np.array([c], np.float32),
                    np.array([c], np.float32), 2, np.array([0.0, 40.0], np.float32))


def test_samples_on_the_kink(ctx, dev):
    w = _kink_workload()
    check_against_oracle(w, run_gpu(ctx, w, dev))


# ------------------------------------------------------------ exact table ----
# dro_exact_table (value counts and prefix sums) must reproduce the oracle's
# exact-spec W table, m_star and optimum bit for bit, for every (e, c, k).

def run_exact_table(ctx, w, dev, k_max=None):
    import torch
    import paper_2607_16892_amd as dro
    print(f"[gpu] exact table {w.name} C={w.C} K={w.K} M={w.M} E={w.E}", flush=True)
    prob = dro.Problem.from_workload(w, dev)
    eps = torch.from_numpy(w.eps).to(dev)
    km = None if k_max is None else torch.from_numpy(np.asarray(k_max, np.int32)).to(dev)
    r = dro.dro_exact_table(ctx, prob, eps, k_max=km)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in r.items() if v is not None}


def check_exact_table(w, g, kmax=None):
    ref = oracle.solve(w, grouped=True, kmax=kmax)
    assert np.array_equal(g["W"].view(np.uint64), ref["W"].view(np.uint64))
    assert np.array_equal(g["m_star"], ref["m_star"])
    assert np.array_equal(g["k_star"], ref["k_star"])
    assert np.array_equal(g["W_star"].view(np.uint64), ref["W_star"].view(np.uint64))
    assert np.array_equal(g["m_at_star"], ref["m_at_star"])


@pytest.mark.parametrize("name", ["lognormal-1x1k", "lognormal-4x100k"])
def test_exact_table_full_config(ctx, dev, name):
    w = make_workload(name)
    check_exact_table(w, run_exact_table(ctx, w, dev))


@pytest.mark.parametrize("case", RANDOM_CASES, ids=lambda c: f"seed{c['seed']}")
def test_exact_table_random(ctx, dev, case):
    w = random_workload(**case)
    check_exact_table(w, run_exact_table(ctx, w, dev))


def test_exact_table_kink_and_capacity(ctx, dev):
    w = _kink_workload()
    check_exact_table(w, run_exact_table(ctx, w, dev))
    w = random_workload(seed=9, C=3, N=(300, 200, 100), L=800, K=65, M=17, E=2)
    kmax = np.array([5, 64, 0], np.int32)
    check_exact_table(w, run_exact_table(ctx, w, dev, k_max=kmax), kmax=kmax)


@pytest.mark.parametrize("name", ["mixture-16x1M", "ratios-8x250k"])
def test_exact_table_large_config_against_stored_oracle(ctx, dev, name):
    gold = _golden(name)
    w = make_workload(name)
    assert w.checksum() == gold["checksum"]
    g = run_exact_table(ctx, w, dev)
    assert np.array_equal(g["k_star"], np.array(gold["k_star"]))
    ws = np.array([[float.fromhex(v) for v in row] for row in gold["W_star"]])
    assert np.array_equal(g["W_star"].view(np.uint64), ws.view(np.uint64))
    assert np.array_equal(g["m_at_star"], np.array(gold["m_at_star"]))
    for c, row in gold["W_rows"].items():
        ref = np.array([float.fromhex(v) for v in row])
        assert np.array_equal(g["W"][0, int(c)].view(np.uint64), ref.view(np.uint64)), f"class {c}"


# ---------------------------------------------------------- maximum sizes ----
# The largest grids and segments the library accepts (K = 2^15 + 1 grid points,
# M = 65536 multipliers, 2^26 samples in one class), each against the oracle.

def test_max_reservation_grid(ctx, dev):
    w = random_workload(seed=41, C=1, N=(3000,), L=32768, K=32769, M=16, E=2)
    assert np.array_equal(w.eta, np.arange(32769))
    check_against_oracle(w, run_gpu(ctx, w, dev))


def test_max_multiplier_grid(ctx, dev):
    w = random_workload(seed=42, C=2, N=(500, 300), L=1000, K=8, M=65536, E=1)
    assert np.all(np.diff(w.lam.astype(np.float64)) > 0)
    check_against_oracle(w, run_gpu(ctx, w, dev))


def test_max_class_size(ctx, dev):
    from workloads.configs import Workload
    from workloads import eta_grid, lam_grid
    n = 1 << 26
    rng = np.random.default_rng(43)
    xi = rng.integers(0, 32769, n, dtype=np.int32)
    L = 32768
    w = Workload("max-class", 1, np.array([0, n], np.int64), None, xi, np.array([L], np.int32),
                 eta_grid(5, L), lam_grid(4), np.array([8.0], np.float32),
                 np.array([1.0], np.float32), 1, np.array([100.0], np.float32))
    check_against_oracle(w, run_gpu(ctx, w, dev))
