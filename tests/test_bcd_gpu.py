"""The fused block step on the GPU against the oracle's sweep (exact results)."""
import json
import os

import numpy as np
import pytest

import oracle
from workloads import make_workload, random_workload

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def ctx(dev):
    import paper_2607_16892_amd as dro
    c = dro.Context(dev.index or 0)
    yield c
    c.close()


def gpu_step(ctx, w, dev, k_prev=None):
    import torch
    import paper_2607_16892_amd as dro
    print(f"[gpu] block step {w.name} iteration={w.meta.get('iteration') if w.meta else None} "
          f"C={w.C} K={w.K} M={w.M} G={w.groups.G}", flush=True)
    prob = dro.Problem.from_workload(w, dev)
    eps = torch.from_numpy(w.eps[: w.C].copy()).to(dev)
    grp = dro.Groups.from_numpy(w.groups.cap, w.groups.conc, w.groups.kappa, dev)
    if k_prev is None:
        kp = dro.bcd_init_state(ctx, prob)
    else:
        kp = torch.from_numpy(np.asarray(k_prev, np.int32)).to(dev)
    k0 = kp.cpu().numpy()
    o = dro.bcd_block_step(ctx, prob, eps, grp, kp)
    torch.cuda.synchronize()
    return k0, {k: v.cpu().numpy() for k, v in o.items()}


@pytest.mark.parametrize("seed", range(6))
def test_block_step_matches_oracle(ctx, dev, seed):
    w = random_workload(seed=900 + seed, C=4, N=(200, 31, 500, 77), L=600, K=33, M=19, E=1,
                        with_groups=True, G=3)
    k0, g = gpu_step(ctx, w, dev)
    assert np.array_equal(k0, oracle.bcd_init(w))
    S = oracle.S_exact(w)
    W, _ = oracle.W_table(w, S)
    o = oracle.bcd_step(w, W[0], k0)
    assert np.array_equal(g["k_next"], o["k_next"])
    assert np.array_equal(g["W_star"].view(np.uint64), o["W_star"].view(np.uint64))
    assert np.array_equal(g["usage"].view(np.uint64), o["usage"].view(np.uint64))
    assert np.array_equal(g["feasible"], o["feasible"])
    qv, _ = oracle.quantile(w)
    assert np.array_equal(g["q_value"], qv)


def test_block_step_from_given_state(ctx, dev):
    w = random_workload(seed=950, C=3, N=(90, 60, 150), L=400, K=21, M=13, E=1, with_groups=True, G=2)
    k_prev = np.array([20, 0, 7], np.int32)
    _, g = gpu_step(ctx, w, dev, k_prev)
    S = oracle.S_exact(w)
    W, _ = oracle.W_table(w, S)
    o = oracle.bcd_step(w, W[0], k_prev)
    assert np.array_equal(g["k_next"], o["k_next"])
    assert np.array_equal(g["W_star"].view(np.uint64), o["W_star"].view(np.uint64))


def _drift_gold():
    path = os.path.join(HERE, "golden", "drift-8x4M_bcd.json")
    if not os.path.exists(path):
        pytest.skip("no stored oracle results for the drifting block-step loop")
    return json.load(open(path))


@pytest.mark.parametrize("first", [0, 10, 20, 30, 40])
def test_drift_iterations_against_stored_oracle(ctx, dev, first):
    # 50 iterations of the drifting loop in chunks of 10; each chunk starts from
    # the stored state entering its first iteration, then chains its own.
    gold = _drift_gold()
    rows = [r for r in gold["rows"] if first <= r["iteration"] < first + 10]
    if not rows:
        pytest.skip(f"the stored loop has no iteration {first}")
    k_prev = None if first == 0 else np.array(rows[0]["k_prev"], np.int32)
    for row in rows:
        w = make_workload("drift-8x4M", iteration=row["iteration"])
        assert w.checksum() == row["checksum"]
        k0, g = gpu_step(ctx, w, dev, k_prev)
        assert k0.tolist() == row["k_prev"]
        assert g["k_next"].tolist() == row["k_next"]
        assert [float(v).hex() for v in g["W_star"]] == row["W_star"]
        assert [float(v).hex() for v in g["usage"]] == row["usage"]
        assert g["feasible"].tolist() == row["feasible"]
        assert g["q_value"].tolist() == row["q_value"]
        k_prev = g["k_next"]


def _drift_tight(n=50_000, cap_scale=0.3):
    """The drifting 8-class workload's grid, costs and routing, the first n
    samples of each class, and capacities scaled down so that groups bind."""
    from workloads.configs import Workload, Groups
    w = make_workload("drift-8x4M", iteration=0)
    parts = [w.samples_of(c)[:n].copy() for c in range(w.C)]
    off = np.zeros(w.C + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in parts])
    g = Groups((w.groups.cap * np.float32(cap_scale)).astype(np.float32), w.groups.conc.copy(),
               w.groups.kappa)
    return Workload("drift-8x4M-tight", w.C, off, None, np.concatenate(parts), w.L, w.eta, w.lam,
                    w.c_p, w.c_w, 1, w.eps.copy(), groups=g)


def test_block_step_with_binding_capacity_at_full_grid(ctx, dev):
    w = _drift_tight()
    k0, g = gpu_step(ctx, w, dev)
    S = oracle.S_exact(w)
    W, _ = oracle.W_table(w, S)
    o = oracle.bcd_step(w, W[0], k0)
    assert np.array_equal(g["k_next"], o["k_next"])
    assert np.array_equal(g["W_star"].view(np.uint64), o["W_star"].view(np.uint64))
    assert np.array_equal(g["usage"].view(np.uint64), o["usage"].view(np.uint64))
    assert np.array_equal(g["feasible"], o["feasible"])
    # the sweep must have been limited by capacity somewhere
    unconstrained, _ = oracle.argmin(W)
    assert not np.array_equal(o["k_next"], unconstrained[0]), "no capacity bound was active"
