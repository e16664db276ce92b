"""The rest of Alg. 1 on the GPU (C ABI) against the oracle (oracle/serving.py).

Bars: service times, queue state, the reservation sweep, prefix caching and
the configuration search are evaluated in the same fixed-order double
arithmetic on both sides and are compared bit for bit.  The routing LP is
solved by a dense simplex on the GPU and by HiGHS in the oracle: optimal
objectives agree to 1e-9 relative and the routings to 1e-7 (the instances
are generic, so the optimum is unique).
"""
import numpy as np
import pytest

import oracle
from oracle import serving as osv
from workloads.configs import serving_workload

pytestmark = pytest.mark.gpu

SMALL = [(1, 1), (2, 1), (4, 1), (2, 2), (4, 2)]


@pytest.fixture(scope="module")
def ctx(dev):
    import paper_2607_16892_amd as dro
    c = dro.Context(dev.index or 0)
    yield c
    c.close()


def _t(a, dt, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).to(dev)


def _setup(ctx, dev, w, svc):
    import paper_2607_16892_amd as dro
    from paper_2607_16892_amd import serving as gs
    print(f"[gpu] serving {w.name} C={w.C} G={svc.G} J={svc.J} K={w.K}", flush=True)
    prob = dro.Problem.from_workload(w, dev)
    s = gs.Service.from_model(svc, dev)
    return prob, s


def _bits(a):
    return np.ascontiguousarray(a, np.float64).view(np.uint64)


def _state(w, svc, seed, T=None):
    """A random state: routing, counts, caching and reservations; with T given,
    the routing is scaled down until every group's memory use is below
    0.9 u_max Mcap (a state with a finite wait)."""
    rng = np.random.default_rng(seed)
    C, G = w.C, svc.G
    z = rng.integers(0, 3, G).astype(np.int32)
    z[0] = max(z[0], 1)
    pi = rng.dirichlet(np.ones(G + 1), C)[:, :G] * (z > 0)[None, :]
    pi[rng.random((C, G)) < 0.3] = 0.0
    delta = (rng.random((C, G)) < 0.3).astype(np.uint8)
    eta_c = rng.integers(0, 400, C).astype(np.int32)
    if T is not None:
        lim = 0.9 * float(svc.u_max) * svc.Mcap.astype(np.float64)
        for g in range(G):
            if (delta[:, g].astype(np.int64) * svc.Lpre).sum() > 0.5 * lim[g]:
                delta[:, g] = 0
        for _ in range(80):
            mem = osv.memory(svc, T, pi, z, eta_c, delta)
            if np.all(mem <= lim):
                break
            pi = pi * 0.5
    return z, pi, delta, eta_c


@pytest.mark.parametrize("seed", [1, 2])
def test_service_times_and_queue_state(ctx, dev, seed):
    import torch
    from paper_2607_16892_amd import serving as gs
    w, svc = serving_workload(C=6, N=20000 * seed, J=24, K=257, M=32, configs=SMALL, seed=seed)
    prob, s = _setup(ctx, dev, w, svc)
    g = gs.bcd_service_times(ctx, prob, s)
    T, ET2 = osv.service_times(svc, w)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(g["T"].cpu().numpy()), _bits(T))
    assert np.array_equal(_bits(g["ET2"].cpu().numpy()), _bits(ET2))
    for trial in range(4):
        z, pi, delta, eta_c = _state(w, svc, 10 * seed + trial)
        q = gs.bcd_queue_state(ctx, w.C, s, g["T"], g["ET2"], _t(pi, np.float64, dev),
                               _t(z, np.int32, dev), _t(eta_c, np.int32, dev),
                               _t(delta, np.uint8, dev))
        mem = osv.memory(svc, T, pi, z, eta_c, delta)
        Wq = osv.queue(svc, T, ET2, pi, z, mem)
        conc, cap = osv.lp2_inputs(svc, T, pi, z, delta)
        torch.cuda.synchronize()
        assert np.array_equal(_bits(q["mem"].cpu().numpy()), _bits(mem))
        assert np.array_equal(_bits(q["Wq"].cpu().numpy()), _bits(Wq))
        assert np.array_equal(_bits(q["conc"].cpu().numpy()), _bits(conc))
        assert np.array_equal(_bits(q["cap"].cpu().numpy()), _bits(cap))
        d = gs.bcd_prefix_cache(ctx, q["conc"])
        torch.cuda.synchronize()
        assert np.array_equal(d.cpu().numpy(), osv.prefix_cache(svc, T, pi, z))


@pytest.mark.parametrize("seed", [3, 4, 5, 6])
def test_routing_lp_matches_highs(ctx, dev, seed):
    import torch
    from paper_2607_16892_amd import serving as gs
    w, svc = serving_workload(C=5 + seed, N=5000, J=24, K=257, M=32, configs=SMALL, seed=seed)
    prob, s = _setup(ctx, dev, w, svc)
    g = gs.bcd_service_times(ctx, prob, s)
    T, ET2 = osv.service_times(svc, w)
    rng = np.random.default_rng(seed)
    for trial in range(3):
        z, pi0, delta, eta_c = _state(w, svc, 100 * seed + trial, T)
        mem = osv.memory(svc, T, pi0, z, eta_c, delta)
        Wq = osv.queue(svc, T, ET2, pi0, z, mem)
        Wc = rng.uniform(50.0, 3000.0, w.C)
        ref_pi, ref_obj = osv.routing_lp(svc, Wc, T, Wq, z, eta_c, delta)
        r = gs.bcd_routing_lp(ctx, w.C, s, _t(Wc, np.float64, dev), g["T"], _t(Wq, np.float64, dev),
                              _t(z, np.int32, dev), _t(eta_c, np.int32, dev),
                              _t(delta, np.uint8, dev))
        torch.cuda.synchronize()
        info = r["info"].cpu().numpy()
        assert info[1] == 0, f"simplex status {info[1]}"
        obj = float(r["objective"].cpu().numpy()[0])
        assert abs(obj - ref_obj) <= 1e-9 * abs(ref_obj), (obj, ref_obj)
        pi = r["pi"].cpu().numpy()
        assert np.max(np.abs(pi - ref_pi)) <= 1e-7, np.max(np.abs(pi - ref_pi))
        # the GPU routing is feasible
        assert np.all(pi.sum(axis=1) <= 1.0 + 1e-12)
        memg = osv.memory(svc, T, pi, z, eta_c, delta)
        assert np.all(memg <= float(svc.u_max) * svc.Mcap.astype(np.float64) * (1 + 1e-12))


@pytest.mark.parametrize("seed", [7, 8])
def test_routing_lp_degenerate(ctx, dev, seed):
    """Identical classes and a wait that makes every SLO row tight at pi = 0:
    many optimal routings and many degenerate pivots.  The optimal objective
    is unique (1e-9 relative to HiGHS) and the GPU routing is feasible and
    attains it."""
    import torch
    from paper_2607_16892_amd import serving as gs
    w, svc = serving_workload(C=12, N=3000, J=24, K=257, M=32, configs=SMALL, seed=seed)
    for name in ("lam", "Lin", "Lpre", "D"):
        getattr(svc, name)[:] = getattr(svc, name)[0]
    s = gs.Service.from_model(svc, dev)
    T, ET2 = osv.service_times(svc, w)
    T = np.repeat(T[:1], w.C, axis=0)
    z = np.ones(svc.G, np.int32)
    delta = np.zeros((w.C, svc.G), np.uint8)
    eta_c = np.full(w.C, 200, np.int32)
    Wq = float(svc.D[0]) - T[0]            # Wq_g + T_cg - D_c = 0 for every row
    Wc = np.full(w.C, 800.0)
    ref_pi, ref_obj = osv.routing_lp(svc, Wc, T, Wq, z, eta_c, delta)
    r = gs.bcd_routing_lp(ctx, w.C, s, _t(Wc, np.float64, dev), _t(T, np.float64, dev),
                          _t(Wq, np.float64, dev), _t(z, np.int32, dev),
                          _t(eta_c, np.int32, dev), _t(delta, np.uint8, dev))
    torch.cuda.synchronize()
    info = r["info"].cpu().numpy()
    assert info[1] == 0, f"simplex status {info[1]}"
    obj = float(r["objective"].cpu().numpy()[0])
    assert abs(obj - ref_obj) <= 1e-9 * abs(ref_obj), (obj, ref_obj)
    pi = r["pi"].cpu().numpy()
    assert np.all(pi >= 0.0) and np.all(pi.sum(axis=1) <= 1.0 + 1e-12)
    memg = osv.memory(svc, T, pi, z, eta_c, delta)
    assert np.all(memg <= float(svc.u_max) * svc.Mcap.astype(np.float64) * (1 + 1e-12))
    slack = np.maximum((pi * (Wq[None, :] + T - svc.D[:, None].astype(np.float64))).sum(1), 0.0)
    lam = svc.lam.astype(np.float64)
    gpu = (svc.tau.astype(np.float64) * svc.pp)[None, :] * T
    val = float(np.sum(lam[:, None] * pi * (Wc[:, None] + float(svc.c_gpu) * gpu
                                            - float(svc.c_rej)))
                + np.sum(lam * float(svc.c_slo) * slack) + np.sum(lam * float(svc.c_rej)))
    assert abs(val - ref_obj) <= 1e-9 * abs(ref_obj), (val, ref_obj)


def test_routing_lp_infeasible_start(ctx, dev):
    import torch
    from paper_2607_16892_amd import serving as gs
    w, svc = serving_workload(C=4, N=3000, J=16, K=129, M=16, configs=SMALL, seed=9)
    prob, s = _setup(ctx, dev, w, svc)
    g = gs.bcd_service_times(ctx, prob, s)
    G = svc.G
    delta = np.ones((w.C, G), np.uint8)
    svc.Mcap[:] = 1.0                      # the cached prefixes alone exceed every capacity
    s = gs.Service.from_model(svc, dev)
    z = np.ones(G, np.int32)
    r = gs.bcd_routing_lp(ctx, w.C, s, _t(np.full(w.C, 100.0), np.float64, dev), g["T"],
                          _t(np.zeros(G), np.float64, dev), _t(z, np.int32, dev),
                          _t(np.zeros(w.C), np.int32, dev), _t(delta, np.uint8, dev))
    torch.cuda.synchronize()
    assert r["info"].cpu().numpy()[1] == 2
    assert np.all(r["pi"].cpu().numpy() == 0.0)


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_reservation_sweep(ctx, dev, seed):
    import torch
    from paper_2607_16892_amd import serving as gs
    w, svc = serving_workload(C=6, N=4000, J=24, K=257, M=32, configs=SMALL, seed=seed)
    prob, s = _setup(ctx, dev, w, svc)
    W1 = oracle.W_table(w, oracle.S_exact(w))[0][0]
    T, ET2 = osv.service_times(svc, w)
    z, pi, delta, _ = _state(w, svc, seed)
    conc, cap = osv.lp2_inputs(svc, T, pi, z, delta)
    cap = cap * np.where(np.arange(svc.G) % 2 == 0, 0.2, 1.0)   # make some bounds bind
    rng = np.random.default_rng(seed)
    k_in = rng.integers(0, w.K, w.C).astype(np.int32)
    k_ref, ok_ref = osv.sweep(W1, w.eta, conc, cap, svc.kappa, k_in)
    r = gs.bcd_reservation_sweep(ctx, _t(W1, np.float64, dev), _t(w.eta, np.int32, dev),
                                 _t(conc, np.float64, dev), _t(cap, np.float64, dev), svc.kappa,
                                 _t(k_in, np.int32, dev))
    torch.cuda.synchronize()
    assert np.array_equal(r["k"].cpu().numpy(), k_ref)
    assert np.array_equal(r["feasible"].cpu().numpy().astype(bool), ok_ref)
    assert not np.array_equal(k_ref, np.argmin(W1, axis=1)), "no capacity bound was active"


@pytest.mark.parametrize("J", [16, 48])
def test_config_search(ctx, dev, J):
    import torch
    from paper_2607_16892_amd import serving as gs
    configs = SMALL if J == 16 else None
    w, svc = serving_workload(C=8, N=3000, J=J, K=129, M=16, configs=configs, seed=J)
    prob, s = _setup(ctx, dev, w, svc)
    g = gs.bcd_service_times(ctx, prob, s)
    T, ET2 = osv.service_times(svc, w)
    rng = np.random.default_rng(J)
    for trial in range(3):
        z = svc.z0.copy()
        pi = rng.dirichlet(np.ones(svc.G + 1), w.C)[:, :svc.G] * (z > 0)[None, :] * 0.3
        delta = (rng.random((w.C, svc.G)) < 0.2).astype(np.uint8)
        eta_c = rng.integers(0, 200, w.C).astype(np.int32)
        Wc = rng.uniform(50.0, 3000.0, w.C)
        zb, best, rank, nfeas = osv.config_search_vec(svc, Wc, T, ET2, pi, eta_c, delta)
        zt = _t(z, np.int32, dev)
        r = gs.bcd_config_search(ctx, w.C, s, _t(Wc, np.float64, dev), g["T"], g["ET2"],
                                 _t(pi, np.float64, dev), _t(eta_c, np.int32, dev),
                                 _t(delta, np.uint8, dev), zt)
        torch.cuda.synchronize()
        assert int(r["n_feasible"].cpu()[0]) == nfeas
        assert int(r["best_rank"].cpu()[0]) == rank
        assert _bits(r["best_objective"].cpu().numpy())[0] == _bits(np.array([best]))[0]
        keep = osv.feasible(svc, T, pi, z, eta_c, delta) and \
            osv.state_objective(svc, Wc, T, ET2, pi, z, eta_c, delta) == best
        assert np.array_equal(zt.cpu().numpy(), z if keep else zb)


@pytest.mark.parametrize("seed", [6, 7, 8, 11, 12, 13, 14, 15])
def test_alg1_matches_oracle(ctx, dev, seed):
    import torch
    from paper_2607_16892_amd import serving as gs
    w, svc = serving_workload(C=5, N=3000, J=16, K=257, M=32, configs=SMALL, seed=seed)
    prob, s = _setup(ctx, dev, w, svc)
    ref = osv.solve(w, svc)
    r = gs.dro_bcd_solve(ctx, prob, _t(w.eps[: w.C], np.float32, dev), s, svc.z0)
    torch.cuda.synchronize()
    print("  info", r["info"], "oracle outer/inner", ref["outer"], ref["inner"], flush=True)
    assert np.array_equal(r["z"].cpu().numpy(), ref["z"])
    assert np.array_equal(r["k"].cpu().numpy(), ref["k"])
    assert np.array_equal(r["delta"].cpu().numpy(), ref["delta"])
    assert np.max(np.abs(r["pi"].cpu().numpy() - ref["pi"])) <= 1e-7
    obj = float(r["objective"].cpu().numpy()[0])
    assert abs(obj - ref["objective"]) <= 1e-9 * abs(ref["objective"])
    assert r["info"]["outer"] == ref["outer"] and r["info"]["inner"] == ref["inner"]
    assert r["info"]["status"] & (1 | 2 | 4) == 0


def test_alg1_full_size_against_stored_oracle(ctx, dev):
    # 15 classes x 1e5 samples, K = 2048, M = 256, 12 configurations, 48 GPUs
    # (747,788 configurations per search)
    import json
    import os
    import torch
    from paper_2607_16892_amd import serving as gs
    path = os.path.join(os.path.dirname(__file__), "golden", "serving-15x100k.json")
    gold = json.load(open(path))
    w, svc = serving_workload(**gold["params"])
    assert w.checksum() == gold["checksum"]
    prob, s = _setup(ctx, dev, w, svc)
    r = gs.dro_bcd_solve(ctx, prob, _t(w.eps[: w.C], np.float32, dev), s, svc.z0)
    torch.cuda.synchronize()
    print("  info", r["info"], flush=True)
    assert r["z"].cpu().numpy().tolist() == gold["z"]
    assert r["k"].cpu().numpy().tolist() == gold["k"]
    assert r["delta"].cpu().numpy().tolist() == gold["delta"]
    ref_pi = np.array([[float.fromhex(v) for v in row] for row in gold["pi"]])
    assert np.max(np.abs(r["pi"].cpu().numpy() - ref_pi)) <= 1e-7
    obj, ref = float(r["objective"].cpu()[0]), float.fromhex(gold["objective"])
    assert abs(obj - ref) <= 1e-9 * abs(ref)
    assert (r["info"]["outer"], r["info"]["inner"]) == (gold["outer"], gold["inner"])
