"""Parity of class_moments and dro_reservation_cost (C ABI) with the CPU oracle.

Bars: every output is an exact integer or the fully specified double
RN(RN(S) / N) of an exact sum, so all of them are compared bit for bit.
"""
import numpy as np
import pytest

import oracle
from workloads import make_workload, random_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx(dev):
    import paper_2607_16892_amd as dro
    c = dro.Context(dev.index or 0)
    yield c
    c.close()


def _gpu(ctx, w, dev, eta_r):
    import torch
    import paper_2607_16892_amd as dro
    print(f"[gpu] reservation cost {w.name} C={w.C} N={w.offsets[-1]} R={eta_r.shape[0]}",
          flush=True)
    prob = dro.Problem.from_workload(w, dev)
    dro.dro_validate(ctx, prob)
    mo = dro.class_moments(ctx, prob)
    rc = dro.dro_reservation_cost(ctx, prob, torch.from_numpy(np.ascontiguousarray(eta_r)).to(dev))
    torch.cuda.synchronize()
    return ({k: v.cpu().numpy() for k, v in mo.items()},
            {k: v.cpu().numpy() for k, v in rc.items()})


def _check(w, mo, rc, eta_r):
    ref_m = oracle.moments(w)
    for k in ("count", "sum", "sumsq", "xmax"):
        assert np.array_equal(mo[k], ref_m[k]), k
    cost, cover, _ = oracle.reservation_cost(w, eta_r)
    assert np.array_equal(rc["cover"], cover)
    assert np.array_equal(rc["cost"].view(np.uint64), cost.view(np.uint64))


RANDOM = [
    dict(seed=301, C=3, N=(50, 7, 130), L=300),
    dict(seed=302, C=5, N=(1, 2, 3000, 17, 40000), L=32768),
    dict(seed=303, C=7, N=(5000, 64, 65, 1023), L=4096, alias=True),
    dict(seed=304, C=2, N=(200_000, 3), L=8192, dist="uniform"),
    dict(seed=306, C=2, N=(999, 1000), L=700, dist="constant"),
]


@pytest.mark.parametrize("case", RANDOM, ids=lambda c: f"seed{c['seed']}")
def test_random_workloads(ctx, dev, case):
    w = random_workload(K=8, M=4, E=1, **case)
    rng = np.random.default_rng(case["seed"])
    L = int(w.L.max())
    eta_r = rng.integers(-3, L + 20, size=(9, w.C)).astype(np.int32)
    eta_r[0] = 0
    eta_r[1] = w.L
    eta_r[2] = -(1 << 31)                    # the extremes of int32
    eta_r[3] = (1 << 31) - 1
    mo, rc = _gpu(ctx, w, dev, eta_r)
    _check(w, mo, rc, eta_r)


def test_full_size_and_critical_fractile(ctx, dev):
    # 16 classes x 1e6 samples: exact at reservations around each class's
    # critical-fractile quantile, where the cost is smallest (Prop. 4.2).
    import torch
    import paper_2607_16892_amd as dro
    w = make_workload("mixture-16x1M")
    prob = dro.Problem.from_workload(w, dev)
    q = dro.class_quantile(ctx, prob)["q_value"].cpu().numpy().astype(np.int64)
    offs = np.array([-50, -7, -1, 0, 1, 7, 50])
    eta_r = (q[None, :] + offs[:, None]).astype(np.int32)
    mo, rc = _gpu(ctx, w, dev, eta_r)
    _check(w, mo, rc, eta_r)
    c = rc["cost"]
    assert np.all(c[3] <= c), "the quantile is not the cheapest reservation"
    # and the smallest such reservation: one token less costs strictly more
    assert np.all(c[2] > c[3])


def test_rejects_bad_arguments(ctx, dev):
    import torch
    import paper_2607_16892_amd as dro
    w = random_workload(seed=305, C=2, N=(10, 12), L=50, K=4, M=3, E=1)
    prob = dro.Problem.from_workload(w, dev)
    with pytest.raises(ValueError):
        dro.dro_reservation_cost(ctx, prob, torch.zeros(3, dtype=torch.int32, device=dev))
    lib = ctx._lib
    import ctypes as ct
    ps = prob.struct()
    stream = ct.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    assert lib.dro_reservation_cost(ctx.handle, ct.byref(ps), 0, None, None, None, stream) == -1
    assert lib.class_moments(ctx.handle, ct.byref(ps), None, None, None, None, stream) == -1
