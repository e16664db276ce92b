"""Error behaviour of the C ABI (include/dro.h), driven from the host.

Every case here is rejected by host-side checks or by dro_validate before any
compute kernel could see the bad data, so no GPU work is done on invalid
inputs.  Outputs of a rejected call must stay untouched.
"""
import ctypes as ct

import numpy as np
import pytest

from workloads import random_workload

pytestmark = pytest.mark.gpu

EINVAL, ERANGE, ELIMIT = -1, -2, -5


@pytest.fixture(scope="module")
def ctx(dev):
    import paper_2607_16892_amd as dro
    c = dro.Context(dev.index or 0)
    yield c
    c.close()


def _problem(dev, **over):
    import paper_2607_16892_amd as dro
    w = random_workload(seed=31, C=2, N=(40, 25), L=200, K=17, M=9, E=1)
    fields = dict(offsets=w.offsets, xi=w.xi, L=w.L, eta=w.eta, lam=w.lam, c_p=w.c_p, c_w=w.c_w,
                  seg=w.seg, C=w.C)
    fields.update(over)
    return w, dro.Problem.from_arrays(dev, **fields)


def _validate_code(ctx, prob, eps=None):
    import paper_2607_16892_amd as dro
    try:
        dro.dro_validate(ctx, prob, eps)
    except dro.DroError as e:
        return e.code
    return 0


def test_valid_problem_passes(ctx, dev):
    import torch
    w, prob = _problem(dev)
    assert _validate_code(ctx, prob, torch.from_numpy(w.eps).to(dev)) == 0


@pytest.mark.parametrize("what, code", [
    ("sample_above_L", ERANGE), ("negative_sample", ERANGE), ("eta_not_ascending", ERANGE),
    ("eta_above_L", ERANGE), ("lam_not_ascending", ERANGE), ("lam_zero", ERANGE),
    ("lam_too_large", ELIMIT), ("cost_too_small", ELIMIT), ("L_too_large", ELIMIT),
    ("negative_eps", ERANGE), ("device_offsets_differ", ERANGE)])
def test_validate_rejects(ctx, dev, what, code):
    import torch
    w, prob = _problem(dev)
    eps = torch.from_numpy(w.eps).to(dev)
    if what == "sample_above_L":
        prob.xi[3] = int(w.L[0]) + 1
    elif what == "negative_sample":
        prob.xi[-1] = -2
    elif what == "eta_not_ascending":
        prob.eta[5] = prob.eta[4]
    elif what == "eta_above_L":
        prob.eta[-1] = int(w.L.min()) + 1
    elif what == "lam_not_ascending":
        prob.lam[3] = prob.lam[2]
    elif what == "lam_zero":
        prob.lam[0] = 0.0
    elif what == "lam_too_large":
        prob.lam[-1] = 1000.0
    elif what == "cost_too_small":
        prob.c_w[1] = 1e-4
    elif what == "L_too_large":
        prob.L[0] = 40000
    elif what == "negative_eps":
        eps[0] = -1.0
    elif what == "device_offsets_differ":
        prob.offsets[1] += 1
    assert _validate_code(ctx, prob, eps) == code


def test_host_checks_and_untouched_outputs(ctx, dev):
    import torch
    import paper_2607_16892_amd as dro
    lib = ctx._lib
    w, prob = _problem(dev)
    eps = torch.from_numpy(w.eps).to(dev)
    W = torch.full((1, w.C, w.K), 7.0, dtype=torch.float64, device=dev)
    stream = ct.c_void_p(torch.cuda.current_stream(dev).cuda_stream)

    def call(ps, E=1, eps_p=eps, W_p=W):
        return lib.dro_cost_eval(ctx.handle, ct.byref(ps), E, ct.c_void_p(eps_p.data_ptr())
                                 if eps_p is not None else None,
                                 ct.c_void_p(W_p.data_ptr()) if W_p is not None else None,
                                 None, None, stream)

    ps = prob.struct()
    ps.K = 0
    assert call(ps) == EINVAL
    ps = prob.struct()
    ps.xi = None
    assert call(ps) == EINVAL
    ps = prob.struct()
    assert call(ps, E=0) == EINVAL
    assert call(ps, W_p=None) == EINVAL
    assert call(ps, eps_p=None) == EINVAL
    # an empty class segment (host offsets) is rejected on the host
    off = w.offsets.copy()
    off[1] = off[0]
    off2 = np.concatenate([off[:2], w.offsets[2:]])
    bad = prob.struct()
    bad.offsets_h = off2.ctypes.data
    assert call(bad) == EINVAL
    # decreasing host offsets
    off3 = w.offsets.copy()
    off3[1] = off3[2] + 1
    bad.offsets_h = off3.ctypes.data
    assert call(bad) == EINVAL
    # a segment map on one side only
    bad = prob.struct()
    seg_h = np.array([0, 1], np.int32)
    bad.seg_h = seg_h.ctypes.data
    assert call(bad) == EINVAL
    # K beyond 2^15 + 1 grid points
    bad = prob.struct()
    bad.K = 40000
    assert call(bad) == ELIMIT
    # K and M each at their limit, but K * M beyond 2^31 - 1 grid pairs
    bad = prob.struct()
    bad.K = 32769
    bad.M = 65536
    assert call(bad) == ELIMIT
    assert "K*M" in ctx.last_error()
    # a class beyond 2^26 samples (rejected from the host offsets alone)
    big = w.offsets.copy()
    big[1:] += (1 << 26) + 1 - int(w.offsets[1])
    bad = prob.struct()
    bad.offsets_h = big.ctypes.data
    assert call(bad) == ELIMIT
    torch.cuda.synchronize()
    assert torch.all(W == 7.0), "a rejected call wrote its output"
    assert "NULL" in ctx.last_error() or "K=" in ctx.last_error() or ctx.last_error()
    # the context still works after the rejected calls
    r = dro.dro_cost_eval(ctx, prob, eps)
    torch.cuda.synchronize()
    assert torch.isfinite(r["W"]).all()


def test_entry_points_reject_null_outputs(ctx, dev):
    import torch
    w, prob = _problem(dev)
    lib = ctx._lib
    ps = prob.struct()
    stream = ct.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    assert lib.class_quantile(ctx.handle, ct.byref(ps), None, None, stream) == EINVAL
    assert lib.bcd_init_state(ctx.handle, ct.byref(ps), None, stream) == EINVAL
    assert lib.dro_argmin_reservation(ctx.handle, ct.byref(ps), 1, None, None, None, None, None,
                                      None, stream) == EINVAL
    assert lib.dro_exact_table(ctx.handle, ct.byref(ps), 1, None, None, None, None, None, None,
                               None, stream) == EINVAL
    assert lib.bcd_block_step(ctx.handle, ct.byref(ps), None, None, None, None, stream) == EINVAL


def test_serving_entry_points_reject_bad_arguments(ctx, dev):
    import torch
    from paper_2607_16892_amd import serving as gs
    from workloads.configs import serving_workload
    w, svc = serving_workload(C=3, N=500, J=8, K=33, M=8, configs=[(1, 1), (2, 1)], seed=1)
    lib = ctx._lib
    stream = ct.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    s = gs.Service.from_model(svc, dev)
    C, G = w.C, svc.G
    T = torch.zeros((C, G), dtype=torch.float64, device=dev)
    pi = torch.zeros((C, G), dtype=torch.float64, device=dev)
    z = torch.ones(G, dtype=torch.int32, device=dev)
    eta_c = torch.zeros(C, dtype=torch.int32, device=dev)
    delta = torch.zeros((C, G), dtype=torch.uint8, device=dev)
    Wq = torch.zeros(G, dtype=torch.float64, device=dev)
    out = torch.zeros(4 * C * G + 8, dtype=torch.float64, device=dev)

    def lp(ss):
        return lib.bcd_routing_lp(ctx.handle, C, ct.byref(ss), out.data_ptr(), T.data_ptr(),
                                  Wq.data_ptr(), z.data_ptr(), eta_c.data_ptr(),
                                  delta.data_ptr(), pi.data_ptr(), out.data_ptr(),
                                  z.data_ptr(), stream)

    ss = s.struct()
    ss.u_max = 1.0
    assert lp(ss) == EINVAL                  # the wait would not stay finite
    ss = s.struct()
    ss.G = 33
    assert lp(ss) == ELIMIT
    ss = s.struct()
    ss.J = 5000
    assert lp(ss) == ELIMIT
    ss = s.struct()
    ss.Lin = None
    assert lp(ss) == EINVAL
    ss = s.struct()
    bad = np.array([0, 1], np.int32)
    ss.tau_h = bad.ctypes.data
    assert lp(ss) == EINVAL                  # a configuration with no GPU
    assert lib.bcd_reservation_sweep(ctx.handle, C, 4, None, None, G, None, None, 0.2, None, None,
                                      None, stream) == EINVAL
    assert lib.bcd_prefix_cache(ctx.handle, 0, G, None, None, stream) == EINVAL
    zz = z.clone()
    ss = s.struct()
    assert lib.bcd_config_search(ctx.handle, C, ct.byref(ss), None, None, None, None, None, None,
                                 zz.data_ptr(), None, None, None, stream) == EINVAL
    torch.cuda.synchronize()
    assert torch.equal(zz, z)
