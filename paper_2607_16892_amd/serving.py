"""Binding of the serving-model entry points (routing LP, prefix caching,
configuration search and the Alg. 1 loop; include/dro.h).  Argument
marshalling only."""
from __future__ import annotations

import ctypes as ct
from dataclasses import dataclass

import numpy as np
import torch

from . import _native
from .api import Context, Problem, _need_dev, _ptr, _stream


@dataclass
class Service:
    """Device-resident serving model (field meanings as in dro_service)."""
    G: int
    tau: torch.Tensor
    pp: torch.Tensor
    tau_h: np.ndarray
    pp_h: np.ndarray
    Mcap: torch.Tensor
    Cc: torch.Tensor
    Bc: torch.Tensor
    lam: torch.Tensor
    Lin: torch.Tensor
    Lpre: torch.Tensor
    D: torch.Tensor
    alpha: float
    beta: float
    t_ar: float
    NL: int
    c_gpu: float
    c_slo: float
    c_rej: float
    kappa: float
    u_max: float
    J: int

    @classmethod
    def from_model(cls, m, device):
        """From any object with the dro_service fields as numpy arrays/scalars."""
        d = torch.device(device)

        def t(a, dt):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).to(d)

        return cls(G=int(len(m.tau)), tau=t(m.tau, np.int32), pp=t(m.pp, np.int32),
                   tau_h=np.ascontiguousarray(m.tau, np.int32),
                   pp_h=np.ascontiguousarray(m.pp, np.int32), Mcap=t(m.Mcap, np.float32),
                   Cc=t(m.Cc, np.float32), Bc=t(m.Bc, np.float32), lam=t(m.lam, np.float32),
                   Lin=t(m.Lin, np.int32), Lpre=t(m.Lpre, np.int32), D=t(m.D, np.float32),
                   alpha=float(m.alpha), beta=float(m.beta), t_ar=float(m.t_ar), NL=int(m.NL),
                   c_gpu=float(m.c_gpu), c_slo=float(m.c_slo), c_rej=float(m.c_rej),
                   kappa=float(m.kappa), u_max=float(m.u_max), J=int(m.J))

    def struct(self) -> _native.ServiceStruct:
        s = _native.ServiceStruct()
        s.G = self.G
        for name in ("tau", "pp", "Mcap", "Cc", "Bc", "lam", "Lin", "Lpre", "D"):
            setattr(s, name, getattr(self, name).data_ptr())
        s.tau_h = self.tau_h.ctypes.data
        s.pp_h = self.pp_h.ctypes.data
        for name in ("alpha", "beta", "t_ar", "c_gpu", "c_slo", "c_rej", "kappa", "u_max"):
            setattr(s, name, getattr(self, name))
        s.NL, s.J = self.NL, self.J
        return s


def _dev_out(shape, dtype, dev):
    return torch.empty(shape, dtype=dtype, device=dev)


def bcd_service_times(ctx: Context, prob: Problem, svc: Service, stream=None) -> dict:
    dev = prob.device
    T = _dev_out((prob.C, svc.G), torch.float64, dev)
    ET2 = _dev_out((prob.C, svc.G), torch.float64, dev)
    ps, ss = prob.struct(), svc.struct()
    rc = ctx._lib.bcd_service_times(ctx.handle, ct.byref(ps), ct.byref(ss), _ptr(T), _ptr(ET2),
                                    _stream(stream, dev))
    ctx.check(rc, "bcd_service_times")
    return dict(T=T, ET2=ET2)


def bcd_queue_state(ctx: Context, C: int, svc: Service, T, ET2, pi, z, eta_c, delta,
                    stream=None) -> dict:
    dev = T.device
    out = dict(Wq=_dev_out(svc.G, torch.float64, dev), cap=_dev_out(svc.G, torch.float64, dev),
               conc=_dev_out((C, svc.G), torch.float64, dev),
               mem=_dev_out(svc.G, torch.float64, dev))
    ss = svc.struct()
    rc = ctx._lib.bcd_queue_state(ctx.handle, C, ct.byref(ss), _ptr(T), _ptr(ET2), _ptr(pi),
                                  _ptr(z), _ptr(eta_c), _ptr(delta), _ptr(out["Wq"]),
                                  _ptr(out["cap"]), _ptr(out["conc"]), _ptr(out["mem"]),
                                  _stream(stream, dev))
    ctx.check(rc, "bcd_queue_state")
    return out


def bcd_routing_lp(ctx: Context, C: int, svc: Service, Wc, T, Wq, z, eta_c, delta,
                   stream=None) -> dict:
    dev = T.device
    for name, t, dt in (("Wc", Wc, torch.float64), ("T", T, torch.float64),
                        ("Wq", Wq, torch.float64), ("z", z, torch.int32),
                        ("eta_c", eta_c, torch.int32), ("delta", delta, torch.uint8)):
        _need_dev(t, dt, name, dev)
    pi = _dev_out((C, svc.G), torch.float64, dev)
    obj = _dev_out(1, torch.float64, dev)
    info = _dev_out(2, torch.int32, dev)
    ss = svc.struct()
    rc = ctx._lib.bcd_routing_lp(ctx.handle, C, ct.byref(ss), _ptr(Wc), _ptr(T), _ptr(Wq), _ptr(z),
                                 _ptr(eta_c), _ptr(delta), _ptr(pi), _ptr(obj), _ptr(info),
                                 _stream(stream, dev))
    ctx.check(rc, "bcd_routing_lp")
    return dict(pi=pi, objective=obj, info=info)


def bcd_reservation_sweep(ctx: Context, W, eta, conc, cap, kappa: float, k_in,
                          stream=None) -> dict:
    dev = W.device
    C, K = W.shape
    G = cap.numel()
    for name, t, dt in (("W", W, torch.float64), ("eta", eta, torch.int32),
                        ("conc", conc, torch.float64), ("cap", cap, torch.float64),
                        ("k_in", k_in, torch.int32)):
        _need_dev(t, dt, name, dev)
    k_out = _dev_out(C, torch.int32, dev)
    feas = _dev_out(C, torch.uint8, dev)
    rc = ctx._lib.bcd_reservation_sweep(ctx.handle, C, K, _ptr(W), _ptr(eta), G, _ptr(conc),
                                        _ptr(cap), float(kappa), _ptr(k_in), _ptr(k_out),
                                        _ptr(feas), _stream(stream, dev))
    ctx.check(rc, "bcd_reservation_sweep")
    return dict(k=k_out, feasible=feas)


def bcd_prefix_cache(ctx: Context, conc, stream=None) -> torch.Tensor:
    dev = conc.device
    _need_dev(conc, torch.float64, "conc", dev)
    C, G = conc.shape
    delta = _dev_out((C, G), torch.uint8, dev)
    rc = ctx._lib.bcd_prefix_cache(ctx.handle, C, G, _ptr(conc), _ptr(delta), _stream(stream, dev))
    ctx.check(rc, "bcd_prefix_cache")
    return delta


def bcd_config_search(ctx: Context, C: int, svc: Service, Wc, T, ET2, pi, eta_c, delta, z,
                      stream=None) -> dict:
    """z (device int32 [G]) is updated in place."""
    dev = T.device
    _need_dev(z, torch.int32, "z", dev)
    best = _dev_out(1, torch.float64, dev)
    rank = _dev_out(1, torch.int64, dev)
    nfeas = _dev_out(1, torch.int64, dev)
    ss = svc.struct()
    rc = ctx._lib.bcd_config_search(ctx.handle, C, ct.byref(ss), _ptr(Wc), _ptr(T), _ptr(ET2),
                                    _ptr(pi), _ptr(eta_c), _ptr(delta), _ptr(z), _ptr(best),
                                    _ptr(rank), _ptr(nfeas), _stream(stream, dev))
    ctx.check(rc, "bcd_config_search")
    return dict(z=z, best_objective=best, best_rank=rank, n_feasible=nfeas)


def dro_bcd_solve(ctx: Context, prob: Problem, eps: torch.Tensor, svc: Service, z0,
                  max_outer: int = 10, max_inner: int = 10, stream=None) -> dict:
    """Alg. 1 (see dro_bcd_solve in dro.h); returns the final state."""
    dev = prob.device
    _need_dev(eps, torch.float32, "eps", dev)
    z = torch.as_tensor(np.ascontiguousarray(z0, np.int32)).to(dev) if not torch.is_tensor(z0) \
        else z0.to(device=dev, dtype=torch.int32).clone()
    C, G = prob.C, svc.G
    out = dict(z=z, k=_dev_out(C, torch.int32, dev), pi=_dev_out((C, G), torch.float64, dev),
               delta=_dev_out((C, G), torch.uint8, dev),
               objective=_dev_out(1, torch.float64, dev))
    info = (ct.c_int32 * 4)()
    ps, ss = prob.struct(), svc.struct()
    rc = ctx._lib.dro_bcd_solve(ctx.handle, ct.byref(ps), _ptr(eps), ct.byref(ss), int(max_outer),
                                int(max_inner), _ptr(out["z"]), _ptr(out["k"]), _ptr(out["pi"]),
                                _ptr(out["delta"]), _ptr(out["objective"]),
                                ct.cast(info, ct.c_void_p), _stream(stream, dev))
    ctx.check(rc, "dro_bcd_solve")
    out["info"] = dict(outer=info[0], inner=info[1], pivots=info[2], status=info[3])
    return out
