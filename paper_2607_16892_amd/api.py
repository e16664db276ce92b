"""Python binding of the C ABI in include/dro.h, with the same entry-point names.

Device memory and streams come from PyTorch; every step of the path runs in
the HIP kernels of libdro.so.  Inputs must be CUDA (ROCm) tensors; nothing
here computes a cost, a dual, a quantile or an argmin.
"""
from __future__ import annotations

import ctypes as ct
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

from . import _native


class DroError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str):
        self.code = code
        super().__init__(f"{where} failed with {code} ({detail})")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ct.c_void_p(t.data_ptr())


def _stream(stream, device) -> ct.c_void_p:
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return ct.c_void_p(s.cuda_stream)


def _need_dev(t: torch.Tensor, dtype, name: str, device):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


class Context:
    """A dro_ctx bound to one HIP device (one per host thread / stream)."""

    def __init__(self, device=0):
        self.device = torch.device("cuda", device) if isinstance(device, int) else torch.device(device)
        self._lib = _native.load()
        h = ct.c_void_p()
        rc = self._lib.dro_create(self.device.index or 0, ct.byref(h))
        if rc != 0:
            raise DroError(rc, "dro_create", self._lib.dro_strerror(rc).decode())
        self._h = h

    @property
    def handle(self):
        return self._h

    def close(self):
        if getattr(self, "_h", None):
            self._lib.dro_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def last_error(self) -> str:
        return self._lib.dro_last_error(self._h).decode()

    def check(self, rc: int, where: str):
        if rc != 0:
            raise DroError(rc, where, f"{self._lib.dro_strerror(rc).decode()}: {self.last_error()}")


@dataclass
class Problem:
    """Device-resident reservation problem (field meanings as in dro_problem)."""
    C: int
    S: int
    K: int
    M: int
    offsets: torch.Tensor          # int64 [S+1] device
    offsets_h: np.ndarray          # int64 [S+1] host copy
    seg: Optional[torch.Tensor]    # int32 [C] device or None
    seg_h: Optional[np.ndarray]    # int32 [C] host copy or None
    xi: torch.Tensor               # int32 device
    L: torch.Tensor                # int32 [C]
    eta: torch.Tensor              # int32 [K]
    lam: torch.Tensor              # float32 [M]
    c_p: torch.Tensor              # float32 [C]
    c_w: torch.Tensor              # float32 [C]

    @property
    def device(self):
        return self.xi.device

    @classmethod
    def from_arrays(cls, device, offsets, xi, L, eta, lam, c_p, c_w, seg=None, C=None):
        dev = torch.device(device)
        off_h = np.ascontiguousarray(offsets, dtype=np.int64)
        seg_h = None if seg is None else np.ascontiguousarray(seg, dtype=np.int32)
        S = int(off_h.shape[0] - 1)
        C = int(len(c_p)) if C is None else int(C)

        def d(a, dt):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).to(dev)

        return cls(C=C, S=S, K=int(len(eta)), M=int(len(lam)), offsets=d(off_h, np.int64),
                   offsets_h=off_h, seg=None if seg_h is None else d(seg_h, np.int32), seg_h=seg_h,
                   xi=d(xi, np.int32), L=d(L, np.int32), eta=d(eta, np.int32),
                   lam=d(lam, np.float32), c_p=d(c_p, np.float32), c_w=d(c_w, np.float32))

    @classmethod
    def from_workload(cls, w, device):
        return cls.from_arrays(device, w.offsets, w.xi, w.L, w.eta, w.lam, w.c_p, w.c_w,
                               seg=w.seg, C=w.C)

    def replace_samples(self, offsets, xi):
        """New samples with the same segment count (drifting data), uploaded in place."""
        off_h = np.ascontiguousarray(offsets, dtype=np.int64)
        if off_h.shape != self.offsets_h.shape:
            raise ValueError("segment count changed")
        self.offsets_h = off_h
        self.offsets.copy_(torch.from_numpy(off_h))
        x = torch.from_numpy(np.ascontiguousarray(xi, dtype=np.int32))
        if x.numel() == self.xi.numel():
            self.xi.copy_(x)
        else:
            self.xi = x.to(self.device)

    def n_of(self, c: int) -> int:
        s = c if self.seg_h is None else int(self.seg_h[c])
        return int(self.offsets_h[s + 1] - self.offsets_h[s])

    def struct(self) -> _native.ProblemStruct:
        for name in ("offsets", "xi", "L", "eta", "lam", "c_p", "c_w"):
            t = getattr(self, name)
            if not t.is_cuda:
                raise TypeError(f"problem field {name} must be a CUDA tensor")
        ps = _native.ProblemStruct()
        ps.C, ps.S, ps.K, ps.M = self.C, self.S, self.K, self.M
        ps.offsets = self.offsets.data_ptr()
        ps.offsets_h = self.offsets_h.ctypes.data
        ps.seg = None if self.seg is None else self.seg.data_ptr()
        ps.seg_h = None if self.seg_h is None else self.seg_h.ctypes.data
        ps.xi = self.xi.data_ptr()
        ps.L = self.L.data_ptr()
        ps.eta = self.eta.data_ptr()
        ps.lam = self.lam.data_ptr()
        ps.c_p = self.c_p.data_ptr()
        ps.c_w = self.c_w.data_ptr()
        return ps


def _out(t, shape, dtype, device, name):
    if t is None:
        return torch.empty(shape, dtype=dtype, device=device)
    _need_dev(t, dtype, name, device)
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}")
    return t


def dro_validate(ctx: Context, prob: Problem, eps: Optional[torch.Tensor] = None, E: int = 0,
                 stream=None) -> None:
    ps = prob.struct()
    if eps is not None:
        _need_dev(eps, torch.float32, "eps", prob.device)
        E = E or eps.numel() // prob.C
    rc = ctx._lib.dro_validate(ctx.handle, ct.byref(ps), E, _ptr(eps), _stream(stream, prob.device))
    ctx.check(rc, "dro_validate")


def dro_cost_eval(ctx: Context, prob: Problem, eps: torch.Tensor, W=None, m_star=None, S=None,
                  want_S: bool = True, want_m_star: bool = True, stream=None) -> dict:
    """S[c,k,m], W[e,c,k] = min_m J and m_star (see dro_cost_eval in dro.h)."""
    dev = prob.device
    _need_dev(eps, torch.float32, "eps", dev)
    E = eps.numel() // prob.C
    if E * prob.C != eps.numel() or E <= 0:
        raise ValueError("eps must hold E*C radii")
    W = _out(W, (E, prob.C, prob.K), torch.float64, dev, "W")
    if want_m_star or m_star is not None:
        m_star = _out(m_star, (E, prob.C, prob.K), torch.int32, dev, "m_star")
    if want_S or S is not None:
        S = _out(S, (prob.C, prob.K, prob.M), torch.float64, dev, "S")
    ps = prob.struct()
    rc = ctx._lib.dro_cost_eval(ctx.handle, ct.byref(ps), E, _ptr(eps), _ptr(W), _ptr(m_star),
                                _ptr(S), _stream(stream, dev))
    ctx.check(rc, "dro_cost_eval")
    return dict(W=W, m_star=m_star, S=S)


def dro_cost_eval_noalloc(ctx: Context, prob: Problem, eps: torch.Tensor, S: torch.Tensor,
                          W: torch.Tensor, m_star: Optional[torch.Tensor] = None,
                          stream=None) -> dict:
    """dro_cost_eval with the library's static scratch array (see dro_cost_eval_noalloc in
    dro.h): every output is the caller's, S included."""
    dev = prob.device
    _need_dev(eps, torch.float32, "eps", dev)
    E = eps.numel() // prob.C
    if E * prob.C != eps.numel() or E <= 0:
        raise ValueError("eps must hold E*C radii")
    S = _out(S, (prob.C, prob.K, prob.M), torch.float64, dev, "S")
    W = _out(W, (E, prob.C, prob.K), torch.float64, dev, "W")
    if m_star is not None:
        m_star = _out(m_star, (E, prob.C, prob.K), torch.int32, dev, "m_star")
    ps = prob.struct()
    rc = ctx._lib.dro_cost_eval_noalloc(ctx.handle, ct.byref(ps), E, _ptr(eps), _ptr(W),
                                        _ptr(m_star), _ptr(S), _stream(stream, dev))
    ctx.check(rc, "dro_cost_eval_noalloc")
    return dict(W=W, m_star=m_star, S=S)


def dro_argmin_reservation(ctx: Context, prob: Problem, eps: torch.Tensor, S: torch.Tensor,
                           k_max: Optional[torch.Tensor] = None, k_star=None, W_star=None,
                           m_at_star=None, stream=None) -> dict:
    """Exact lowest-index optimum per (e, c) (see dro_argmin_reservation in dro.h)."""
    dev = prob.device
    _need_dev(eps, torch.float32, "eps", dev)
    _need_dev(S, torch.float64, "S", dev)
    if k_max is not None:
        _need_dev(k_max, torch.int32, "k_max", dev)
    E = eps.numel() // prob.C
    k_star = _out(k_star, (E, prob.C), torch.int32, dev, "k_star")
    W_star = _out(W_star, (E, prob.C), torch.float64, dev, "W_star")
    m_at_star = _out(m_at_star, (E, prob.C), torch.int32, dev, "m_at_star")
    ps = prob.struct()
    rc = ctx._lib.dro_argmin_reservation(ctx.handle, ct.byref(ps), E, _ptr(eps), _ptr(S),
                                         _ptr(k_max), _ptr(k_star), _ptr(W_star), _ptr(m_at_star),
                                         _stream(stream, dev))
    ctx.check(rc, "dro_argmin_reservation")
    return dict(k_star=k_star, W_star=W_star, m_at_star=m_at_star)


def dro_exact_table(ctx: Context, prob: Problem, eps: torch.Tensor,
                    k_max: Optional[torch.Tensor] = None, want_argmin: bool = True,
                    stream=None) -> dict:
    """Exact W table, m_star and optimum from value counts (see dro_exact_table in dro.h)."""
    dev = prob.device
    _need_dev(eps, torch.float32, "eps", dev)
    if k_max is not None:
        _need_dev(k_max, torch.int32, "k_max", dev)
    E = eps.numel() // prob.C
    if E * prob.C != eps.numel() or E <= 0:
        raise ValueError("eps must hold E*C radii")
    W = torch.empty((E, prob.C, prob.K), dtype=torch.float64, device=dev)
    m_star = torch.empty((E, prob.C, prob.K), dtype=torch.int32, device=dev)
    k_star = W_star = m_at_star = None
    if want_argmin:
        k_star = torch.empty((E, prob.C), dtype=torch.int32, device=dev)
        W_star = torch.empty((E, prob.C), dtype=torch.float64, device=dev)
        m_at_star = torch.empty((E, prob.C), dtype=torch.int32, device=dev)
    ps = prob.struct()
    rc = ctx._lib.dro_exact_table(ctx.handle, ct.byref(ps), E, _ptr(eps), _ptr(k_max), _ptr(W),
                                  _ptr(m_star), _ptr(k_star), _ptr(W_star), _ptr(m_at_star),
                                  _stream(stream, dev))
    ctx.check(rc, "dro_exact_table")
    return dict(W=W, m_star=m_star, k_star=k_star, W_star=W_star, m_at_star=m_at_star)


def dro_continuous_dual(ctx: Context, prob: Problem, eps: torch.Tensor, stream=None) -> dict:
    """min over continuous gamma >= 0 of the dual, per (e, c, k) (see dro_continuous_dual in dro.h)."""
    dev = prob.device
    _need_dev(eps, torch.float32, "eps", dev)
    E = eps.numel() // prob.C
    if E * prob.C != eps.numel() or E <= 0:
        raise ValueError("eps must hold E*C radii")
    W = torch.empty((E, prob.C, prob.K), dtype=torch.float64, device=dev)
    gamma = torch.empty((E, prob.C, prob.K), dtype=torch.float64, device=dev)
    ps = prob.struct()
    rc = ctx._lib.dro_continuous_dual(ctx.handle, ct.byref(ps), E, _ptr(eps), _ptr(W), _ptr(gamma),
                                      _stream(stream, dev))
    ctx.check(rc, "dro_continuous_dual")
    return dict(W=W, gamma=gamma)


def class_quantile(ctx: Context, prob: Problem, q_value=None, q_rank=None, stream=None) -> dict:
    dev = prob.device
    q_value = _out(q_value, (prob.C,), torch.int32, dev, "q_value")
    q_rank = _out(q_rank, (prob.C,), torch.int64, dev, "q_rank")
    ps = prob.struct()
    rc = ctx._lib.class_quantile(ctx.handle, ct.byref(ps), _ptr(q_value), _ptr(q_rank),
                                 _stream(stream, dev))
    ctx.check(rc, "class_quantile")
    return dict(q_value=q_value, q_rank=q_rank)


def class_moments(ctx: Context, prob: Problem, stream=None) -> dict:
    """Per-class count, sum, sum of squares and largest sample (see class_moments in dro.h)."""
    dev = prob.device
    out = dict(count=torch.empty(prob.C, dtype=torch.int64, device=dev),
               sum=torch.empty(prob.C, dtype=torch.int64, device=dev),
               sumsq=torch.empty(prob.C, dtype=torch.int64, device=dev),
               xmax=torch.empty(prob.C, dtype=torch.int32, device=dev))
    ps = prob.struct()
    rc = ctx._lib.class_moments(ctx.handle, ct.byref(ps), _ptr(out["count"]), _ptr(out["sum"]),
                                _ptr(out["sumsq"]), _ptr(out["xmax"]), _stream(stream, dev))
    ctx.check(rc, "class_moments")
    return out


def dro_baseline_reservations(ctx: Context, moments: dict, L: torch.Tensor, k_sigma=(),
                              q: Optional[torch.Tensor] = None, block: int = 16,
                              stream=None) -> dict:
    """Mean, mean + k sigma and block-aligned reservations from class moments
    (see dro_baseline_reservations in dro.h)."""
    dev = L.device
    C = int(L.shape[0])
    for name in ("count", "sum", "sumsq"):
        _need_dev(moments[name], torch.int64, name, dev)
    _need_dev(L, torch.int32, "L", dev)
    if q is not None:
        _need_dev(q, torch.int32, "q", dev)
    ks = np.ascontiguousarray(list(k_sigma), dtype=np.int32)
    out = dict(mean=torch.empty(C, dtype=torch.int32, device=dev),
               lp=torch.empty((len(ks), C), dtype=torch.int32, device=dev),
               block=None if q is None else torch.empty(C, dtype=torch.int32, device=dev))
    rc = ctx._lib.dro_baseline_reservations(
        ctx.handle, C, _ptr(moments["count"]), _ptr(moments["sum"]), _ptr(moments["sumsq"]),
        _ptr(L), len(ks), ks.ctypes.data if len(ks) else None, _ptr(q), block, _ptr(out["mean"]),
        _ptr(out["lp"]) if len(ks) else None, _ptr(out["block"]), _stream(stream, dev))
    ctx.check(rc, "dro_baseline_reservations")
    return out


def dro_reservation_cost(ctx: Context, prob: Problem, eta_r: torch.Tensor, stream=None) -> dict:
    """Average cost of reservations eta_r[R, C] (see dro_reservation_cost in dro.h)."""
    dev = prob.device
    _need_dev(eta_r, torch.int32, "eta_r", dev)
    R = eta_r.numel() // prob.C
    if R * prob.C != eta_r.numel() or R <= 0:
        raise ValueError("eta_r must hold R*C reservations")
    cost = torch.empty((R, prob.C), dtype=torch.float64, device=dev)
    cover = torch.empty((R, prob.C), dtype=torch.int64, device=dev)
    ps = prob.struct()
    rc = ctx._lib.dro_reservation_cost(ctx.handle, ct.byref(ps), R, _ptr(eta_r), _ptr(cost),
                                       _ptr(cover), _stream(stream, dev))
    ctx.check(rc, "dro_reservation_cost")
    return dict(cost=cost, cover=cover)


def bcd_init_state(ctx: Context, prob: Problem, k0=None, stream=None) -> torch.Tensor:
    dev = prob.device
    k0 = _out(k0, (prob.C,), torch.int32, dev, "k0")
    ps = prob.struct()
    rc = ctx._lib.bcd_init_state(ctx.handle, ct.byref(ps), _ptr(k0), _stream(stream, dev))
    ctx.check(rc, "bcd_init_state")
    return k0


@dataclass
class Groups:
    cap: torch.Tensor     # float32 [G]
    conc: torch.Tensor    # float32 [C*G]
    kappa: float

    @classmethod
    def from_numpy(cls, cap, conc, kappa, device):
        d = torch.device(device)
        return cls(torch.from_numpy(np.ascontiguousarray(cap, np.float32)).to(d),
                   torch.from_numpy(np.ascontiguousarray(conc, np.float32)).to(d), float(kappa))


def bcd_block_step(ctx: Context, prob: Problem, eps: torch.Tensor, groups: Groups,
                   k_prev: torch.Tensor, out: Optional[dict] = None, stream=None) -> dict:
    """One capacity-constrained reservation sweep (see bcd_block_step in dro.h)."""
    dev = prob.device
    _need_dev(eps, torch.float32, "eps", dev)
    _need_dev(k_prev, torch.int32, "k_prev", dev)
    _need_dev(groups.cap, torch.float32, "cap", dev)
    _need_dev(groups.conc, torch.float32, "conc", dev)
    G = groups.cap.numel()
    if groups.conc.numel() != G * prob.C:
        raise ValueError("conc must hold C*G entries")
    out = out or {}
    o = dict(k_next=_out(out.get("k_next"), (prob.C,), torch.int32, dev, "k_next"),
             W_star=_out(out.get("W_star"), (prob.C,), torch.float64, dev, "W_star"),
             q_value=_out(out.get("q_value"), (prob.C,), torch.int32, dev, "q_value"),
             usage=_out(out.get("usage"), (G,), torch.float64, dev, "usage"),
             feasible=_out(out.get("feasible"), (prob.C,), torch.uint8, dev, "feasible"))
    gs = _native.GroupsStruct(G, groups.cap.data_ptr(), groups.conc.data_ptr(), groups.kappa)
    so = _native.StepOutStruct(o["k_next"].data_ptr(), o["W_star"].data_ptr(),
                               o["q_value"].data_ptr(), o["usage"].data_ptr(),
                               o["feasible"].data_ptr())
    ps = prob.struct()
    rc = ctx._lib.bcd_block_step(ctx.handle, ct.byref(ps), _ptr(eps), ct.byref(gs), _ptr(k_prev),
                                 ct.byref(so), _stream(stream, dev))
    ctx.check(rc, "bcd_block_step")
    return o
