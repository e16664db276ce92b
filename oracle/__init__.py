"""CPU oracle for the Wasserstein-DRO reservation path.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The product library never imports,
links or executes anything in this directory, and this package imports
nothing from the product.

`dro_oracle.c` holds the arithmetic (paper, Appendix A, Prop. A.1; Sec. 4.2
Prop. 4.2; Alg. 1); this module marshals numpy arrays into it.  The small
pure-Python routines in `brute.py` pin it to things other than itself.
"""
from __future__ import annotations

import ctypes as ct
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dro_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (fp64, no FMA contraction, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-std=gnu11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
               "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB):
                build(force=True)
            lib = ct.CDLL(_LIB)
            P = ct.c_void_p
            i32, i64, f32 = ct.c_int32, ct.c_int64, ct.c_float
            lib.oracle_threads.restype = ct.c_int
            lib.oracle_phi.restype = ct.c_double
            lib.oracle_phi.argtypes = [i32, i32, i32, f32, f32, f32]
            lib.oracle_phi_fix.restype = i64
            lib.oracle_phi_fix.argtypes = [i32, i32, i32, f32, f32, f32]
            lib.oracle_fix_ok.restype = ct.c_int
            lib.oracle_fix_ok.argtypes = [f32]
            lib.oracle_S_f64.restype = None
            lib.oracle_S_f64.argtypes = [i32, P, P, P, P, i32, P, i32, P, P, P, P]
            lib.oracle_S_exact.restype = ct.c_int
            lib.oracle_S_exact.argtypes = [i32, P, P, P, P, i32, P, i32, P, P, P, ct.c_int, P, P]
            lib.oracle_S_exact_at.restype = ct.c_int
            lib.oracle_S_exact_at.argtypes = [i32, P, P, P, P, P, P, P, P, i32, P, P, P, P, P]
            lib.oracle_fix_to_double.restype = ct.c_double
            lib.oracle_fix_to_double.argtypes = [i64, ct.c_uint64]
            lib.oracle_fix_to_double_n.restype = None
            lib.oracle_fix_to_double_n.argtypes = [i64, P, P, P]
            lib.oracle_J.restype = ct.c_double
            lib.oracle_J.argtypes = [i64, ct.c_uint64, f32, f32, i64]
            lib.oracle_W.restype = None
            lib.oracle_W.argtypes = [i32, i32, i32, i32, P, P, P, P, P, P, P]
            lib.oracle_argmin.restype = None
            lib.oracle_argmin.argtypes = [i32, i32, i32, P, P, P, P]
            lib.oracle_rank.restype = i64
            lib.oracle_rank.argtypes = [f32, f32, i64]
            lib.oracle_quantile.restype = None
            lib.oracle_quantile.argtypes = [i32, P, P, P, P, P, P, P]
            lib.oracle_bcd_step.restype = None
            lib.oracle_bcd_step.argtypes = [i32, i32, P, P, i32, P, P, f32, P, P, P, P, P]
            lib.oracle_bcd_init.restype = None
            lib.oracle_bcd_init.argtypes = [i32, P, P, P, i32, P, P]
            lib.oracle_moments.restype = None
            lib.oracle_moments.argtypes = [i32, P, P, P, P, P, P, P]
            lib.oracle_reservation_cost.restype = ct.c_int
            lib.oracle_reservation_cost.argtypes = [i32, P, P, P, P, P, i32, P, P, P, P, P]
            _lib = lib
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ct.c_void_p)


def _c(a, dt):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


def threads() -> int:
    return int(_load().oracle_threads())


def phi(eta, x, L, cp, cw, lam) -> float:
    """fp64 phi of App. A, Step 4 (three candidate points)."""
    return float(_load().oracle_phi(int(eta), int(x), int(L), float(cp), float(cw), float(lam)))


def phi_fix(eta, x, L, cp, cw, lam) -> int:
    """Exact phi in units of 2^-33."""
    return int(_load().oracle_phi_fix(int(eta), int(x), int(L), float(cp), float(cw), float(lam)))


def fix_ok(v) -> bool:
    return bool(_load().oracle_fix_ok(float(v)))


def _prob(w):
    return (_c(w.offsets, np.int64), None if w.seg is None else _c(w.seg, np.int32),
            _c(w.xi, np.int32), _c(w.L, np.int32), _c(w.eta, np.int32), _c(w.lam, np.float32),
            _c(w.c_p, np.float32), _c(w.c_w, np.float32))


def N_of(w) -> np.ndarray:
    return np.array([w.n_of(c) for c in range(w.C)], dtype=np.int64)


def S_f64(w) -> np.ndarray:
    """Dense fp64 S[c,k,m], every term evaluated, summed in sample order."""
    off, seg, xi, L, eta, lam, cp, cw = _prob(w)
    S = np.empty((w.C, w.K, w.M), np.float64)
    _load().oracle_S_f64(w.C, _p(off), _p(seg), _p(xi), _p(L), w.K, _p(eta), w.M, _p(lam),
                         _p(cp), _p(cw), _p(S))
    return S


class ExactS:
    """Exact S as 128-bit integers in units of 2^-33, kept as (hi, lo) words."""

    def __init__(self, hi: np.ndarray, lo: np.ndarray):
        self.hi, self.lo = hi, lo

    def as_int(self, idx) -> int:
        return (int(self.hi[idx]) << 64) | int(self.lo[idx])

    def to_double(self) -> np.ndarray:
        h = np.ascontiguousarray(self.hi, np.int64)
        l = np.ascontiguousarray(self.lo, np.uint64)
        out = np.empty(h.shape, np.float64)
        _load().oracle_fix_to_double_n(h.size, _p(h), _p(l), _p(out))
        return out


def S_exact(w, grouped: bool = True) -> ExactS:
    off, seg, xi, L, eta, lam, cp, cw = _prob(w)
    hi = np.empty((w.C, w.K, w.M), np.int64)
    lo = np.empty((w.C, w.K, w.M), np.uint64)
    rc = _load().oracle_S_exact(w.C, _p(off), _p(seg), _p(xi), _p(L), w.K, _p(eta), w.M, _p(lam),
                                _p(cp), _p(cw), int(bool(grouped)), _p(hi), _p(lo))
    if rc != 0:
        raise ValueError("a coefficient is outside the exact fixed-point range")
    return ExactS(hi, lo)


def S_exact_at(w, cs, ks, ms) -> ExactS:
    off, seg, xi, L, eta, lam, cp, cw = _prob(w)
    cs, ks, ms = (_c(a, np.int32) for a in (cs, ks, ms))
    P = cs.size
    hi = np.empty(P, np.int64)
    lo = np.empty(P, np.uint64)
    rc = _load().oracle_S_exact_at(w.C, _p(off), _p(seg), _p(xi), _p(L), _p(eta), _p(lam), _p(cp),
                                   _p(cw), P, _p(cs), _p(ks), _p(ms), _p(hi), _p(lo))
    if rc != 0:
        raise ValueError("a coefficient is outside the exact fixed-point range")
    return ExactS(hi, lo)


def J(hi: int, lo: int, lam: float, eps: float, N: int) -> float:
    return float(_load().oracle_J(int(hi), int(lo) & ((1 << 64) - 1), float(lam), float(eps), int(N)))


def W_table(w, S: ExactS, eps=None, E=None):
    """W[e,c,k] = min over m of J and the lowest minimising m."""
    eps = _c(w.eps if eps is None else eps, np.float32)
    E = w.E if E is None else E
    W = np.empty((E, w.C, w.K), np.float64)
    ms = np.empty((E, w.C, w.K), np.int32)
    _load().oracle_W(w.C, w.K, w.M, E, _p(_c(w.lam, np.float32)), _p(eps), _p(N_of(w)),
                     _p(S.hi), _p(S.lo), _p(W), _p(ms))
    return W, ms


def argmin(W: np.ndarray, kmax=None):
    E, C, K = W.shape
    ks = np.empty((E, C), np.int32)
    ws = np.empty((E, C), np.float64)
    _load().oracle_argmin(C, K, E, _p(_c(W, np.float64)), _p(_c(kmax, np.int32)), _p(ks), _p(ws))
    return ks, ws


def rank(cp, cw, N) -> int:
    return int(_load().oracle_rank(float(cp), float(cw), int(N)))


def quantile(w):
    off, seg, xi, L, eta, lam, cp, cw = _prob(w)
    qv = np.empty(w.C, np.int32)
    qr = np.empty(w.C, np.int64)
    _load().oracle_quantile(w.C, _p(off), _p(seg), _p(xi), _p(cp), _p(cw), _p(qv), _p(qr))
    return qv, qr


def bcd_init(w) -> np.ndarray:
    off, seg, xi, L, eta, lam, cp, cw = _prob(w)
    k0 = np.empty(w.C, np.int32)
    _load().oracle_bcd_init(w.C, _p(off), _p(seg), _p(xi), w.K, _p(eta), _p(k0))
    return k0


def bcd_step(w, W1: np.ndarray, k_prev):
    """One sweep; W1 is the [C, K] table of the single radius row."""
    g = w.groups
    C, K = w.C, w.K
    out = dict(k_next=np.empty(C, np.int32), W_star=np.empty(C, np.float64),
               usage=np.empty(g.G, np.float64), feasible=np.empty(C, np.uint8))
    _load().oracle_bcd_step(C, K, _p(_c(w.eta, np.int32)), _p(_c(W1, np.float64)), g.G,
                            _p(_c(g.cap, np.float32)), _p(_c(g.conc, np.float32)), float(g.kappa),
                            _p(_c(k_prev, np.int32)), _p(out["k_next"]), _p(out["W_star"]),
                            _p(out["usage"]), _p(out["feasible"]))
    return out


def solve(w, grouped: bool = True, kmax=None):
    """Everything the reservation path returns, computed exactly."""
    S = S_exact(w, grouped=grouped)
    W, ms = W_table(w, S)
    ks, ws = argmin(W, kmax)
    qv, qr = quantile(w)
    E = W.shape[0]
    m_at = np.array([[ms[e, c, ks[e, c]] for c in range(w.C)] for e in range(E)], np.int32)
    return dict(S=S, W=W, m_star=ms, k_star=ks, W_star=ws, m_at_star=m_at, q_value=qv, q_rank=qr)


def moments(w):
    """Per class: count, sum, sum of squares and largest sample (exact integers)."""
    off, seg, xi, L, eta, lam, cp, cw = _prob(w)
    out = dict(count=np.empty(w.C, np.int64), sum=np.empty(w.C, np.int64),
               sumsq=np.empty(w.C, np.int64), xmax=np.empty(w.C, np.int32))
    _load().oracle_moments(w.C, _p(off), _p(seg), _p(xi), _p(out["count"]), _p(out["sum"]),
                           _p(out["sumsq"]), _p(out["xmax"]))
    return out


def reservation_cost(w, eta_r):
    """Average cost of reservations eta_r[R, C] over each class's samples.

    Returns (cost [R, C] float64, cover [R, C] int64, exact sums as ExactS).
    """
    off, seg, xi, L, eta, lam, cp, cw = _prob(w)
    eta_r = np.ascontiguousarray(eta_r, dtype=np.int32).reshape(-1, w.C)
    R = eta_r.shape[0]
    cost = np.empty((R, w.C), np.float64)
    cover = np.empty((R, w.C), np.int64)
    hi = np.empty((R, w.C), np.int64)
    lo = np.empty((R, w.C), np.uint64)
    rc = _load().oracle_reservation_cost(w.C, _p(off), _p(seg), _p(xi), _p(cp), _p(cw), R,
                                         _p(eta_r), _p(cost), _p(cover), _p(hi), _p(lo))
    if rc != 0:
        raise ValueError("a coefficient is outside the exact fixed-point range")
    return cost, cover, ExactS(hi, lo)
