"""Seeded synthetic stand-ins for the paper's output-length traces.

The paper evaluates on production traces (BurstGPT, Azure LLM 2024, ShareGPT;
Sec. 5.1 "Experiment Setup") that are not available here.  The five workloads
below are synthetic, seeded and heavy-tailed, with the class counts, sample
counts, grid sizes, radii and cost ratios of the benchmark configurations:

  lognormal-1x1k    1 class x 1,000       lognormal(5, 1), clip [1, 4096]         K=64   M=32
  lognormal-4x100k  4 classes x 100,000   lognormal, means 50/300/1500/600         K=512  M=128
  mixture-16x1M     16 classes x 1e6      2-component lognormal mixture + Lomax    K=2048 M=256
  ratios-8x250k     8 segments x 250,000, 16 cost ratios x 16 radii                K=1024 M=128
  drift-8x4M        8 classes x 4e6, mean drifting 1 %/iteration, 6 groups         K=2048 M=256

Everything here is input generation: draws, rounding to integer lengths,
the reservation and multiplier grids, radii as a fraction of the sample mean,
and cost coefficients.  Nothing computes a cost, a dual, a quantile or an
argmin.
"""
from __future__ import annotations

import functools
import math
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

CONFIG_NAMES = ("lognormal-1x1k", "lognormal-4x100k", "mixture-16x1M", "ratios-8x250k",
                "drift-8x4M")

# Sample lengths, grid points and support bounds are integers no larger than
# 2**15; cost coefficients and multipliers lie in [2**-10, 2**7].
MAX_LEN = 1 << 15


@dataclass
class Groups:
    """Serving-group capacity data for one block step (the memory-capacity constraint of Sec. 3.4)."""
    cap: np.ndarray      # float32 [G]   KV capacity of each group, tokens
    conc: np.ndarray     # float32 [C*G] expected concurrent class-c requests on group g
    kappa: float         # safety factor (float32 value)

    @property
    def G(self) -> int:
        return int(self.cap.shape[0])


@dataclass
class Workload:
    name: str
    C: int                       # classes (problem rows)
    offsets: np.ndarray          # int64 [S+1] CSR bounds of the sample segments
    seg: Optional[np.ndarray]    # int32 [C] segment of each class, None = identity
    xi: np.ndarray               # int32 [offsets[-1]] output-length samples
    L: np.ndarray                # int32 [C] support upper bound of each class
    eta: np.ndarray              # int32 [K] ascending reservation (buffer) grid
    lam: np.ndarray              # float32 [M] ascending multiplier grid
    c_p: np.ndarray              # float32 [C] preemption cost per token
    c_w: np.ndarray              # float32 [C] waste cost per token
    E: int                       # radii per class
    eps: np.ndarray              # float32 [E*C] Wasserstein radius, tokens, row e*C + c
    groups: Optional[Groups] = None
    meta: dict = field(default_factory=dict)

    @property
    def K(self) -> int:
        return int(self.eta.shape[0])

    @property
    def M(self) -> int:
        return int(self.lam.shape[0])

    @property
    def S(self) -> int:
        return int(self.offsets.shape[0] - 1)

    def seg_of(self, c: int) -> int:
        return c if self.seg is None else int(self.seg[c])

    def n_of(self, c: int) -> int:
        s = self.seg_of(c)
        return int(self.offsets[s + 1] - self.offsets[s])

    def samples_of(self, c: int) -> np.ndarray:
        s = self.seg_of(c)
        return self.xi[self.offsets[s]:self.offsets[s + 1]]

    @property
    def evals(self) -> int:
        """Number of (class, grid point, multiplier, sample) terms."""
        return sum(self.n_of(c) for c in range(self.C)) * self.K * self.M

    def checksum(self) -> str:
        """Content hash of every input array (detects generator drift)."""
        import hashlib
        h = hashlib.sha256()
        for a in (self.offsets, self.xi, self.L, self.eta, self.lam, self.c_p, self.c_w, self.eps):
            h.update(np.ascontiguousarray(a).tobytes())
        if self.seg is not None:
            h.update(np.ascontiguousarray(self.seg).tobytes())
        if self.groups is not None:
            h.update(self.groups.cap.tobytes())
            h.update(self.groups.conc.tobytes())
        return h.hexdigest()[:16]


# ---------------------------------------------------------------- grids ----

def eta_grid(K: int, L: int) -> np.ndarray:
    """K integer reservation levels spread uniformly over [0, L].

    Point k is k*L/(K-1) rounded half-up, i.e. floor((2kL + K - 1) / (2(K-1))),
    so the grid holds 0 and L and is strictly ascending whenever K - 1 <= L.
    """
    if K == 1:
        return np.zeros(1, dtype=np.int32)
    k = np.arange(K, dtype=np.int64)
    return ((2 * k * L + K - 1) // (2 * (K - 1))).astype(np.int32)


def lam_grid(M: int, lo: float = 1e-3, hi: float = 1e2) -> np.ndarray:
    """M multipliers log-spaced on [lo, hi], each rounded once to float32."""
    if M == 1:
        return np.array([hi], dtype=np.float32)
    a, b = math.log10(lo), math.log10(hi)
    vals = [10.0 ** (a + (b - a) * m / (M - 1)) for m in range(M)]
    return np.array(vals, dtype=np.float64).astype(np.float32)


def _f32(v) -> np.ndarray:
    return np.asarray(v, dtype=np.float64).astype(np.float32)


def _clip_round(x: np.ndarray, lo: int, hi: int) -> np.ndarray:
    """Round half-to-even to an integer length, then clip into [lo, hi]."""
    return np.clip(np.rint(x), lo, hi).astype(np.int32)


def _lognormal_by_mean(rng, mean: float, sigma: float, n: int) -> np.ndarray:
    mu = math.log(mean) - 0.5 * sigma * sigma
    return rng.lognormal(mu, sigma, n)


def _csr(parts) -> tuple[np.ndarray, np.ndarray]:
    offsets = np.zeros(len(parts) + 1, dtype=np.int64)
    offsets[1:] = np.cumsum([len(p) for p in parts])
    xi = np.concatenate(parts).astype(np.int32) if parts else np.zeros(0, np.int32)
    return offsets, xi


def _mean(x: np.ndarray) -> float:
    """Exact integer sum divided once (deterministic across machines)."""
    return int(x.astype(np.int64).sum()) / len(x)


# -------------------------------------------------------------- configs ----

def _lognormal_1x1k() -> Workload:
    rng = np.random.default_rng(0)
    L = 4096
    x = _clip_round(rng.lognormal(5.0, 1.0, 1000), 1, L)
    offsets, xi = _csr([x])
    return Workload("lognormal-1x1k", 1, offsets, None, xi, np.array([L], np.int32),
                    eta_grid(64, L), lam_grid(32), _f32([8.0]), _f32([1.0]),
                    1, _f32([10.0]),
                    meta=dict(desc="1 class x 1,000 lognormal(5,1) lengths, clip [1,4096]"))


def _lognormal_4x100k() -> Workload:
    rng = np.random.default_rng(1)
    L = 8192
    means, sig = (50.0, 300.0, 1500.0, 600.0), (0.8, 1.0, 1.2, 0.9)
    parts = [_clip_round(_lognormal_by_mean(rng, m, s, 100_000), 1, L) for m, s in zip(means, sig)]
    offsets, xi = _csr(parts)
    eps = _f32([0.05 * _mean(p) for p in parts])
    return Workload("lognormal-4x100k", 4, offsets, None, xi, np.full(4, L, np.int32),
                    eta_grid(512, L), lam_grid(128), _f32([4, 8, 16, 32]), _f32([1] * 4),
                    1, eps,
                    meta=dict(desc="4 classes x 1e5 lognormal lengths, clip [1,8192]"))


def _mixture_16x1M() -> Workload:
    rng = np.random.default_rng(2)
    L, C, N = 32768, 16, 1_000_000
    parts, cps = [], []
    for _ in range(C):
        m1, m2 = rng.uniform(20.0, 3000.0, 2)
        comp = rng.random(N) < 0.7
        a = _lognormal_by_mean(rng, m1, 1.0, N)
        b = _lognormal_by_mean(rng, m2, 1.0, N)
        x = np.where(comp, a, b)
        tail = rng.random(N) < 0.02
        xm = max(m1, m2)
        x = np.where(tail, xm * (1.0 + rng.pareto(1.5, N)), x)
        parts.append(_clip_round(x, 1, L))
        cps.append(math.exp(rng.uniform(math.log(2.0), math.log(64.0))))
    offsets, xi = _csr(parts)
    eps = _f32([0.02 * _mean(p) for p in parts])
    return Workload("mixture-16x1M", C, offsets, None, xi, np.full(C, L, np.int32),
                    eta_grid(2048, L), lam_grid(256), _f32(cps), _f32([1.0] * C),
                    1, eps,
                    meta=dict(desc="16 classes x 1e6: 0.7/0.3 lognormal mixture (means U[20,3000], "
                                   "sigma 1) + 2% Lomax(1.5) tail, clip [1,32768]"))


def _ratios_8x250k() -> Workload:
    """8 sample segments shared by 16 cost ratios: class c = ratio*8 + segment."""
    rng = np.random.default_rng(3)
    L, S, N, R, E = 32768, 8, 250_000, 16, 16
    means = [40.0 * 100.0 ** (s / 7.0) for s in range(S)]
    parts = [_clip_round(_lognormal_by_mean(rng, m, 1.0, N), 1, L) for m in means]
    offsets, xi = _csr(parts)
    C = R * S
    seg = np.array([c % S for c in range(C)], np.int32)
    rho = [128.0 ** (i / 15.0) for i in range(R)]
    c_w = _f32([0.5] * C)
    c_p = _f32([0.5 * rho[c // S] for c in range(C)])
    smean = [_mean(p) for p in parts]
    eps = np.empty(E * C, np.float32)
    for e in range(E):
        for c in range(C):
            eps[e * C + c] = np.float32(0.2 * smean[c % S] * e / 15.0)
    return Workload("ratios-8x250k", C, offsets, seg, xi, np.full(C, L, np.int32),
                    eta_grid(1024, L), lam_grid(128), c_p, c_w, E, eps,
                    meta=dict(desc="8 segments x 2.5e5 lognormal (means 40..4000), "
                                   "x 16 ratios in [1,128] x 16 radii in [0, 0.2 mean]",
                              rho=rho))


@functools.lru_cache(maxsize=1)
def _drift_base():
    rng = np.random.default_rng(4)
    C, N, G = 8, 4_000_000, 6
    means = [40.0 * 100.0 ** (c / 7.0) for c in range(C)]
    base = [_lognormal_by_mean(rng, m, 1.0, N) for m in means]
    cps = [math.exp(rng.uniform(math.log(2.0), math.log(64.0))) for _ in range(C)]
    cap = rng.uniform(20_000.0, 400_000.0, G)
    mask = rng.random((C, G)) < 0.5
    for c in range(C):
        if not mask[c].any():
            mask[c, rng.integers(G)] = True
    conc = np.where(mask, rng.uniform(0.5, 4.0, (C, G)), 0.0)
    return base, cps, cap, conc


def drift_base_draws() -> list:
    """The fixed per-class draws of drift-8x4M before rounding: iteration t
    holds clip(rint(draw * 1.01**t), 1, 32768) of each (fp64 throughout)."""
    return _drift_base()[0]


def _drift_8x4M(iteration: int = 0) -> Workload:
    base, cps, cap, conc = _drift_base()
    L, C = 32768, 8
    drift = 1.01 ** iteration
    parts = [_clip_round(b * drift, 1, L) for b in base]
    offsets, xi = _csr(parts)
    eps = _f32([0.02 * _mean(p) for p in parts])
    groups = Groups(_f32(cap), _f32(conc.reshape(-1)), float(np.float32(0.2)))
    return Workload("drift-8x4M", C, offsets, None, xi, np.full(C, L, np.int32),
                    eta_grid(2048, L), lam_grid(256), _f32(cps), _f32([1.0] * C),
                    1, eps, groups=groups,
                    meta=dict(desc="8 classes x 4e6 lognormal (means 40..4000) drifting 1%/iteration; "
                                   "6 groups, capacities U[20k,400k]", iteration=iteration))


def make_workload(name: str, **kw) -> Workload:
    if name == "lognormal-1x1k":
        return _lognormal_1x1k()
    if name == "lognormal-4x100k":
        return _lognormal_4x100k()
    if name == "mixture-16x1M":
        return _mixture_16x1M()
    if name == "ratios-8x250k":
        return _ratios_8x250k()
    if name == "drift-8x4M":
        return _drift_8x4M(kw.get("iteration", 0))
    if name == "random":
        return random_workload(**kw)
    raise ValueError(f"unknown workload {name!r}")


def random_workload(seed: int = 0, C: int = 3, N=(50, 7, 130), L: int = 300, K: int = 16,
                    M: int = 12, E: int = 2, lam_lo: float = 1e-3, lam_hi: float = 1e2,
                    cost_choices=None, alias: bool = False, with_groups: bool = False,
                    G: int = 2, dist: str = "lognormal") -> Workload:
    """Small ragged workload for parity and property tests.

    N may be an int or a per-segment tuple (ragged segments).  With `alias`,
    classes share segments (seg[c] = c % S with S = len(N)).
    """
    rng = np.random.default_rng(seed)
    Ns = [N] * C if isinstance(N, int) else list(N)
    S = len(Ns)
    parts = []
    for s, n in enumerate(Ns):
        if dist == "lognormal":
            mean = float(rng.uniform(0.05, 0.6) * L)
            x = _clip_round(_lognormal_by_mean(rng, mean, float(rng.uniform(0.3, 1.3)), n), 0, L)
        elif dist == "uniform":
            x = rng.integers(0, L + 1, n).astype(np.int32)
        elif dist == "constant":
            x = np.full(n, int(rng.integers(0, L + 1)), np.int32)
        else:
            raise ValueError(dist)
        parts.append(x)
    offsets, xi = _csr(parts)
    if alias:
        seg = np.array([c % S for c in range(C)], np.int32)
    else:
        if S != C:
            raise ValueError("without aliasing there must be one segment per class")
        seg = None
    if cost_choices is None:
        c_p = _f32(np.exp(rng.uniform(math.log(0.5), math.log(64.0), C)))
        c_w = _f32(np.exp(rng.uniform(math.log(0.25), math.log(4.0), C)))
    else:
        c_p = _f32([cost_choices[int(i)][0] for i in rng.integers(len(cost_choices), size=C)])
        c_w = _f32([cost_choices[int(i)][1] for i in rng.integers(len(cost_choices), size=C)])
    eps = _f32(rng.uniform(0.0, 0.2 * L, E * C))
    if E * C:
        eps[: min(C, E * C)] = 0.0     # one radius row at exactly zero
    groups = None
    if with_groups:
        conc = np.where(rng.random((C, G)) < 0.6, rng.uniform(0.5, 4.0, (C, G)), 0.0)
        for c in range(C):
            if not (conc[c] > 0).any():
                conc[c, rng.integers(G)] = float(rng.uniform(0.5, 4.0))
        cap = rng.uniform(0.3, 2.0, G) * L * C
        groups = Groups(_f32(cap), _f32(conc.reshape(-1)), float(np.float32(0.2)))
    return Workload(f"random{seed}", C, offsets, seg, xi, np.full(C, L, np.int32),
                    eta_grid(K, L), lam_grid(M, lam_lo, lam_hi), c_p, c_w, E, eps,
                    groups=groups, meta=dict(desc=f"random seed={seed}"))


# ------------------------------------------------- policy comparison ----
# Lognormal stand-ins fitted to the summary statistics the paper prints for
# its traces (Sec. 5.1): mean, P90 and P99 of the output length in tokens.
TRACE_STATS = {
    "burst": (125.0, 276.0, 1586.0),      # BurstGPT
    "sharegpt": (265.0, 486.0, 768.0),    # ShareGPT
}


def fit_lognormal(mean: float, p90: float, p99: float) -> tuple[float, float]:
    """(mu, sigma) of the lognormal with the given mean and P90.

    mean = exp(mu + sigma^2 / 2) and P90 = exp(mu + z90 sigma) leave a
    quadratic in sigma with two roots; the root whose P99 lies nearer the
    printed P99 is taken.
    """
    from statistics import NormalDist
    z90, z99 = NormalDist().inv_cdf(0.90), NormalDist().inv_cdf(0.99)
    c = math.log(p90 / mean)
    disc = z90 * z90 - 2.0 * c
    if disc < 0:
        raise ValueError("no lognormal has this mean and P90")
    roots = (z90 - math.sqrt(disc), z90 + math.sqrt(disc))

    def p99_err(s):
        return abs(math.log(mean) - 0.5 * s * s + z99 * s - math.log(p99))

    sigma = min(roots, key=p99_err)
    return math.log(mean) - 0.5 * sigma * sigma, sigma


def policy_workloads(trace: str = "burst", n_train: int = 1_000_000, n_eval: int = 1_000_000,
                     rhos=(2, 5, 10, 20, 50, 100), shifts=(1.0, 1.5, 2.0, 2.5, 3.0),
                     eps_fracs=(0.0, 0.05, 0.1, 0.15, 0.2, 0.3, 0.5), L: int = 8192,
                     K: Optional[int] = None, M: int = 256, seed: int = 5):
    """Training and evaluation sets for pricing reservation policies.

    Training: n_train draws of one trace stand-in, rounded half-to-even and
    clipped to [1, L], shared by one class per cost ratio rho (c_w = 1,
    c_p = rho) through the segment map; radii eps = RN32(frac * sample mean)
    for every frac in eps_fracs (row e of the radii).
    Evaluation: for every shift factor s, n_eval fresh draws of the same
    stand-in scaled by s before rounding and clipping (s is the ratio of the
    evaluation mean to the training mean); class s * len(rhos) + i is
    segment s priced at rho_i.  K defaults to every integer reservation
    0..L.  Returns (train, eval) Workloads.
    """
    mu, sigma = fit_lognormal(*TRACE_STATS[trace])
    rng = np.random.default_rng(seed)
    x_train = _clip_round(rng.lognormal(mu, sigma, n_train), 1, L)
    y_eval = rng.lognormal(mu, sigma, n_eval)
    nr = len(rhos)
    K = L + 1 if K is None else K
    eta, lam = eta_grid(K, L), lam_grid(M)
    mean = _mean(x_train)
    eps = _f32([f * mean for f in eps_fracs for _ in range(nr)])
    c_p, c_w = _f32(rhos), _f32([1.0] * nr)
    off, xi = _csr([x_train])
    desc = (f"{trace} stand-in lognormal(mu={mu:.4f}, sigma={sigma:.4f}), clip [1, {L}]: "
            f"{n_train} training samples, {nr} cost ratios, {len(eps_fracs)} radii")
    train = Workload(f"policy-{trace}-train", nr, off, np.zeros(nr, np.int32), xi,
                     np.full(nr, L, np.int32), eta, lam, c_p, c_w, len(eps_fracs), eps,
                     meta=dict(desc=desc, rhos=list(rhos), eps_fracs=list(eps_fracs)))
    parts = [_clip_round(s * y_eval, 1, L) for s in shifts]
    off_e, xi_e = _csr(parts)
    ce = nr * len(shifts)
    ev = Workload(f"policy-{trace}-eval", ce, off_e,
                  np.array([c // nr for c in range(ce)], np.int32), xi_e,
                  np.full(ce, L, np.int32), eta, lam, _f32([rhos[c % nr] for c in range(ce)]),
                  _f32([1.0] * ce), 1, np.zeros(ce, np.float32),
                  meta=dict(desc=f"{n_eval} fresh draws x shifts {list(shifts)}",
                            shifts=list(shifts), rhos=list(rhos)))
    return train, ev


# ------------------------------------------------------- serving model ----

@dataclass
class Service:
    """Serving-model inputs of Alg. 1 beyond the reservation data (Sec. 3.1-3.4).

    The paper prints the cost ratios and kappa but not the service-time or
    capacity constants; these are synthetic.
    """
    tau: np.ndarray      # int32 [G] tensor-parallel degree of configuration g
    pp: np.ndarray       # int32 [G] pipeline-parallel degree
    Mcap: np.ndarray     # float32 [G] KV capacity of one serving group, tokens
    Cc: np.ndarray       # float32 [G] prefill rate, tokens/s
    Bc: np.ndarray       # float32 [G] decode rate, tokens/s
    lam: np.ndarray      # float32 [C] arrival rate, requests/s
    Lin: np.ndarray      # int32 [C] input length, tokens
    Lpre: np.ndarray     # int32 [C] shared (cacheable) prefix, tokens
    D: np.ndarray        # float32 [C] latency SLO, s
    alpha: float         # prefill work per input token (float32 value)
    beta: float          # decode work per output token (float32 value)
    t_ar: float          # all-reduce latency, s (float32 value)
    NL: int              # layers
    c_gpu: float         # cost per GPU-second (float32 values below)
    c_slo: float         # cost per second of SLO excess
    c_rej: float         # cost per rejected request
    kappa: float         # memory-headroom factor
    u_max: float         # largest admissible memory utilisation of a group
    J: int               # GPU budget
    z0: np.ndarray       # int32 [G] initial configuration counts

    @property
    def G(self) -> int:
        return int(self.tau.shape[0])


def serving_workload(C: int = 15, N: int = 100_000, J: int = 48, L: int = 8192, K: int = 2048,
                     M: int = 256, seed: int = 6, configs=None):
    """Reservation data of C classes plus a synthetic serving model.

    Classes: lognormal output lengths (means log-spaced 20..600 tokens, sigma
    U[0.6, 1.3]), clip [1, L]; c_w = 1, c_p = 10 (rho = 10); eps = 0.15 x
    mean; arrival rates U[0.2, 2] requests/s; input 50..2000 tokens with a
    10-60 % shared prefix; SLO U[2, 20] s.  Configurations: every (TP, PP) in
    configs (default TP 1, 2, 4, 8 x PP 1, 2, 4) with KV capacity
    ~4000 tokens per GPU, prefill ~8000 tokens/s and decode ~40 tokens/s per
    request per unit of TP.  Cost weights in units of c_w: c_slo = 5,
    c_rej = 5000, c_gpu = 0.5; kappa = 0.2 (the paper's printed ratios).
    The start z0 adds one group of each configuration in turn while the
    budget allows.
    Returns (Workload, Service).
    """
    rng = np.random.default_rng(seed)
    means = [20.0 * (30.0 ** (c / max(C - 1, 1))) for c in range(C)]
    parts = [_clip_round(_lognormal_by_mean(rng, m, float(rng.uniform(0.6, 1.3)), N), 1, L)
             for m in means]
    offsets, xi = _csr(parts)
    eps = _f32([0.15 * _mean(p) for p in parts])
    w = Workload(f"serving-{C}x{N}", C, offsets, None, xi, np.full(C, L, np.int32),
                 eta_grid(K, L), lam_grid(M), _f32([10.0] * C), _f32([1.0] * C), 1, eps,
                 meta=dict(desc=f"{C} classes x {N} lognormal lengths (means 20..600), "
                                f"rho = 10, eps = 0.15 x mean"))
    if configs is None:
        configs = [(t, p) for t in (1, 2, 4, 8) for p in (1, 2, 4)]
    G = len(configs)
    tau = np.array([t for t, _ in configs], np.int32)
    pp = np.array([p for _, p in configs], np.int32)
    gpus = (tau * pp).astype(np.float64)
    Mcap = _f32(4000.0 * gpus * rng.uniform(0.8, 1.2, G))
    Cc = _f32(8000.0 * tau * rng.uniform(0.8, 1.0, G))
    Bc = _f32(40.0 * tau * rng.uniform(0.8, 1.0, G) / np.sqrt(pp))
    lam = _f32(rng.uniform(0.2, 2.0, C))
    Lin = rng.integers(50, 2000, C).astype(np.int32)
    Lpre = (Lin * rng.uniform(0.1, 0.6, C)).astype(np.int32)
    D = _f32(rng.uniform(2.0, 20.0, C))
    z0 = np.zeros(G, np.int32)          # round-robin: one group of each configuration
    used, grew = 0, True                 # in turn while the budget allows
    while grew:
        grew = False
        for g in range(G):
            if used + int(gpus[g]) <= J:
                z0[g] += 1
                used += int(gpus[g])
                grew = True
    svc = Service(tau, pp, Mcap, Cc, Bc, lam, Lin, Lpre, D,
                  alpha=float(np.float32(1.0)), beta=float(np.float32(1.0)),
                  t_ar=float(np.float32(2e-5)), NL=80, c_gpu=float(np.float32(0.5)),
                  c_slo=float(np.float32(5.0)), c_rej=float(np.float32(5000.0)),
                  kappa=float(np.float32(0.2)), u_max=float(np.float32(0.95)), J=J, z0=z0)
    return w, svc
