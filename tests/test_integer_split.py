"""The integer split that the dense kernel relies on, checked on the CPU.

In units of 2^-33 the three candidates of phi (App. A, Step 4) are the larger
of two lines whose difference is De x - Nu.  With t = floor(Nu / De) and
r = Nu - De t, for every integer sample x (case c_w <= c_p)

    phi = B - A1 x + De relu(x - t) - r [x > t],

and the mirror image around t = ceil(Nu / De) when c_w > c_p; summed over a
class, sum relu(x - t) = (sum x - N t + sum |x - t|) / 2 with t clamped to
the range a 16-bit sample code can meet.  This test evaluates that split with
Python integers (per-sample |x - t|, then the clamps and counts exactly as
stated) and compares every sum with the oracle's exact S, bit for bit, on
ragged and aliased classes and at cost ratios from 2^-17 to 2^17.
"""
import numpy as np
import pytest

import oracle
from workloads import eta_grid, lam_grid, random_workload
from workloads.configs import Workload


def _fix33(v) -> int:
    return int(np.float64(np.float32(v)) * 2 ** 33)


def _split_sums(w):
    out = {}
    for c in range(w.C):
        xs = w.samples_of(c).astype(np.int64)
        N, sx = len(xs), int(xs.sum())
        cnt = np.bincount(xs, minlength=32769).cumsum()

        def count_le(v):
            return 0 if v < 0 else (N if v >= 32768 else int(cnt[v]))

        CP, CW, L = _fix33(w.c_p[c]), _fix33(w.c_w[c]), int(w.L[c])
        upper = np.float32(w.c_w[c]) <= np.float32(w.c_p[c])
        for k in range(w.K):
            eta = int(w.eta[k])
            for m in range(w.M):
                G = _fix33(w.lam[m])
                B, Cc = CW * eta, CP * (L - eta)
                A1, A2 = min(G, CW), min(G, CP)
                De, Nu = A1 + A2, B - Cc + A2 * L
                if upper:
                    t = Nu // De
                    tc = min(max(t, -1), L)
                    sad = int(np.abs(xs - tc).sum())
                    Rt = (sx - N * tc + sad) // 2 + N * max(tc - t, 0)
                    S = N * B - A1 * sx + De * Rt - (Nu - De * t) * (N - count_le(t))
                else:
                    t = -((-Nu) // De)
                    tc = min(max(t, 0), L + 1)
                    sad = int(np.abs(xs - tc).sum())
                    Rt = (N * tc - sx + sad) // 2 + N * max(t - tc, 0)
                    S = N * (Cc - A2 * L) + A2 * sx + De * Rt - (De * t - Nu) * count_le(t - 1)
                out[(c, k, m)] = S
    return out


def _check(w):
    ref = oracle.S_exact(w, grouped=True)
    for (c, k, m), v in _split_sums(w).items():
        assert v == ref.as_int((c, k, m)), (w.name, c, k, m)


@pytest.mark.parametrize("case", [
    dict(seed=1, C=2, N=(300, 41), L=500, K=17, M=9, E=1),
    dict(seed=2, C=4, N=(1, 2, 3, 100), L=500, K=20, M=10, E=1),                 # N = 1
    dict(seed=3, C=5, N=(60, 9), alias=True, L=200, K=25, M=11, E=1),            # aliased
    dict(seed=4, C=2, N=(300, 57), L=32768, K=33, M=13, E=1),                    # largest support
    dict(seed=5, C=3, N=(40, 40, 40), dist="constant", L=100, K=21, M=9, E=1),   # all equal
    dict(seed=8, C=5, N=(204, 105, 409, 77, 31), L=4096, K=33, M=20, E=1,
         cost_choices=[(4.0, 1.0), (8.0, 1.0), (2.0, 2.0), (1.0, 8.0), (0.5, 64.0)]),
], ids=lambda c: f"seed{c['seed']}")
def test_integer_split_equals_the_exact_sums(case):
    _check(random_workload(**case))


@pytest.mark.parametrize("cp,cw", [(2.0 ** 7, 2.0 ** -3), (2.0 ** 7, 2.0 ** -10),
                                   (2.0 ** -10, 2.0 ** 7), (1.0, 1.0)])
def test_integer_split_at_extreme_cost_ratios(cp, cw):
    L, K, M = 32768, 65, 24
    xs = np.random.default_rng(7).integers(0, L + 1, 400).astype(np.int32)
    w = Workload(f"ratio{cp / cw:g}", 1, np.array([0, xs.size], np.int64), None, xs,
                 np.array([L], np.int32), eta_grid(K, L), lam_grid(M), np.array([cp], np.float32),
                 np.array([cw], np.float32), 1, np.array([10.0], np.float32))
    _check(w)
