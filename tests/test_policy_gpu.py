"""The reservation-policy comparison on the GPU against the oracle's (exact).

Every policy's reservation, in-sample cost and cover, and cost and cover on
each shifted evaluation set are compared bit for bit: the reservations are
integers and every cost is the fully specified RN(RN(S) / N) of an exact sum.
"""
import json
import os

import numpy as np
import pytest

from workloads import policy_workloads

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def ctx(dev):
    import paper_2607_16892_amd as dro
    c = dro.Context(dev.index or 0)
    yield c
    c.close()


def gpu_table(ctx, dev, tr, ev, eps_fracs):
    import torch
    import paper_2607_16892_amd as dro
    from paper_2607_16892_amd import policies
    print(f"[gpu] policy table {tr.name} N={tr.offsets[-1]} K={tr.K} M={tr.M} E={tr.E}; "
          f"{ev.name} C={ev.C} N={ev.offsets[-1]}", flush=True)
    train = dro.Problem.from_workload(tr, dev)
    evalp = dro.Problem.from_workload(ev, dev)
    eps = torch.from_numpy(tr.eps).to(dev)
    dro.dro_validate(ctx, train, eps)
    dro.dro_validate(ctx, evalp)
    t = policies.table(ctx, train, evalp, eps, eps_fracs)
    torch.cuda.synchronize()
    return {k: (v.cpu().numpy() if hasattr(v, "cpu") else v) for k, v in t.items()}


def _same(g, ref):
    assert g["names"] == ref["names"]
    for k in ("eta", "cover", "cover_train"):
        assert np.array_equal(np.asarray(g[k]), np.asarray(ref[k])), k
    for k in ("cost", "cost_train"):
        assert np.array_equal(np.asarray(g[k]).view(np.uint64),
                              np.asarray(ref[k], np.float64).view(np.uint64)), k


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_small_table_matches_oracle(ctx, dev, seed):
    from oracle import policies as opol
    fr = (0.0, 0.05, 0.15, 0.5)
    tr, ev = policy_workloads(n_train=5000 + 1000 * seed, n_eval=3000, rhos=(2, 5, 10, 100),
                              shifts=(1.0, 1.7, 3.0), eps_fracs=fr, L=2000, K=1001, M=64,
                              seed=40 + seed)
    _same(gpu_table(ctx, dev, tr, ev, fr), opol.table(tr, ev, fr))


def test_full_table_against_stored_oracle(ctx, dev):
    path = os.path.join(HERE, "golden", "policy-burst.json")
    gold = json.load(open(path))
    tr, ev = policy_workloads(**gold["params"])
    assert tr.checksum() == gold["checksum_train"] and ev.checksum() == gold["checksum_eval"]
    g = gpu_table(ctx, dev, tr, ev, gold["params"]["eps_fracs"])
    ref = dict(names=gold["names"], eta=gold["eta"], cover=gold["cover"],
               cover_train=gold["cover_train"],
               cost=np.array([[[float.fromhex(v) for v in r] for r in rs] for rs in gold["cost"]]),
               cost_train=np.array([[float.fromhex(v) for v in r] for r in gold["cost_train"]]))
    _same(g, ref)


@pytest.mark.parametrize("dist", ["lognormal", "constant"])
def test_baseline_reservations_against_oracle(ctx, dev, dist):
    """dro_baseline_reservations (mean, mean + k sigma for k = 0, 1, 2, 3, 8, and
    a block-aligned quantile) against the oracle's rational definitions, on
    ragged classes: one sample, all-equal samples, the largest support."""
    import math
    from fractions import Fraction

    import torch
    import oracle.policies as op
    import paper_2607_16892_amd as dro
    from workloads import random_workload
    w = random_workload(seed=78, C=5, N=(1, 40, 2000, 777, 5000), L=32768, K=9, M=4, E=1,
                        dist=dist)
    print(f"[gpu] baseline reservations {w.name} dist={dist} N={w.offsets[-1]}", flush=True)
    prob = dro.Problem.from_workload(w, dev)
    ks = (0, 1, 2, 3, 8)
    q = dro.class_quantile(ctx, prob)["q_value"]
    b = dro.dro_baseline_reservations(ctx, dro.class_moments(ctx, prob), prob.L, k_sigma=ks, q=q,
                                      block=16)
    torch.cuda.synchronize()
    qh = q.cpu().numpy()
    for c in range(w.C):
        xs = w.samples_of(c)
        L = int(w.L[c])
        assert int(b["mean"][c]) == math.ceil(Fraction(int(xs.astype(np.int64).sum()), len(xs)))
        for i, k in enumerate(ks):
            assert int(b["lp"][i, c]) == op._mean_plus(xs, k, L), (c, k)
        assert int(b["block"][c]) == -(-int(qh[c]) // 16) * 16
