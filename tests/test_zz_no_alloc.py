"""dro_cost_eval_noalloc (the entry point that allocates nothing) against dro_cost_eval.

Both compute the exact sums S, the table W and m_star, so every output must be
bit-identical.  Two calls in a row share the library's static scratch array;
the second has fewer segments, grid points and samples than the first, so
stale contents of the array from the first call would show.
"""
import numpy as np
import pytest

from workloads import make_workload, random_workload

pytestmark = pytest.mark.gpu


def _both(ctx, w, dev):
    import torch
    import paper_2607_16892_amd as dro
    print(f"[gpu] no-alloc {w.name} C={w.C} S={w.offsets.size - 1} K={w.K} M={w.M} E={w.E}",
          flush=True)
    prob = dro.Problem.from_workload(w, dev)
    eps = torch.from_numpy(w.eps.copy()).to(dev)
    ref = dro.dro_cost_eval(ctx, prob, eps)
    S = torch.full((w.C, w.K, w.M), float("nan"), dtype=torch.float64, device=dev)
    W = torch.full((w.E, w.C, w.K), float("nan"), dtype=torch.float64, device=dev)
    m = torch.full((w.E, w.C, w.K), -1, dtype=torch.int32, device=dev)
    got = dro.dro_cost_eval_noalloc(ctx, prob, eps, S, W, m)
    torch.cuda.synchronize()
    for key in ("S", "W", "m_star"):
        a, b = got[key].cpu().numpy(), ref[key].cpu().numpy()
        assert a.tobytes() == b.tobytes(), f"{w.name}: {key} differs from dro_cost_eval"


def test_noalloc_matches_dro_cost_eval_two_calls(dev):
    import paper_2607_16892_amd as dro
    with dro.Context(dev.index or 0) as ctx:
        _both(ctx, make_workload("lognormal-4x100k"), dev)
        # smaller: fewer samples, grid points and multipliers, aliased segments, 3 radii
        _both(ctx, random_workload(seed=3, C=5, N=(60, 9), alias=True, L=200, K=25, M=11, E=3),
              dev)


def test_noalloc_rejects_problems_beyond_its_array(dev):
    import torch
    import paper_2607_16892_amd as dro
    # 80 segments need about 42 MB of scratch, more than the 32 MiB array
    w = random_workload(seed=5, C=80, N=5, L=100, K=8, M=4, E=1)
    with dro.Context(dev.index or 0) as ctx:
        prob = dro.Problem.from_workload(w, dev)
        eps = torch.from_numpy(w.eps.copy()).to(dev)
        S = torch.full((w.C, w.K, w.M), 7.0, dtype=torch.float64, device=dev)
        W = torch.full((w.E, w.C, w.K), 7.0, dtype=torch.float64, device=dev)
        with pytest.raises(dro.DroError) as ei:
            dro.dro_cost_eval_noalloc(ctx, prob, eps, S, W)
        assert "no-allocation array" in str(ei.value)
        torch.cuda.synchronize()
        assert bool((S == 7.0).all()) and bool((W == 7.0).all()), "outputs were written"
