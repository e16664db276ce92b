"""Two contexts working at once on two streams of one device.

Each context owns its workspace and flag word, and every compute call only
enqueues on the stream it is given, so two contexts on two streams must give
the same bits as one context on the default stream, call for call.
"""
import numpy as np
import pytest

from workloads import make_workload, random_workload

pytestmark = pytest.mark.gpu


def _calls(ctx, w, dev, stream):
    import torch
    import paper_2607_16892_amd as dro
    with torch.cuda.stream(stream):
        prob = dro.Problem.from_workload(w, dev)
        eps = torch.from_numpy(w.eps).to(dev)
        r = dro.dro_cost_eval(ctx, prob, eps, stream=stream)
        a = dro.dro_argmin_reservation(ctx, prob, eps, r["S"], stream=stream)
        q = dro.class_quantile(ctx, prob, stream=stream)
        x = dro.dro_exact_table(ctx, prob, eps, stream=stream)
        m = dro.class_moments(ctx, prob, stream=stream)
    return {**{k: v for k, v in r.items() if v is not None},
            **{k: v for k, v in a.items() if v is not None},
            **q, **{"x_" + k: v for k, v in x.items()}, **{"mo_" + k: v for k, v in m.items()}}


def test_two_contexts_on_two_streams(dev):
    import torch
    import paper_2607_16892_amd as dro
    w1 = make_workload("lognormal-4x100k")
    w2 = random_workload(seed=8, C=3, N=(2049, 1025, 4097), L=4096, K=513, M=70, E=1,
                         cost_choices=[(4.0, 1.0), (8.0, 1.0), (2.0, 2.0)])
    print(f"[gpu] streams: {w1.name} and {w2.name}", flush=True)
    ref_ctx = dro.Context(dev.index or 0)
    default = torch.cuda.current_stream(dev)
    ref = [_calls(ref_ctx, w, dev, default) for w in (w1, w2)]
    torch.cuda.synchronize()
    ref = [{k: v.cpu().numpy() for k, v in d.items()} for d in ref]
    ref_ctx.close()

    c1, c2 = dro.Context(dev.index or 0), dro.Context(dev.index or 0)
    s1, s2 = torch.cuda.Stream(dev), torch.cuda.Stream(dev)
    torch.cuda.synchronize()
    for rep in range(2):   # the second round reuses the grown workspaces
        g1 = _calls(c1, w1, dev, s1)
        g2 = _calls(c2, w2, dev, s2)
        torch.cuda.synchronize()
        for g, r, name in ((g1, ref[0], w1.name), (g2, ref[1], w2.name)):
            assert set(g) == set(r)
            for k in r:
                assert g[k].cpu().numpy().tobytes() == r[k].tobytes(), (name, rep, k)
    c1.close()
    c2.close()


def test_alg1_on_a_side_stream_beside_other_work(dev):
    """dro_bcd_solve synchronises only its own stream: a second context's
    work queued on another stream runs beside it, and both match their
    default-stream results bit for bit."""
    import torch
    import paper_2607_16892_amd as dro
    from paper_2607_16892_amd import serving as gs
    from workloads.configs import serving_workload
    configs = [(1, 1), (2, 1), (4, 1), (2, 2), (4, 2)]
    w, svc = serving_workload(C=5, N=3000, J=16, K=257, M=32, configs=configs, seed=7)
    w2 = make_workload("lognormal-4x100k")
    print(f"[gpu] streams: {w.name} solve beside {w2.name}", flush=True)

    def solve(ctx, stream):
        with torch.cuda.stream(stream):
            prob = dro.Problem.from_workload(w, dev)
            s = gs.Service.from_model(svc, dev)
            eps = torch.from_numpy(np.ascontiguousarray(w.eps[: w.C], np.float32)).to(dev)
            r = gs.dro_bcd_solve(ctx, prob, eps, s, svc.z0, stream=stream)
        return r

    ctx = dro.Context(dev.index or 0)
    default = torch.cuda.current_stream(dev)
    ref = solve(ctx, default)
    ref_other = _calls(ctx, w2, dev, default)
    torch.cuda.synchronize()
    ref = {k: (v.cpu().numpy() if torch.is_tensor(v) else v) for k, v in ref.items()}
    ref_other = {k: v.cpu().numpy() for k, v in ref_other.items()}
    ctx.close()

    c1, c2 = dro.Context(dev.index or 0), dro.Context(dev.index or 0)
    s1, s2 = torch.cuda.Stream(dev), torch.cuda.Stream(dev)
    torch.cuda.synchronize()
    other = _calls(c2, w2, dev, s2)        # queued, still running
    r = solve(c1, s1)
    torch.cuda.synchronize()
    for k in ("z", "k", "pi", "delta", "objective"):
        assert r[k].cpu().numpy().tobytes() == ref[k].tobytes(), k
    assert r["info"] == ref["info"]
    for k in ref_other:
        assert other[k].cpu().numpy().tobytes() == ref_other[k].tobytes(), k
    c1.close()
    c2.close()
