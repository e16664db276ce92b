#!/usr/bin/env python3
"""Throughput of the DRO reservation path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload mixture-16x1M]

One step is one pass of the whole hot path over the resident samples of the
workload: the critical-fractile quantile of every class (class_quantile),
the dense worst-case sums and the minimum over the multiplier grid
(dro_cost_eval), and the exact lowest-index optimum (dro_argmin_reservation).
The default workload is 16 classes x 1e6 heavy-tailed synthetic lengths,
K = 2048 reservation levels, M = 256 multipliers.  The fused block step is
timed separately on the drifting 8-class x 4e6 workload (6 serving groups).

Prints ONE JSON line.  `value` is evaluations per second of the whole step
(one evaluation = one (class, reservation, multiplier, sample) term).
`roofline` prices the dense kernel's algorithmic fp32 work (7 operations per
evaluation: two multiply-adds, a 3-way max, an accumulate) against the fp32
vector peak; `cpu_baseline` times the CPU oracle's dense fp64 evaluation on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP32_PEAK_TFLOPS = 157.3          # MI355X fp32 vector: 256 CU x 64 lanes x 2 (FMA) x 2 (packed) x 2.4 GHz
FLOPS_PER_EVAL = 7                # 2 FMA (4) + 3-way max (2) + accumulate (1)
METRIC = "DRO cost evals/sec (class×r×λ×sample per s) + % fp32 VALU peak"
VALU_ISSUE_PEAK = 256 * 128 * 2.4e9   # lane-instructions/s of double-rate fp32 add/fma on MI355X

# Hardware-counter figures of the dense kernel on the 16 x 1e6 workload, from
# profiles/dense_kernel_mixture-16x1M_counters.md.  They describe one version of the
# dense kernel's code and launch plan (csrc/dense.hip, the constants of
# csrc/dro_internal.h and plan_dense of csrc/api.hip, comments and layout
# stripped, identified by the hash prefix) and are
# reported as null for any other code or workload.
DENSE_COUNTERS = {
    "dense_code_sha256_16": "82911c48cda0bfd3",
    "workload": "mixture-16x1M",
    "valu_instr_per_eval": 2.0597,       # SQ_INSTS_VALU x 64 / evaluations
    "hbm_bytes_per_launch": 1638297.24 * 1024,  # FETCH_SIZE x 2.000 + WRITE_SIZE x 1.000 (copy-calibrated)
    "source": "profiles/dense_kernel_mixture-16x1M_counters.md",
}


def dense_code_hash() -> str:
    """Hash of the dense kernel's code, of its constants (the dense section of
    csrc/dro_internal.h) and of its launch plan (the plan_dense function of
    csrc/api.hip, which sets the number of sample slices and so the
    partial-sum traffic), comments and whitespace removed."""
    import hashlib
    import re
    def code(name):
        with open(os.path.join(ROOT, "paper_2607_16892_amd", "csrc", name)) as f:
            text = re.sub(r"/\*.*?\*/", " ", f.read(), flags=re.S)
        return re.sub(r"//[^\n]*", " ", text)

    hdr = code("dro_internal.h")
    i = hdr.index("struct DensePlan")  # the dense section's constants come before its structs
    consts = [ln for ln in hdr[:i].splitlines() if "constexpr" in ln]
    api = code("api.hip")
    i = api.index("constexpr long long kMinWaves")
    plan = api[i:api.index("return pl;", i)]
    text = code("dense.hip") + "\n" + "\n".join(consts) + "\n" + plan
    return hashlib.sha256(" ".join(text.split()).encode()).hexdigest()[:16]


def _counters_for(workload: str):
    try:
        h = dense_code_hash()
    except OSError:
        return None
    if h != DENSE_COUNTERS["dense_code_sha256_16"] or workload != DENSE_COUNTERS["workload"]:
        return None
    return DENSE_COUNTERS


def _log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_baseline(w, n_samples: int):
    """Oracle dense fp64 on the first n samples of class 0, every grid point and multiplier."""
    import numpy as np
    import oracle
    from workloads.configs import Workload
    xs = w.samples_of(0)[:n_samples].copy()
    sub = Workload("sample", 1, np.array([0, len(xs)], np.int64), None, xs, w.L[:1].copy(), w.eta,
                   w.lam, w.c_p[:1].copy(), w.c_w[:1].copy(), 1, w.eps[:1].copy())
    t = time.perf_counter()
    oracle.S_f64(sub)
    dt = time.perf_counter() - t
    return dict(value=sub.evals / dt, unit="evals/s", cores=oracle.threads(), kind="oracle",
                sample=f"class 0 of {w.name}, first {len(xs)} samples x K={w.K} x M={w.M} "
                       f"({sub.evals:.3g} evaluations, dense fp64, {dt:.1f} s)")


def bench_bcd(ctx, dev, iters: int):
    """Fused block step on the drifting workload: the median ms per iteration
    (inputs resident; each iteration's drifted samples are generated and
    uploaded outside the timed region), the fastest and the total.  The
    workload's full run is 50 iterations (--bcd-iters 50)."""
    import torch
    import numpy as np
    import paper_2607_16892_amd as dro
    from workloads import make_workload
    w = make_workload("drift-8x4M", iteration=0)
    prob = dro.Problem.from_workload(w, dev)
    grp = dro.Groups.from_numpy(w.groups.cap, w.groups.conc, w.groups.kappa, dev)
    k = dro.bcd_init_state(ctx, prob)
    times = []
    binding = 0
    for it in range(iters):
        if it:
            w = make_workload("drift-8x4M", iteration=it)
            prob.replace_samples(w.offsets, w.xi)
        eps = torch.from_numpy(w.eps.copy()).to(dev)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        o = dro.bcd_block_step(ctx, prob, eps, grp, k)
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
        if (it + 1) % 10 == 0:
            _log(f"block step iteration {it + 1}/{iters}: {times[-1]:.1f} ms")
        k = o["k_next"]
        usage = o["usage"].cpu().numpy()
        binding = int((usage > 0.98 * w.groups.cap).sum())
    flags = ctx.take_flags()
    ms = float(np.median(times)) if times else None
    return dict(workload="drift-8x4M: 8 classes x 4e6 drifting lognormal, K=2048, M=256, G=6",
                iters=iters, ms_per_iter=ms, ms_min=float(np.min(times)) if times else None,
                ms_total=float(np.sum(times)), evals_per_iter=w.evals,
                evals_per_s=(w.evals / (ms / 1e3)) if ms else None,
                binding_groups_last_iter=binding, flags=flags)


def bench_policy(ctx, dev):
    """Reservation policies priced on held-out and shifted samples (the
    synthetic analogue of Tables 2 and 5, Fig. 2b and Fig. 3b)."""
    import numpy as np
    import torch
    import paper_2607_16892_amd as dro
    from paper_2607_16892_amd import policies
    from workloads import policy_workloads
    fr = [0.0, 0.05, 0.1, 0.15, 0.2, 0.3, 0.5]
    tr, ev = policy_workloads(eps_fracs=fr)
    train = dro.Problem.from_workload(tr, dev)
    evalp = dro.Problem.from_workload(ev, dev)
    eps = torch.from_numpy(tr.eps).to(dev)
    policies.table(ctx, train, evalp, eps, fr)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    t = policies.table(ctx, train, evalp, eps, fr)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3
    names = t["names"]
    cost = t["cost"].cpu().numpy()                 # [R, shifts, rhos]
    cov_tr = t["cover_train"].cpu().numpy()
    rhos, shifts = tr.meta["rhos"], ev.meta["shifts"]
    i = {n: names.index(n) for n in names}
    dro_i = i["DRO(eps=0.15*mean)"]
    n_tr = tr.n_of(0)

    def r3(a):
        return [float(f"{v:.4g}") for v in a]

    return {
        "workload": tr.meta["desc"] + f"; evaluation: {ev.meta['desc']}",
        "ms_table": ms,
        "rhos": rhos, "shifts": shifts,
        "reservation": {n: t["eta"][i[n]].cpu().tolist() for n in names},
        "cost_no_shift": {n: r3(cost[i[n], 0]) for n in names},
        "dro_gain_vs_p90": r3(1.0 - cost[dro_i, 0] / cost[i["P90"], 0]),
        "dro_gain_vs_p95": r3(1.0 - cost[dro_i, 0] / cost[i["P95"], 0]),
        "dro_level_vs_qstar": {"level": r3(cov_tr[dro_i] / n_tr),
                               "q_star": r3([r / (r + 1.0) for r in rhos])},
        "saa_over_dro_by_shift": {str(s): r3(cost[i["SAA"], j] / cost[dro_i, j])
                                  for j, s in enumerate(shifts)},
        "dro_by_radius_at_largest_shift": {n: r3(cost[i[n], -1]) for n in names
                                           if n.startswith("DRO")},
        "note": "DRO at eps = 0.15 x mean (the paper's default); costs are the average "
                "c_p (x - r)^+ + c_w (r - x)^+ over 1e6 held-out draws per shift, c_w = 1, "
                "c_p = rho",
    }


def bench_serving(ctx, dev):
    """The rest of Alg. 1 (routing LP, prefix caching, configuration search)
    on 15 classes x 1e5 samples, 12 (TP, PP) configurations, 48 GPUs."""
    import numpy as np
    import torch
    import paper_2607_16892_amd as dro
    from paper_2607_16892_amd import serving as gs
    from workloads.configs import serving_workload
    w, svc = serving_workload()
    prob = dro.Problem.from_workload(w, dev)
    s = gs.Service.from_model(svc, dev)
    eps = torch.from_numpy(w.eps[: w.C].copy()).to(dev)
    gs.dro_bcd_solve(ctx, prob, eps, s, svc.z0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    r = gs.dro_bcd_solve(ctx, prob, eps, s, svc.z0)
    torch.cuda.synchronize()
    solve_ms = (time.perf_counter() - t0) * 1e3
    # the configuration search alone at the final state
    tt = gs.bcd_service_times(ctx, prob, s)
    k = r["k"].long()
    ex = dro.dro_exact_table(ctx, prob, eps)
    Wc = ex["W"][0].gather(1, k[:, None])[:, 0].contiguous()
    eta_c = prob.eta[k].contiguous()
    times = []
    for _ in range(6):
        z = r["z"].clone()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        cs = gs.bcd_config_search(ctx, w.C, s, Wc, tt["T"], tt["ET2"], r["pi"], eta_c, r["delta"], z)
        b.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b))
    search_ms = float(np.median(times[1:]))
    # |Z| = number of z >= 0 with sum_g z_g tau_g pp_g <= J (counted on the host)
    gpus = [int(t) * int(p) for t, p in zip(svc.tau, svc.pp)]
    ways = [1] * (svc.J + 1)
    for gp in reversed(gpus):
        ways = [sum(ways[b - u * gp] for u in range(b // gp + 1)) for b in range(svc.J + 1)]
    nz = ways[svc.J]
    return dict(workload=f"{w.name}: {w.meta['desc']}; {svc.G} (TP, PP) configurations, "
                         f"J = {svc.J} GPUs",
                solve_ms=solve_ms, info=r["info"], z=r["z"].cpu().tolist(),
                objective=float(r["objective"].cpu()[0]),
                config_search_ms=search_ms, configurations=nz,
                configurations_per_s=nz / (search_ms / 1e3),
                n_feasible=int(cs["n_feasible"].cpu()[0]))


def bench_alg1_scaling(ctx, dev):
    """Solve time of the whole Alg. 1 loop over the problem sizes of Table 3
    (classes x configurations x samples), synthetic serving model."""
    import torch
    import paper_2607_16892_amd as dro
    from paper_2607_16892_amd import serving as gs
    from workloads.configs import serving_workload
    sizes = [(3, 4, 100, 8), (4, 4, 150, 8), (5, 5, 200, 8), (6, 6, 300, 8), (8, 6, 500, 8),
             (10, 8, 1000, 48), (15, 12, 2000, 48)]
    every = [(t, p) for t in (1, 2, 4, 8) for p in (1, 2, 4)]
    rows = []
    for C, G, N, J in sizes:
        w, svc = serving_workload(C=C, N=N, J=J, K=2048, M=256, seed=20 + C, configs=every[:G])
        prob = dro.Problem.from_workload(w, dev)
        s = gs.Service.from_model(svc, dev)
        eps = torch.from_numpy(w.eps[: w.C].copy()).to(dev)
        gs.dro_bcd_solve(ctx, prob, eps, s, svc.z0)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        r = gs.dro_bcd_solve(ctx, prob, eps, s, svc.z0)
        torch.cuda.synchronize()
        rows.append({"classes": C, "configurations": G, "samples": N, "gpus": J,
                     "solve_ms": (time.perf_counter() - t0) * 1e3, "outer": r["info"]["outer"],
                     "inner": r["info"]["inner"], "status": r["info"]["status"]})
    return rows


def _platform(dev) -> dict:
    import torch
    p = torch.cuda.get_device_properties(dev)
    return {"device": p.name, "arch": getattr(p, "gcnArchName", None),
            "compute_units": p.multi_processor_count, "hip": torch.version.hip,
            "torch": torch.__version__}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mixture-16x1M")
    ap.add_argument("--cpu-samples", type=int, default=81920)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--bcd-iters", type=int, default=3)
    ap.add_argument("--no-policy", action="store_true",
                    help="skip the reservation-policy comparison")
    ap.add_argument("--no-serving", action="store_true",
                    help="skip the routing / caching / configuration loop")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (scale reference for HBM byte counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(the work shards over classes with no exchange). Use --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2607_16892_amd as dro
    from workloads import make_workload

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    _log(f"generating {args.workload}")
    w = make_workload(args.workload)
    ctx = dro.Context(0)
    prob = dro.Problem.from_workload(w, dev)
    eps = torch.from_numpy(w.eps.copy()).to(dev)
    dro.dro_validate(ctx, prob, eps)
    E = w.E
    S = torch.empty((w.C, w.K, w.M), dtype=torch.float64, device=dev)
    W = torch.empty((E, w.C, w.K), dtype=torch.float64, device=dev)
    m_star = torch.empty((E, w.C, w.K), dtype=torch.int32, device=dev)
    outs = {}

    def step(ev=None):
        if ev:
            ev[0].record()
        dro.class_quantile(ctx, prob)
        if ev:
            ev[1].record()
        dro.dro_cost_eval(ctx, prob, eps, W=W, m_star=m_star, S=S)
        if ev:
            ev[2].record()
        outs.update(dro.dro_argmin_reservation(ctx, prob, eps, S))
        if ev:
            ev[3].record()

    _log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    pairs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(4))
             for _ in range(args.steps)]
    _log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(pairs[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    flags = ctx.take_flags()
    ms_step = (t1 - t0) * 1e3 / max(args.steps, 1)
    launch_times = [e[1].elapsed_time(e[2]) for e in pairs]
    dense_ms = float(np.mean(launch_times))
    breakdown = {"quantile_ms": float(np.median([e[0].elapsed_time(e[1]) for e in pairs])),
                 "cost_eval_ms": float(np.median(launch_times)),
                 "argmin_ms": float(np.median([e[2].elapsed_time(e[3]) for e in pairs])),
                 "note": "HIP events on the launch stream around class_quantile, dro_cost_eval "
                         "and dro_argmin_reservation; medians over the timed steps"}
    evals = w.evals
    value = evals / (ms_step / 1e3)
    achieved = evals * FLOPS_PER_EVAL / (dense_ms / 1e3) / 1e12
    _log(f"step {ms_step:.2f} ms, dense {dense_ms:.2f} ms, {value:.3e} evals/s, flags={flags}")
    cnt = _counters_for(w.name)

    # Exact table from value counts (not the per-term metric; reported beside it)
    torch.cuda.synchronize()
    dro.dro_exact_table(ctx, prob, eps)
    torch.cuda.synchronize()
    xt = []
    for _ in range(max(args.steps, 1)):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        ex = dro.dro_exact_table(ctx, prob, eps)
        b.record()
        torch.cuda.synchronize()
        xt.append(a.elapsed_time(b))
    exact_ms = float(np.median(xt))
    same_k = bool(torch.equal(ex["k_star"], outs["k_star"]))
    same_w = bool(torch.equal(ex["W_star"], outs["W_star"]))
    _log(f"exact table {exact_ms:.3f} ms (same optimum as the dense path: {same_k and same_w})")
    # Continuous-multiplier dual (the paper's min over gamma >= 0, no grid)
    cd = dro.dro_continuous_dual(ctx, prob, eps)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    cd = dro.dro_continuous_dual(ctx, prob, eps)
    b.record()
    torch.cuda.synchronize()
    cont_ms = a.elapsed_time(b)
    gap = ((ex["W"] - cd["W"]) / ex["W"]).cpu().numpy()
    cont = {"ms": cont_ms, "grid_gap_max": float(gap.max()), "grid_gap_median": float(np.median(gap)),
            "grid_gap_at_optimum_max": float(((ex["W_star"] - cd["W"].amin(dim=2)) / ex["W_star"]).max()),
            "note": "dro_continuous_dual: min over continuous gamma >= 0; grid_gap = "
                    "(W_grid - W_continuous) / W_grid over every (c, k)"}
    _log(f"continuous dual {cont_ms:.3f} ms, grid gap max {cont['grid_gap_max']:.2e}")

    if args.calibrate_copy:
        src = torch.ones(1 << 28, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        _log("copy calibration: 1 GiB read + 1 GiB written")
        del src, dst

    bcd = None
    if args.bcd_iters > 0:
        _log(f"block step, {args.bcd_iters} iterations")
        bcd = bench_bcd(ctx, dev, args.bcd_iters)
    srv = None
    if not args.no_serving:
        _log("serving loop (routing LP, prefix caching, configuration search)")
        srv = bench_serving(ctx, dev)
        srv["scaling"] = bench_alg1_scaling(ctx, dev)
    pol = None
    if not args.no_policy:
        _log("policy comparison")
        pol = bench_policy(ctx, dev)
    cpu = None
    if not args.no_cpu_baseline:
        _log("cpu baseline (oracle)")
        cpu = cpu_baseline(w, args.cpu_samples)

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "evals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.meta.get('desc', '')}", "C": w.C, "N_per_class": w.n_of(0),
                   "K": w.K, "M": w.M, "E": E, "evals_per_step": evals},
        "pct_fp32_valu_peak": 100.0 * achieved / FP32_PEAK_TFLOPS,
        "roofline": {"bound": "alu", "kernel": "dense_kernel (dro_cost_eval)",
                     "achieved": achieved, "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / FP32_PEAK_TFLOPS,
                     "traffic": cnt["hbm_bytes_per_launch"] if cnt else None,
                     "algorithmic_bytes": 4 * int(w.offsets[-1]) + 8 * w.C * w.K * w.M,
                     "traffic_note": "algorithmic bytes = the int32 samples read once plus the fp64 "
                                     "S table written once; the samples are read once, and the launch "
                                     "writes S as P sample-slice partials (P = 24 on mixture-16x1M, "
                                     "so that the grid runs 32 short waves of blocks) that a "
                                     "deterministic reduce sums: 1.6 GB at about 7 GB/s, which the "
                                     "VALU-bound kernel does not feel",
                     "launch_ms": dense_ms, "launch_ms_median": float(np.median(launch_times)),
                     "launch_ms_min": float(np.min(launch_times)), "flops_per_eval": FLOPS_PER_EVAL,
                     "evals_per_launch": evals,
                     "note": "frac counts the paper-form 7 fp32 ops per evaluation; the kernel's "
                             "exact two-line form issues valu_instr_per_eval instructions, so "
                             "valu_issue_frac is the hardware utilisation",
                     "valu_instr_per_eval": cnt["valu_instr_per_eval"] if cnt else None,
                     "valu_issue_frac": (evals * cnt["valu_instr_per_eval"] / (dense_ms / 1e3)
                                         / VALU_ISSUE_PEAK) if cnt else None,
                     "counters": cnt["source"] if cnt else None},
        "step_breakdown": breakdown,
        "cpu_baseline": cpu,
        "block_step": bcd,
        "policy_comparison": pol,
        "serving_loop": srv,
        "continuous_dual": cont,
        "exact_table": {"ms": exact_ms, "same_optimum_as_dense_path": same_k and same_w,
                        "note": "dro_exact_table: the same W table from value counts and prefix "
                                "sums in 128-bit integers; it does not evaluate per-sample terms, "
                                "so it is reported beside the metric, not as it",
                        "equivalent_evals_per_s": evals / (exact_ms / 1e3)},
        "flags": flags,
        "platform": _platform(dev),
    }
    print(json.dumps(line), flush=True)
    ctx.close()


if __name__ == "__main__":
    main()
