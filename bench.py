#!/usr/bin/env python3
"""Throughput of the DRO reservation path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload mixture-16x1M]

One step is one pass of the whole hot path over the resident samples of the
workload: the critical-fractile quantile of every class (class_quantile),
the dense worst-case sums and the minimum over the multiplier grid
(dro_cost_eval), and the exact lowest-index optimum (dro_argmin_reservation).
The default workload is 16 classes x 1e6 heavy-tailed synthetic lengths,
K = 2048 reservation levels, M = 256 multipliers.  The fused block step runs
all 50 iterations of the drifting 8-class x 4e6 workload (6 serving groups).

Prints ONE JSON line.  `value` is evaluations per second of the whole step
(one evaluation = one (class, reservation, multiplier, sample) term).

`roofline` prices the dense kernel against the issue rate of the instruction
it executes.  Each evaluation's per-sample part is |x - t| in 16-bit
integers, and one v_sad_u16 evaluates two of them; the VALU issues
single-rate integer instructions at 256 CU x 64 lanes x 2.4 GHz, so the
kernel cannot exceed 2 x 3.93e13 = 7.86e13 evaluations/s.  `frac` is the
achieved rate over that ceiling.  The paper's three-candidate form would take
7 fp32 operations per evaluation; that equivalent rate is reported
separately, labelled as such, and is not executed work.

`cpu_baseline` times the CPU oracle's dense fp64 evaluation on a bounded
sample of the same workload (a quarter of one class, about 40 s), and the exact value-grouped oracle
that validates parity on the whole workload.
"""
from __future__ import annotations

import argparse
import json
import os
import platform as _pf
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "DRO cost evals/sec (class×r×λ×sample per s) + % fp32 VALU peak"
CLOCK_HZ = 2.4e9
VALU_SINGLE_RATE = 256 * 64 * CLOCK_HZ   # lane-instructions/s of single-rate VALU on MI355X
EVALS_PER_SAD = 2                        # v_sad_u16: two 16-bit halves per lane-instruction
EVAL_PEAK = EVALS_PER_SAD * VALU_SINGLE_RATE
FP32_PEAK_TFLOPS = 157.3                 # MI355X fp32 vector (256 CU x 64 x 2 (FMA) x 2 (packed) x 2.4 GHz)
PAPER_FLOPS_PER_EVAL = 7                 # 2 multiply-adds (4), a 3-way max (2), an accumulate (1)

# Hardware-counter figures of the dense kernel on the 16 x 1e6 workload, from
# profiles/dense_kernel_mixture-16x1M_counters.md.  They describe one version
# of the dense kernel's code and launch plan (csrc/dense.hip, the constants of
# csrc/dro_internal.h and plan_dense of csrc/api.hip, comments and layout
# stripped, identified by the hash prefix) and are reported as null for any
# other code or workload.
DENSE_COUNTERS = {
    "dense_code_sha256_16": "2d58a6d03fe9d642",
    "workload": "mixture-16x1M",
    "valu_instr_per_eval": 0.50312,    # SQ_INSTS_VALU x 64 / evaluations
    "clock_ghz": 2.371,                # GRBM_GUI_ACTIVE / 8 XCDs / duration
    "hbm_bytes_per_launch": 222985011,  # FETCH_SIZE x 2.000 + WRITE_SIZE x 1.000 (copy-calibrated)
    "source": "profiles/dense_kernel_mixture-16x1M_counters.md",
}


def dense_code_hash() -> str:
    """Hash of the dense kernel's code (the part of csrc/dense.hip before the
    fill, epilogue and minimum kernels), of its constants (the dense section of
    csrc/dro_internal.h) and of its launch plan (the plan constants and the
    plan_dense function of csrc/api.hip, which set the slices and the grid),
    comments and whitespace removed."""
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
    plan_consts = [ln for ln in api.splitlines()
                   if any(f"constexpr long long {k} " in ln for k in ("kDirectSampleTiles", "kSlicesPerBlock",
                                                                      "kMaxSliceN", "kBalanceSliceN",
                                                                      "kMinSliceN", "kMaxDirectSlices"))]
    i = api.index("DensePlan plan_dense(")
    plan = api[i:api.index("return pl;", i)]
    dense = code("dense.hip")
    dense = dense[:dense.index("zero_u64_u32_kernel")]  # the dense kernel, its helpers and launch
    text = dense + "\n" + "\n".join(consts + plan_consts) + "\n" + plan
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


def host_info() -> dict:
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = os.cpu_count()
    return {"cpu_model": model or _pf.processor() or None, "logical_cpus": os.cpu_count(),
            "usable_cpus": usable}


def cpu_baseline(w, n_samples: int, grouped: bool):
    """The oracle's dense fp64 evaluation on the first n samples of class 0 at
    every grid point and multiplier (a bounded sample of the workload), and,
    with `grouped`, the wall time of the exact value-grouped oracle on the
    whole workload."""
    import numpy as np
    import oracle
    from workloads.configs import Workload
    xs = w.samples_of(0)[:n_samples].copy()
    sub = Workload("sample", 1, np.array([0, len(xs)], np.int64), None, xs, w.L[:1].copy(), w.eta,
                   w.lam, w.c_p[:1].copy(), w.c_w[:1].copy(), 1, w.eps[:1].copy())
    t = time.perf_counter()
    oracle.S_f64(sub)
    dt = time.perf_counter() - t
    out = dict(value=sub.evals / dt, unit="evals/s", cores=oracle.threads(), kind="oracle",
               sample=f"class 0 of {w.name}, first {len(xs)} of its {w.n_of(0)} samples x "
                      f"K={w.K} x M={w.M} ({sub.evals:.3g} evaluations, dense fp64, "
                      f"{dt:.1f} s; {sub.evals / (w.n_of(0) * w.K * w.M):.1%} of one class)",
               host=host_info())
    if grouped:
        t = time.perf_counter()
        oracle.solve(w, grouped=True)
        out["grouped_exact_oracle_s"] = time.perf_counter() - t
        out["grouped_exact_note"] = ("the exact value-grouped oracle (S, W, argmin, quantiles of "
                                     "the whole workload) that the parity tests compare with; it "
                                     "groups equal sample values, so it does different work")
    return out


def bench_bcd(ctx, dev, iters: int):
    """Fused block step on the drifting workload: every iteration's ms, the
    median, fastest and total.  Inputs stay resident: each iteration's drifted
    samples are formed on the device from the fixed fp64 draws (multiply by
    1.01^t, round half to even, clip) outside the timed region; iterations 0
    and iters-1 are checked bit for bit against the host generator."""
    import numpy as np
    import torch
    import paper_2607_16892_amd as dro
    from workloads import make_workload
    from workloads.configs import drift_base_draws
    w0 = make_workload("drift-8x4M", iteration=0)
    base = torch.from_numpy(np.concatenate(drift_base_draws())).to(dev)
    L = int(w0.L[0])

    def samples(t):
        return torch.clamp(torch.round(base * (1.01 ** t)), 1, L).to(torch.int32)

    sizes = [int(n) for n in np.diff(w0.offsets)]

    def eps_of(xi):  # 2 % of each class mean, the mean as the exact sum divided once
        sums = torch.stack([p.to(torch.int64).sum() for p in torch.split(xi, sizes)]).cpu()
        return np.asarray([0.02 * (int(s) / n) for s, n in zip(sums, sizes)],
                          np.float64).astype(np.float32)

    checked = []
    for t in sorted({0, iters - 1}):
        wt = w0 if t == 0 else make_workload("drift-8x4M", iteration=t)
        same = bool(np.array_equal(samples(t).cpu().numpy(), wt.xi)) and \
            bool(np.array_equal(eps_of(samples(t)), wt.eps))
        checked.append({"iteration": t, "identical_to_host_generator": same})
        if not same:
            raise RuntimeError(f"device-side drift samples differ from the host's at iteration {t}")
    prob = dro.Problem.from_workload(w0, dev)
    grp = dro.Groups.from_numpy(w0.groups.cap, w0.groups.conc, w0.groups.kappa, dev)
    k = dro.bcd_init_state(ctx, prob)
    times = []
    binding = 0
    for it in range(iters):
        xi = samples(it)
        prob.xi.copy_(xi)
        eps = torch.from_numpy(eps_of(xi)).to(dev)
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
        binding = int((usage > 0.98 * w0.groups.cap).sum())
    ms = float(np.median(times)) if times else None
    return dict(workload="drift-8x4M: 8 classes x 4e6 lognormal drifting 1%/iteration, K=2048, "
                         "M=256, G=6",
                iters=iters, ms_per_iter=ms, ms_min=float(np.min(times)) if times else None,
                ms_max=float(np.max(times)) if times else None,
                ms_total=float(np.sum(times)), evals_per_iter=w0.evals,
                evals_per_s=(w0.evals / (ms / 1e3)) if ms else None,
                binding_groups_last_iter=binding, k_final=k.cpu().tolist(),
                generator_check=checked)


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
    on 15 classes x 1e5 samples, 12 (TP, PP) configurations, 48 GPUs, with
    synthetic model constants (so no time here is comparable to the paper's
    solver times)."""
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
                         f"J = {svc.J} GPUs, synthetic model constants",
                solve_ms=solve_ms, info=r["info"], z=r["z"].cpu().tolist(),
                objective=float(r["objective"].cpu()[0]),
                config_search_ms=search_ms, configurations=nz,
                configurations_per_s=nz / (search_ms / 1e3),
                n_feasible=int(cs["n_feasible"].cpu()[0]))


def _platform(dev) -> dict:
    import torch
    p = torch.cuda.get_device_properties(dev)
    return {"device": p.name, "arch": getattr(p, "gcnArchName", None),
            "compute_units": p.multi_processor_count, "hip": torch.version.hip,
            "torch": torch.__version__, "host": host_info()}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mixture-16x1M")
    ap.add_argument("--cpu-samples", type=int, default=250_000,
                    help="samples of class 0 in the oracle's timed dense sample (a quarter of a "
                         "class of the default workload, about 40 s)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-grouped-oracle", action="store_true",
                    help="skip timing the exact value-grouped oracle on the whole workload")
    ap.add_argument("--bcd-iters", type=int, default=50)
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
    q_value = torch.empty(w.C, dtype=torch.int32, device=dev)
    q_rank = torch.empty(w.C, dtype=torch.int64, device=dev)
    outs = {}

    # every call goes to torch's current stream, where the events are recorded
    def step(ev=None):
        if ev:
            ev[0].record()
        dro.class_quantile(ctx, prob, q_value=q_value, q_rank=q_rank)
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
    ms_step = (t1 - t0) * 1e3 / max(args.steps, 1)
    launch_times = [e[1].elapsed_time(e[2]) for e in pairs]
    dense_ms = float(np.mean(launch_times))
    q_ms = float(np.median([e[0].elapsed_time(e[1]) for e in pairs]))
    q_bytes = 4 * int(w.offsets[-1])  # the int32 samples, each read once
    breakdown = {"quantile_ms": q_ms,
                 "quantile_sample_bytes": q_bytes,
                 "quantile_gbs": q_bytes / (q_ms * 1e-3) / 1e9,
                 "cost_eval_ms": float(np.median(launch_times)),
                 "argmin_ms": float(np.median([e[2].elapsed_time(e[3]) for e in pairs])),
                 "note": "HIP events on the launch stream around class_quantile, dro_cost_eval "
                         "and dro_argmin_reservation; medians over the timed steps; "
                         "quantile_gbs = the samples' bytes over the whole call's time "
                         "(both launches and the gaps between the events)"}
    evals = w.evals
    value = evals / (ms_step / 1e3)
    dense_rate = evals / (dense_ms / 1e3)
    _log(f"step {ms_step:.2f} ms, dense {dense_ms:.2f} ms, {value:.3e} evals/s")
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
    same_table = bool(torch.equal(ex["W"], W)) and bool(torch.equal(ex["m_star"], m_star))
    _log(f"exact table {exact_ms:.3f} ms (same table and optimum as the dense path: "
         f"{same_table and same_k and same_w})")
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
    pol = None
    if not args.no_policy:
        _log("policy comparison")
        pol = bench_policy(ctx, dev)
    cpu = None
    if not args.no_cpu_baseline:
        _log("cpu baseline (oracle)")
        cpu = cpu_baseline(w, args.cpu_samples, not args.no_grouped_oracle)

    algo_bytes = 4 * int(w.offsets[-1]) + 8 * w.C * w.K * w.M
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
        "dtype": "u16",
        "dtype_note": "each evaluation's per-sample part |x - t| in unsigned 16-bit halves, summed "
                      "in 32- and 64-bit integers; the epilogue in 128-bit integers; J in f64 "
                      "(every S, W and argmin exact)",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.meta.get('desc', '')}", "C": w.C,
                   "N_per_class": w.n_of(0), "K": w.K, "M": w.M, "E": E,
                   "evals_per_step": evals},
        "pct_valu_peak": 100.0 * dense_rate / EVAL_PEAK,
        "roofline": {"bound": "alu", "kernel": "dense_kernel (dro_cost_eval)",
                     "achieved": dense_rate / 1e12, "peak": EVAL_PEAK / 1e12, "unit": "Tevals/s",
                     "frac": dense_rate / EVAL_PEAK,
                     "peak_note": "one v_sad_u16 lane-instruction evaluates two terms, and the "
                                  "VALU issues 256 CU x 64 lanes x 2.4 GHz = 3.93e13 single-rate "
                                  "lane-instructions/s",
                     "traffic": cnt["hbm_bytes_per_launch"] if cnt else None,
                     "algorithmic_bytes": algo_bytes,
                     "traffic_note": "algorithmic bytes = the int32 samples read once plus the "
                                     "fp64 S table written once; traffic = copy-calibrated "
                                     "FETCH_SIZE + WRITE_SIZE of the committed counter profile: "
                                     "the samples are fetched about once, and a block adds a "
                                     "tile's exact sums to the table with one 64-bit atomic per "
                                     "pair each time it leaves that tile (about 2.3 times per "
                                     "pair), about 8 bytes of write traffic each",
                     "launch_ms": dense_ms, "launch_ms_median": float(np.median(launch_times)),
                     "launch_ms_min": float(np.min(launch_times)), "evals_per_launch": evals,
                     "launch_note": "HIP events around dro_cost_eval on its stream: the dense "
                                    "kernel plus the histogram, prefix, fill, exact epilogue and "
                                    "minimum over the multipliers (about 0.15 ms)",
                     "valu_instr_per_eval": cnt["valu_instr_per_eval"] if cnt else None,
                     "valu_issue_frac": (evals * cnt["valu_instr_per_eval"] / (dense_ms / 1e3)
                                         / VALU_SINGLE_RATE) if cnt else None,
                     "clock_ghz": cnt["clock_ghz"] if cnt else None,
                     "counters": cnt["source"] if cnt else None},
        "paper_form_equivalent": {
            "tflops": dense_rate * PAPER_FLOPS_PER_EVAL / 1e12,
            "fraction_of_fp32_peak": dense_rate * PAPER_FLOPS_PER_EVAL / 1e12 / FP32_PEAK_TFLOPS,
            "note": "the rate the paper's three-candidate form would need at 7 fp32 operations "
                    "per evaluation against the 157.3 TFLOP/s fp32 vector peak; not executed "
                    "work (the kernel runs an exact integer form), so it is not a roofline "
                    "fraction"},
        "step_breakdown": breakdown,
        "cpu_baseline": cpu,
        "block_step": bcd,
        "policy_comparison": pol,
        "serving_loop": srv,
        "continuous_dual": cont,
        "exact_table": {"ms": exact_ms,
                        "same_table_and_optimum_as_dense_path": same_table and same_k and same_w,
                        "note": "dro_exact_table: the same W table from value counts and prefix "
                                "sums in 128-bit integers; it does not evaluate per-sample terms, "
                                "so it is reported beside the metric, not as it",
                        "equivalent_evals_per_s": evals / (exact_ms / 1e3)},
        "platform": _platform(dev),
    }
    print(json.dumps(line), flush=True)
    ctx.close()


if __name__ == "__main__":
    main()
