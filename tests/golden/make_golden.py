"""Write the stored oracle results of the benchmark workloads.

    python tests/golden/make_golden.py lognormal-1x1k lognormal-4x100k mixture-16x1M \
        ratios-8x250k [drift-8x4M:ITERS] [policy-burst] [serving-15x100k]

Calls only `oracle/` (exact 128-bit evaluation, value-grouped) and the seeded
generator in `workloads/`.  Each file records the generator checksum of its
inputs, so a test can tell a changed input from a wrong result.  Doubles are
stored as hex strings (bit-exact).
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from workloads import make_workload  # noqa: E402


def _hex(a):
    return [[float(v).hex() for v in row] for row in np.asarray(a, np.float64)]


def golden_static(name: str) -> dict:
    w = make_workload(name)
    t0 = time.time()
    r = oracle.solve(w, grouped=True)
    out = dict(workload=name, checksum=w.checksum(), oracle_seconds=round(time.time() - t0, 1),
               oracle_threads=oracle.threads(),
               k_star=r["k_star"].tolist(), W_star=_hex(r["W_star"]),
               m_at_star=r["m_at_star"].tolist(), q_value=r["q_value"].tolist(),
               q_rank=r["q_rank"].tolist(),
               # a few full W rows (e = 0) for the table tolerance check
               W_rows={str(c): [float(v).hex() for v in r["W"][0, c]] for c in range(min(w.C, 4))})
    return out


def golden_bcd(iters: int) -> dict:
    rows = []
    k_prev = None
    for it in range(iters):
        w = make_workload("drift-8x4M", iteration=it)
        t0 = time.time()
        S = oracle.S_exact(w, grouped=True)
        W, _ = oracle.W_table(w, S)
        if k_prev is None:
            k_prev = oracle.bcd_init(w)
            k0 = k_prev.tolist()
        o = oracle.bcd_step(w, W[0], k_prev)
        qv, qr = oracle.quantile(w)
        rows.append(dict(iteration=it, checksum=w.checksum(), k_prev=k_prev.tolist(),
                         k_next=o["k_next"].tolist(), W_star=[float(v).hex() for v in o["W_star"]],
                         usage=[float(v).hex() for v in o["usage"]],
                         feasible=o["feasible"].tolist(), q_value=qv.tolist(),
                         seconds=round(time.time() - t0, 1)))
        print(f"drift-8x4M iteration {it}: {rows[-1]['seconds']} s", flush=True)
        k_prev = o["k_next"]
    return dict(workload="drift-8x4M", iterations=iters, k0=k0, rows=rows)


def golden_policy() -> dict:
    from oracle import policies
    from workloads import policy_workloads
    params = dict(trace="burst", n_train=1_000_000, n_eval=1_000_000,
                  rhos=[2, 5, 10, 20, 50, 100], shifts=[1.0, 1.5, 2.0, 2.5, 3.0],
                  eps_fracs=[0.0, 0.05, 0.1, 0.15, 0.2, 0.3, 0.5], L=8192, M=256, seed=5)
    tr, ev = policy_workloads(**params)
    t0 = time.time()
    t = policies.table(tr, ev, params["eps_fracs"])
    return dict(workload="policy-burst", params=params, checksum_train=tr.checksum(),
                checksum_eval=ev.checksum(), oracle_seconds=round(time.time() - t0, 1),
                names=t["names"], eta=t["eta"].tolist(), cover=t["cover"].tolist(),
                cover_train=t["cover_train"].tolist(),
                cost=[[[float(v).hex() for v in r] for r in rs] for rs in t["cost"]],
                cost_train=[[float(v).hex() for v in r] for r in t["cost_train"]])


def golden_serving() -> dict:
    from oracle import serving
    from workloads.configs import serving_workload
    params = dict(C=15, N=100_000, J=48, seed=6)
    w, svc = serving_workload(**params)
    t0 = time.time()
    r = serving.solve(w, svc)
    return dict(workload=w.name, params=params, checksum=w.checksum(),
                oracle_seconds=round(time.time() - t0, 1), z=r["z"].tolist(), k=r["k"].tolist(),
                delta=r["delta"].tolist(), pi=[[float(v).hex() for v in row] for row in r["pi"]],
                objective=float(r["objective"]).hex(), outer=r["outer"], inner=r["inner"])


def main(argv):
    for arg in argv:
        if arg == "serving-15x100k":
            data = golden_serving()
            path = os.path.join(HERE, "serving-15x100k.json")
        elif arg == "policy-burst":
            data = golden_policy()
            path = os.path.join(HERE, "policy-burst.json")
        elif arg.startswith("drift-8x4M"):
            iters = int(arg.split(":")[1]) if ":" in arg else 50
            data = golden_bcd(iters)
            path = os.path.join(HERE, "drift-8x4M_bcd.json")
        else:
            data = golden_static(arg)
            path = os.path.join(HERE, f"{arg}.json")
        with open(path, "w") as f:
            json.dump(data, f, indent=1)
        print(f"wrote {path}", flush=True)


if __name__ == "__main__":
    main(sys.argv[1:])
