"""Reservation policies priced against each other (Sec. 5.1-5.4, Tables 2 and 5).

Forms every policy's reservation per training class from the library's
outputs, then prices it on held-out (optionally shifted) samples with
dro_reservation_cost:

  DRO(eps)   eta[k*] of dro_exact_table, one per radius row
  SAA        class_quantile at the class costs (Prop. 4.2, eps = 0)
  P90, P99   class_quantile at c_p : c_w = 9 : 1 and 99 : 1, i.e. the
             ceil(qN)-th smallest sample
  P95        class_quantile at 19 : 1, rounded up to a multiple of 16 tokens
             (the KV-cache block)
  Mean       the smallest integer >= the mean (class_moments)
  Max        L
  LP+k sigma the smallest integer >= mean + k * population standard
             deviation (class_moments), at most L, for k = 1, 2

Every reservation is computed by the library (the moment-based and
block-aligned ones by dro_baseline_reservations, exactly in integers); this
module only selects and stacks them.
"""
from __future__ import annotations

import dataclasses

import torch

from .api import (Context, Problem, class_moments, class_quantile, dro_baseline_reservations,
                  dro_exact_table, dro_reservation_cost)

BLOCK = 16
BASELINES = ("SAA", "P90", "P95", "P99", "Mean", "Max", "LP+1sigma", "LP+2sigma")


def policy_names(eps_fracs) -> list[str]:
    return [f"DRO(eps={f:g}*mean)" for f in eps_fracs] + list(BASELINES)


def _quantile_at(ctx: Context, prob: Problem, cp: float, cw: float) -> torch.Tensor:
    dev = prob.device
    p = dataclasses.replace(prob, c_p=torch.full((prob.C,), cp, dtype=torch.float32, device=dev),
                            c_w=torch.full((prob.C,), cw, dtype=torch.float32, device=dev))
    return class_quantile(ctx, p)["q_value"]


def reservations(ctx: Context, train: Problem, eps: torch.Tensor) -> torch.Tensor:
    """[R, C] int32 device tensor of every policy's reservation per class."""
    ex = dro_exact_table(ctx, train, eps)
    rows = [train.eta[ex["k_star"][e].long()] for e in range(ex["k_star"].shape[0])]
    rows.append(class_quantile(ctx, train)["q_value"])
    rows.append(_quantile_at(ctx, train, 9.0, 1.0))
    p95 = _quantile_at(ctx, train, 19.0, 1.0)
    b = dro_baseline_reservations(ctx, class_moments(ctx, train), train.L, k_sigma=(1, 2), q=p95,
                                  block=BLOCK)
    rows.append(b["block"])
    rows.append(_quantile_at(ctx, train, 99.0, 1.0))
    rows.append(b["mean"])
    rows.append(train.L)
    rows.append(b["lp"][0])
    rows.append(b["lp"][1])
    return torch.stack([r.to(torch.int32) for r in rows])


def price(ctx: Context, evalp: Problem, eta_train: torch.Tensor) -> dict:
    """Cost and cover of [R, C] training-class reservations on every shifted
    set: evaluation class s * C + i is shift s priced as training class i.
    Returns cost [R, S, C] (float64) and cover [R, S, C] (int64)."""
    R, C = eta_train.shape
    S = evalp.C // C
    if S * C != evalp.C:
        raise ValueError("the evaluation classes must be shifts x training classes")
    out = dro_reservation_cost(ctx, evalp, eta_train.repeat(1, S).contiguous())
    return dict(cost=out["cost"].view(R, S, C), cover=out["cover"].view(R, S, C))


def table(ctx: Context, train: Problem, evalp: Problem, eps: torch.Tensor, eps_fracs) -> dict:
    """Every policy's reservation, its in-sample cost and cover, and its cost
    and cover on each shifted evaluation set."""
    eta = reservations(ctx, train, eps)
    ins = dro_reservation_cost(ctx, train, eta)
    out = price(ctx, evalp, eta)
    return dict(names=policy_names(eps_fracs), eta=eta, cost=out["cost"], cover=out["cover"],
                cost_train=ins["cost"], cover_train=ins["cover"])
