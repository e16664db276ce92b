"""Seeded synthetic workloads for the DRO reservation path.

This module is shared by the product path and the oracle: it draws the
sample sets, the grids, the radii and the cost coefficients, and holds none
of the method's arithmetic (no cost, no dual, no quantile, no argmin).
"""
from .configs import (Workload, Groups, make_workload, random_workload, policy_workloads,
                      fit_lognormal, TRACE_STATS, CONFIG_NAMES, eta_grid, lam_grid)

__all__ = ["Workload", "Groups", "make_workload", "random_workload", "policy_workloads",
           "fit_lognormal", "TRACE_STATS", "CONFIG_NAMES", "eta_grid", "lam_grid"]
