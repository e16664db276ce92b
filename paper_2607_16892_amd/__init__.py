"""MI355X (gfx950) Wasserstein-DRO KV-cache reservation path.

The compute path is the HIP library libdro.so (C ABI in include/dro.h); this
package is its thin Python binding, with the entry points under the same
names.  Import fails loudly at first use if the library is not built.
"""
from .api import (Context, Problem, Groups, DroError, dro_validate, dro_cost_eval,
                  dro_cost_eval_noalloc,
                  dro_argmin_reservation, dro_exact_table, dro_continuous_dual, class_quantile,
                  class_moments, dro_reservation_cost, dro_baseline_reservations, bcd_init_state,
                  bcd_block_step)
from ._native import LIB_PATH, NativeMissing, load as load_native

__all__ = ["Context", "Problem", "Groups", "DroError", "dro_validate", "dro_cost_eval",
           "dro_cost_eval_noalloc",
           "dro_argmin_reservation", "dro_exact_table", "dro_continuous_dual", "class_quantile",
           "class_moments", "dro_reservation_cost", "dro_baseline_reservations", "bcd_init_state",
           "bcd_block_step",
           "LIB_PATH", "NativeMissing",
           "load_native"]
