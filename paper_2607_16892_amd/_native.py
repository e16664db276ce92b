"""ctypes view of libdro.so (include/dro.h).  Argument marshalling only."""
from __future__ import annotations

import ctypes as ct
import os
import threading

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdro.so")

_lock = threading.Lock()
_lib = None

P = ct.c_void_p
i32 = ct.c_int32


class ProblemStruct(ct.Structure):
    _fields_ = [("C", i32), ("S", i32), ("offsets", P), ("offsets_h", P), ("seg", P), ("seg_h", P),
                ("xi", P), ("L", P), ("K", i32), ("eta", P), ("M", i32), ("lam", P), ("c_p", P),
                ("c_w", P)]


class GroupsStruct(ct.Structure):
    _fields_ = [("G", i32), ("cap", P), ("conc", P), ("kappa", ct.c_float)]


class ServiceStruct(ct.Structure):
    _fields_ = [("G", i32), ("tau", P), ("pp", P), ("tau_h", P), ("pp_h", P), ("Mcap", P),
                ("Cc", P), ("Bc", P), ("lam", P), ("Lin", P), ("Lpre", P), ("D", P),
                ("alpha", ct.c_float), ("beta", ct.c_float), ("t_ar", ct.c_float), ("NL", i32),
                ("c_gpu", ct.c_float), ("c_slo", ct.c_float), ("c_rej", ct.c_float),
                ("kappa", ct.c_float), ("u_max", ct.c_float), ("J", i32)]


class StepOutStruct(ct.Structure):
    _fields_ = [("k_next", P), ("W_star", P), ("q_value", P), ("usage", P), ("feasible", P)]


EXPORTS = {
    "dro_strerror": (ct.c_char_p, [ct.c_int]),
    "dro_create": (ct.c_int, [ct.c_int, ct.POINTER(P)]),
    "dro_destroy": (None, [P]),
    "dro_last_error": (ct.c_char_p, [P]),
    "dro_validate": (ct.c_int, [P, ct.POINTER(ProblemStruct), i32, P, P]),
    "dro_cost_eval": (ct.c_int, [P, ct.POINTER(ProblemStruct), i32, P, P, P, P, P]),
    "dro_cost_eval_noalloc": (ct.c_int, [P, ct.POINTER(ProblemStruct), i32, P, P, P, P, P]),
    "dro_argmin_reservation": (ct.c_int, [P, ct.POINTER(ProblemStruct), i32, P, P, P, P, P, P, P]),
    "class_quantile": (ct.c_int, [P, ct.POINTER(ProblemStruct), P, P, P]),
    "dro_exact_table": (ct.c_int, [P, ct.POINTER(ProblemStruct), i32, P, P, P, P, P, P, P, P]),
    "dro_continuous_dual": (ct.c_int, [P, ct.POINTER(ProblemStruct), i32, P, P, P, P]),
    "class_moments": (ct.c_int, [P, ct.POINTER(ProblemStruct), P, P, P, P, P]),
    "dro_reservation_cost": (ct.c_int, [P, ct.POINTER(ProblemStruct), i32, P, P, P, P]),
    "dro_baseline_reservations": (ct.c_int, [P, i32, P, P, P, P, i32, P, P, i32, P, P, P, P]),
    "bcd_init_state": (ct.c_int, [P, ct.POINTER(ProblemStruct), P, P]),
    "bcd_service_times": (ct.c_int, [P, ct.POINTER(ProblemStruct), ct.POINTER(ServiceStruct), P, P,
                                     P]),
    "bcd_queue_state": (ct.c_int, [P, i32, ct.POINTER(ServiceStruct), P, P, P, P, P, P, P, P, P,
                                   P, P]),
    "bcd_routing_lp": (ct.c_int, [P, i32, ct.POINTER(ServiceStruct), P, P, P, P, P, P, P, P, P,
                                  P]),
    "bcd_reservation_sweep": (ct.c_int, [P, i32, i32, P, P, i32, P, P, ct.c_float, P, P, P, P]),
    "bcd_prefix_cache": (ct.c_int, [P, i32, i32, P, P, P]),
    "bcd_config_search": (ct.c_int, [P, i32, ct.POINTER(ServiceStruct), P, P, P, P, P, P, P, P, P,
                                     P, P]),
    "dro_bcd_solve": (ct.c_int, [P, ct.POINTER(ProblemStruct), P, ct.POINTER(ServiceStruct), i32,
                                 i32, P, P, P, P, P, P, P]),
    "bcd_block_step": (ct.c_int, [P, ct.POINTER(ProblemStruct), P, ct.POINTER(GroupsStruct), P,
                                  ct.POINTER(StepOutStruct), P]),
}


class NativeMissing(RuntimeError):
    pass


def load():
    """The loaded library; raises NativeMissing if libdro.so was not built."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise NativeMissing(
                    f"{LIB_PATH} is missing: build it with `python -m paper_2607_16892_amd.build` "
                    "(the reservation path has no fallback)")
            lib = ct.CDLL(LIB_PATH)
            for name, (res, args) in EXPORTS.items():
                fn = getattr(lib, name)
                fn.restype = res
                fn.argtypes = args
            _lib = lib
    return _lib
