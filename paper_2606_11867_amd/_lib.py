"""ctypes declarations of libforemoe.so (the C ABI in include/foremoe.h)."""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libforemoe.so")

OK = 0
EINVAL = -1
EUNSUPPORTED = -2
EHIP = -3
F32 = 0
BF16 = 1
WS_INVALID_IDS = 0
WS_DROPPED = 1
WS_PLAN_ERRORS = 2
MAX_EXPERTS = 1024
MAX_SLOTS = 1024
MAX_REPLICAS = 16
MAX_TOPK = 64
MAX_SOURCES = 64
MAX_WGRAD_STEPS = 16
STATIC_SCRATCH_BYTES = 8 << 20
XFER_PARAMS = 1
XFER_GRADS = 2
XFER_ASSIGN = 0
XFER_ADD = 1
MAX_XFER_RECORDS = 64

c_i32, c_i64, c_sz, c_p = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p


class Plan(ctypes.Structure):
    _fields_ = [
        ("E", c_i32), ("S", c_i32), ("R_max", c_i32), ("n_src", c_i32),
        ("slot_expert", c_p), ("slot_replica", c_p), ("expert_nrep", c_p),
        ("expert_rep_weight", c_p), ("slot_widx", c_p), ("slot_gidx", c_p),
        ("src_token_begin", c_p), ("src_rep_weight", c_p),
    ]


PPlan = ctypes.POINTER(Plan)


class Machine(ctypes.Structure):
    _fields_ = [("M", c_i32), ("R", c_i32), ("N_b", c_i32), ("N_r", c_i32)]


PMachine = ctypes.POINTER(Machine)


class WgradStep(ctypes.Structure):
    _fields_ = [("a", c_p), ("b", c_p), ("slot_offset", c_p), ("slot_gidx", c_p), ("S", c_i32), ("n_cap", c_i64)]


PWgradStep = ctypes.POINTER(WgradStep)

# name -> (restype, argtypes)
SIGNATURES = {
    "foremoe_workspace_size": (c_sz, [c_i64, c_i32, c_i32]),
    "foremoe_histogram": (ctypes.c_int, [c_p, c_i64, c_i32, c_i32, c_p, c_p, c_sz, c_p]),
    "foremoe_histogram_src": (ctypes.c_int, [c_p, c_i64, c_i32, c_i32, c_i32, c_p, c_p, c_p, c_sz, c_p]),
    "foremoe_assign_replicas": (ctypes.c_int, [c_p, PPlan, c_p, c_p, c_p, c_p, c_sz, c_p]),
    "foremoe_histogram_assign": (ctypes.c_int, [c_p, c_i64, c_i32, PPlan, c_p, c_p, c_p, c_p, c_p, c_sz, c_p]),
    "foremoe_permute": (ctypes.c_int, [c_p, c_i32, c_i64, c_i32, c_p, c_i32, PPlan, c_p, c_p, c_i64,
                                       c_p, c_p, c_p, c_p, c_sz, c_p]),
    "foremoe_dispatch_static": (ctypes.c_int, [c_p, c_i64, c_i32, PPlan, c_p, c_i32, c_i32, c_i64, c_p, c_p,
                                               c_p, c_p, c_p, c_p, c_p, c_p, c_p]),
    "foremoe_ffn_workspace_size": (c_sz, []),
    "foremoe_grouped_ffn_fwd": (ctypes.c_int, [c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_i32, c_p, c_p,
                                               c_i64, c_p, c_p, c_p, c_p, c_sz, c_p]),
    "foremoe_ffn_gate_up_fwd": (ctypes.c_int, [c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_i32, c_p, c_i64,
                                               c_p, c_p, c_p, c_sz, c_p]),
    "foremoe_ffn_down_fwd": (ctypes.c_int, [c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_i32, c_p, c_i64,
                                            c_p, c_p, c_sz, c_p]),
    "foremoe_grouped_ffn_dgrad": (ctypes.c_int, [c_p, c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_i32, c_p,
                                                 c_p, c_i64, c_p, c_p, c_p, c_sz, c_p]),
    "foremoe_ffn_down_dgrad": (ctypes.c_int, [c_p, c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_i32, c_p,
                                              c_i64, c_p, c_p, c_sz, c_p]),
    "foremoe_ffn_gate_up_dgrad": (ctypes.c_int, [c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_i32, c_p,
                                                 c_i64, c_p, c_p, c_sz, c_p]),
    "foremoe_wgrad_workspace_size": (c_sz, [c_i32, c_i32]),
    "foremoe_grouped_ffn_wgrad": (ctypes.c_int, [c_p, c_p, c_p, c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p,
                                                 c_i32, c_i64, c_p, c_p, c_p, c_sz, c_p]),
    "foremoe_ffn_gate_up_wgrad": (ctypes.c_int, [c_p, c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_i32,
                                                 c_i64, c_p, c_p, c_sz, c_p]),
    "foremoe_ffn_down_wgrad": (ctypes.c_int, [c_p, c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_i32,
                                              c_i64, c_p, c_p, c_sz, c_p]),
    "foremoe_ffn_gate_up_wgrad_steps": (ctypes.c_int, [PWgradStep, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32,
                                                       c_p, c_p, c_sz, c_p]),
    "foremoe_ffn_down_wgrad_steps": (ctypes.c_int, [PWgradStep, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32,
                                                    c_p, c_p, c_sz, c_p]),
    "foremoe_combine": (ctypes.c_int, [c_p, c_i32, c_p, c_p, c_i64, c_i32, c_i32, c_i64, c_p, c_i32, c_p]),
    "foremoe_combine_bwd": (ctypes.c_int, [c_p, c_p, c_i32, c_p, c_p, c_i64, c_i32, c_i32, c_i64, c_p, c_p,
                                           c_p]),
    "foremoe_permute_bwd": (ctypes.c_int, [c_p, c_i32, c_p, c_i64, c_i32, c_i32, c_i64, c_p, c_i32, c_p]),
    "foremoe_xfer_record_bytes": (c_sz, [c_i32, c_i32, c_i32, c_i32]),
    "foremoe_copy_out": (ctypes.c_int, [c_p, c_p, c_i32, c_i32, c_p, c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p,
                                        c_i32, c_p, c_sz, c_p]),
    "foremoe_copy_in": (ctypes.c_int, [c_p, c_sz, c_i32, c_p, c_p, c_p, c_i32, c_p, c_p, c_i32, c_i32, c_p, c_p,
                                       c_i32, c_i32, c_i32, c_p]),
    "foremoe_plan_prefetch": (ctypes.c_int, [c_p, c_i32, c_p, c_i32, c_p, c_p, c_p, c_p]),
    "foremoe_prefetch_experts": (ctypes.c_int, [c_p, c_p, c_i32, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_p, c_p,
                                                c_i32, c_p]),
    "foremoe_plan_base": (ctypes.c_int, [c_p, c_i32, PMachine, c_i64, c_i64, c_p]),
    "foremoe_plan_micro_step": (ctypes.c_int, [c_p, c_i32, PMachine, c_p, c_i32, c_p, c_p, c_p]),
    "foremoe_plan_rank_slots": (ctypes.c_int, [c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_p, c_p, c_p, c_p, c_p]),
    "foremoe_ffn_gate_up_fwd_timed": (ctypes.c_int, [c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_i32, c_p,
                                                     c_i64, c_p, c_p, c_p, c_sz, c_p, c_p, c_p]),
    "foremoe_ffn_down_fwd_timed": (ctypes.c_int, [c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_i32, c_p, c_i64,
                                                  c_p, c_p, c_sz, c_p, c_p, c_p]),
    "foremoe_ffn_down_dgrad_timed": (ctypes.c_int, [c_p, c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_i32, c_p,
                                                    c_i64, c_p, c_p, c_sz, c_p, c_p, c_p]),
    "foremoe_ffn_gate_up_dgrad_timed": (ctypes.c_int, [c_p, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_i32, c_p,
                                                       c_i64, c_p, c_p, c_sz, c_p, c_p, c_p]),
    "foremoe_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "foremoe_last_error": (ctypes.c_char_p, []),
    "foremoe_version": (ctypes.c_char_p, []),
}

_lib = None


def load() -> ctypes.CDLL:
    """Load libforemoe.so from the package directory; raise if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is not built; run `python -m paper_2606_11867_amd.build` "
                "(the expert layer has no fallback path)")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


class ForeMoEError(RuntimeError):
    def __init__(self, status: int, where: str):
        lib = load()
        msg = lib.foremoe_last_error().decode(errors="replace")
        super().__init__(f"{where}: {lib.foremoe_status_string(status).decode()} ({status}): {msg}")
        self.status = status


def check(status: int, where: str) -> None:
    if status != OK:
        raise ForeMoEError(status, where)
