"""ctypes declarations of the streambeam C ABI (include/streambeam.h).

Argument marshalling only: every step of the search runs in the HIP library.
Loading fails loudly when the library has not been built; there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
import re
import numpy as np
from ctypes import POINTER, c_char_p, c_double, c_int32, c_int64, c_size_t, c_uint16, c_void_p

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "_lib", "libstreambeam.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "streambeam.h")

# Workspace limit of sb_create_noalloc (SB_NOALLOC_SCRATCH_BYTES in the header).
SB_NOALLOC_SCRATCH_BYTES = 64 << 20

SB_OK, SB_E_INVALID_ARG, SB_E_WORKSPACE, SB_E_STATE, SB_E_QUEUE_FULL, SB_E_TRUNCATED, \
    SB_E_HIP, SB_E_UNSUPPORTED = range(8)
SB_FIXED, SB_VAR_BATCH, SB_VAR_STREAM, SB_VAR_FIFO, SB_FIXED_STREAM, SB_VAR_CAP = 0, 1, 2, 3, 4, 5
SB_RULE_PAPER, SB_RULE_FAIRSEQ = 0, 1
SB_F32, SB_BF16 = 0, 1
SCHEDULERS = {"fixed": SB_FIXED, "var_batch": SB_VAR_BATCH, "var_stream": SB_VAR_STREAM,
              "var_fifo": SB_VAR_FIFO, "fixed_stream": SB_FIXED_STREAM, "var_cap": SB_VAR_CAP}
# Scheduler names that also pick the Fairseq finalization rule.
FAIRSEQ_SCHEDULERS = {"fixed_fairseq": SB_FIXED, "fixed_fairseq_stream": SB_FIXED_STREAM}


class SbParams(ctypes.Structure):
    _fields_ = [("k", c_int32), ("n", c_int32), ("eps", c_double), ("delta", c_double),
                ("max_per_node", c_int32), ("sched", c_int32), ("max_len_cap", c_int32),
                ("max_inputs", c_int32), ("finalize_rule", c_int32), ("pool", c_int32)]


class SbModel(ctypes.Structure):
    _fields_ = [("vocab", c_int32), ("d", c_int32), ("dtype", c_int32), ("eos_beta", ctypes.c_float),
                ("W_h", c_void_p), ("E", c_void_p), ("W_out", c_void_p),
                ("kv_layers", c_int32), ("W_kv", c_void_p), ("attn", c_int32)]


class SbHyp(ctypes.Structure):
    _fields_ = [("input", c_int64), ("rank", c_int32), ("length", c_int32), ("status", c_int32),
                ("finalize_step", c_int32), ("score", c_double), ("tok_offset", c_int64)]


# The same record as a numpy structured type (collect results as arrays).
SB_HYP_DTYPE = np.dtype({"names": [f for f, _ in SbHyp._fields_],
                         "formats": [np.int64, np.int32, np.int32, np.int32, np.int32, np.float64, np.int64],
                         "offsets": [getattr(SbHyp, f).offset for f, _ in SbHyp._fields_],
                         "itemsize": ctypes.sizeof(SbHyp)})


class SbStats(ctypes.Structure):
    _fields_ = [("timesteps", c_int64), ("expansions", c_int64), ("noops", c_int64),
                ("refills", c_int64), ("admitted", c_int64), ("hyps", c_int64), ("finished", c_int64),
                ("positions", c_int64), ("tile_recomputes", c_int64)]


class StreambeamError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        self.status = status
        super().__init__(f"{where}: status {status}" + (f" ({detail})" if detail else ""))


_lib = None


def header_symbols():
    """Names of every function declared in include/streambeam.h."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(sb_[a-z_]+)\s*\(", text)))


def lib():
    """The loaded library (built in-tree by paper_2010_02164_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"streambeam HIP library not built: {LIB_PATH} is missing; run "
                          "`python -m paper_2010_02164_amd.build` (or __graft_entry__.build())")
    L = ctypes.CDLL(LIB_PATH)
    P = POINTER
    sig = {
        "sb_workspace_bytes": (c_size_t, [P(SbModel), P(SbParams)]),
        "sb_validate": (c_int32, [P(SbModel), P(SbParams)]),
        "sb_create": (c_int32, [P(SbModel), P(SbParams), c_void_p, c_size_t, c_void_p, P(c_void_p)]),
        "sb_create_noalloc": (c_int32, [P(SbModel), P(SbParams), c_void_p, P(c_void_p)]),
        "sb_submit": (c_int32, [c_void_p, c_int32, P(c_int64), c_void_p, P(c_int32), P(c_int32)]),
        "sb_step": (c_int32, [c_void_p, P(c_int32)]),
        "sb_run": (c_int32, [c_void_p]),
        "sb_collect": (c_int32, [c_void_p, P(SbHyp), c_int64, P(c_int32), c_int64, P(c_int64), P(c_int64)]),
        "sb_stats": (c_int32, [c_void_p, P(SbStats)]),
        "sb_reset": (c_int32, [c_void_p]),
        "sb_rows_histogram": (c_int32, [c_void_p, P(c_int64), P(c_int32)]),
        "sb_set_timing": (c_int32, [c_void_p, c_int32]),
        "sb_timing": (c_int32, [c_void_p, P(c_double), P(c_int64)]),
        "sb_debug_expand": (c_int32, [c_void_p, c_int32, c_void_p, P(c_int32), P(c_int32), P(c_int32),
                                      c_void_p, P(c_double), P(c_double), P(c_int32)]),
        "sb_debug_slot": (c_int32, [c_void_p, c_int32, c_int32, P(c_int32), P(c_double), P(c_int64),
                                    P(c_int32), P(c_int32), c_int32, P(c_int32), P(c_uint16), c_int64]),
        "sb_destroy": (c_int32, [c_void_p]),
        "sb_last_error": (c_char_p, [c_void_p]),
        "sb_status_string": (c_char_p, [c_int32]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L
