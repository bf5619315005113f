"""ctypes loader of liblaep_moe.so and the C signatures (include/laep_moe.h).

The library is loaded from the package directory only.  If it has not been
built, every call raises -- there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
import threading

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblaep_moe.so")

LAEP_F32 = 0
LAEP_BF16 = 1

LAEP_CALL_ROUTE = 0
LAEP_CALL_COUNTS = 1
LAEP_CALL_FFN_FWD = 2
LAEP_CALL_FFN_BWD = 3
LAEP_CALL_ROUTE_BWD = 4

ERROR_NAMES = {
    1: "LAEP_ERR_INVALID_ARG",
    2: "LAEP_ERR_UNSUPPORTED",
    3: "LAEP_ERR_WORKSPACE",
    4: "LAEP_ERR_HIP",
    5: "LAEP_ERR_INFEASIBLE",
}


class LaepError(RuntimeError):
    """A C-ABI call returned an error code."""

    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERROR_NAMES.get(code, code)}: {msg}")
        self.code = code
        self.msg = msg


_p = ctypes.c_void_p
_i = ctypes.c_int
_i64 = ctypes.c_int64
_sz = ctypes.c_size_t
_d = ctypes.c_double

# name -> (restype, argtypes)
SIGNATURES = {
    "moe_route": (_i, [_p, _p, _p, _p, _i, _i, _i, _i, _i, _i, _p, _p, _p, _p, _sz, _p]),
    "moe_route_bwd": (_i, [_p, _p, _p, _p, _p, _p, _p, _p, _p, _i, _i, _i, _i, _i, _i, _p, _p,
                           _p, _p, _i, _p, _sz, _p]),
    "moe_expert_counts": (_i, [_p, _i, _i, _i, _p, _p, _p, _p, _p, _p, _sz, _p]),
    "moe_route_count": (_i, [_p, _p, _p, _p, _i, _i, _i, _i, _i, _i, _p, _p, _p, _p, _p, _p, _p,
                             _p, _p, _sz, _p]),
    "moe_route_count_noalloc": (_i, [_p, _p, _p, _p, _i, _i, _i, _i, _i, _i, _p, _p, _p, _p, _p,
                                     _p, _p, _p, _p]),
    "laep_prune_mask": (_i, [_p, _i, _i64, _d, _d, _p, _p, _p]),
    "laep_expert_pruning": (_i, [_p, _i, _i, _i, _i64, _p, _d, _p, _p, _p, _p]),
    "laep_compact_experts": (_i, [_p, _i, _i, _p, _p, _p]),
    "laep_repack_experts": (_i, [_p, _i, _i, _i, _i, _i, _p, _p, _p, _p, _p, _p, _p, _p, _p]),
    "moe_permute": (_i, [_p, _i, _p, _i, _i, _i, _p, _p]),
    "moe_grouped_ffn_fwd": (_i, [_p, _p, _p, _p, _p, _i, _i, _i, _i, _i64, _p, _p, _p, _sz, _p]),
    "moe_grouped_ffn_fwd_gather": (_i, [_p, _p, _i, _i, _p, _p, _p, _p, _i, _i, _i, _i, _i64,
                                        _p, _p, _p, _p, _sz, _p]),
    "moe_grouped_ffn_fwd_gather_combine": (_i, [_p, _p, _i, _i, _p, _p, _p, _p, _p, _i, _i, _i,
                                                _i, _i64, _p, _p, _p, _p, _p, _sz, _p]),
    "moe_grouped_ffn_bwd": (_i, [_p, _p, _p, _p, _p, _p, _p, _p, _i, _i, _i, _i, _i64, _p, _p, _p,
                                 _i, _p, _sz, _p]),
    "moe_grouped_ffn_bwd_gather": (_i, [_p, _p, _p, _p, _p, _i, _i, _p, _p, _p, _p, _p, _p, _i,
                                        _i, _i, _i, _i64, _p, _p, _p, _i, _p, _sz, _p]),
    "laep_ws_hb_offset": (_sz, [_i64, _i, _i]),
    "moe_combine": (_i, [_p, _p, _p, _i, _i, _i, _i, _p, _p]),
    "moe_combine_bwd": (_i, [_p, _p, _p, _p, _i, _i, _i, _i, _p, _p, _p]),
    "moe_permute_bwd": (_i, [_p, _p, _i, _i, _i, _i, _p, _p]),
    "moe_workspace_bytes": (_sz, [_i, _i, _i, _i, _i, _i]),
    "laep_rearrange": (_i, [_p, _i, _i, _p, _p, _p]),
    "laep_last_error": (ctypes.c_char_p, []),
    # measurement kernels (laep_calib.h)
    "laep_calib_copy": (_i, [_p, _p, _sz, _p]),
    "laep_calib_mfma": (_i, [_i, _i, _p, _p]),
    "laep_calib_read": (_i, [_p, _sz, _i, _p, _p]),
}

_lock = threading.Lock()
_lib = None


def bind(handle):
    """Apply the C signatures to a loaded handle of the library."""
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(handle, name)
        fn.restype = res
        fn.argtypes = args
    return handle


def lib():
    """The loaded library (raises if it was not built)."""
    global _lib
    if _lib is None:
        with _lock:
            if _lib is None:
                if not os.path.exists(LIB_PATH):
                    raise RuntimeError(
                        f"{LIB_PATH} is missing: build it with `python -c 'import "
                        f"__graft_entry__ as g; g.build()'` (no fallback implementation exists)")
                _lib = bind(ctypes.CDLL(LIB_PATH))
    return _lib


def check(rc: int):
    if rc != 0:
        msg = lib().laep_last_error().decode(errors="replace")
        raise LaepError(rc, msg)
