"""ctypes loader for libacceptmoe.so (the C ABI in include/acceptmoe.h).

Loading fails loudly when the library has not been built: there is no
fallback implementation of any step.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libacceptmoe.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_UNSUPPORTED = -2
ERR_WORKSPACE = -3
ERR_HIP = -4

F32 = 0
BF16 = 1

MODE_SELF_SIZING = 0
MODE_ALL_EXPERTS = 1
MODE_FIXED_BUDGET = 2
MODE_MOESPEC = 3
MODE_COUNT = 4

NUM_STATS = 10

# offload pool counters (int64[POOL_NUM_STATS], accumulated by acceptmoe_pool_serve_wave)
POOL_WAVES, POOL_ACCESSES, POOL_HITS, POOL_MISSES, POOL_H2D_BYTES = range(5)
POOL_NUM_STATS = 5
MAX_EXPERTS = 512
MAX_TOPK = 32
MAX_TREES = 256
MAX_TREE_NODES = 1024
SELECT_NOALLOC_MAX_WORKSPACE = 8 << 20

_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_sz = ctypes.c_size_t

SIGNATURES = {
    "acceptmoe_packed_router_bytes": (ctypes.c_size_t, [_i32, _i32]),
    "acceptmoe_pack_router_weights": (_i32, [_vp, _i32, _i32, _vp, _vp]),
    "acceptmoe_route": (_i32, [_vp, _i32, _vp, _i32, _i32, _i32, _vp, _vp]),
    "acceptmoe_select_workspace_size": (_sz, [_i32, _i32, _i32]),
    "acceptmoe_select": (_i32, [_vp, _vp, _vp, _vp, ctypes.POINTER(_i32), _i32, _i32, _i32, _i32,
                                ctypes.c_double, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _sz,
                                _vp]),
    "acceptmoe_select_noalloc": (_i32, [_vp, _vp, _vp, _vp, ctypes.POINTER(_i32), _i32, _i32, _i32, _i32,
                                        ctypes.c_double, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp]),
    "acceptmoe_packed_weights_bytes": (_sz, [_i32, _i32, _i32, _i32]),
    "acceptmoe_pack_expert_weights": (_i32, [_vp, _i32, _i32, _i32, _i32, _vp, _vp]),
    "acceptmoe_moe_forward_workspace_size": (_sz, [_i32, _i32, _i32, _i32, _i32, _i32]),
    "acceptmoe_packed_gate_up_bytes": (_sz, [_i32, _i32, _i32, _i32]),
    "acceptmoe_pack_gate_up_weights": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _vp, _vp]),
    "acceptmoe_moe_forward": (_i32, [_vp, _i32, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp,
                                     _vp, _vp, _sz, _vp]),
    "acceptmoe_residual_add": (_i32, [_vp, _i32, _vp, _i32, _i32, _vp, _vp]),
    "acceptmoe_commit_count": (_i32, [_vp, _vp, _i32, _i32, _vp, _vp]),
    "acceptmoe_commit_estimate": (_i32, [_vp, _vp, _i32, _vp]),
    "acceptmoe_commit_expand": (_i32, [_vp, _i32, _vp, _i32, _vp, _vp]),
    "acceptmoe_pool_state_bytes": (_sz, [_i32, _i32]),
    "acceptmoe_pool_init": (_i32, [_vp, _sz, _i32, _i32]),
    "acceptmoe_pool_resident_mask": (_i32, [_vp, _vp]),
    "acceptmoe_pool_plan_waves": (_i32, [_vp, _i32, _i32, _i32, _i32, _vp, _vp]),
    "acceptmoe_pool_serve_wave": (_i32, [_vp, _vp, _vp, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _sz, _sz, _vp, _vp,
                                         _vp]),
    "acceptmoe_copy_rows": (_i32, [_vp, _vp, _vp, _i32, _i32, _i32, _vp]),
    "acceptmoe_stream_read": (_i32, [_vp, _sz, _vp, _i32, _vp]),
    "acceptmoe_last_error": (ctypes.c_char_p, []),
    "acceptmoe_version": (_i32, []),
}

_LIB = None


class AcceptMoEError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"acceptmoe status {status}: {message}")
        self.status = status


def lib() -> ctypes.CDLL:
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"HIP library {LIB_PATH} is not built; run __graft_entry__.build() "
                               "(python -m paper_2608_02989_amd.build) first")
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = h
    return _LIB


def check(status: int) -> None:
    if status != OK:
        msg = lib().acceptmoe_last_error().decode(errors="replace")
        raise AcceptMoEError(status, msg)
