"""ctypes declarations of the C ABI in include/rrf.h (same names).

Argument marshalling only: every step of the method runs in librrf's HIP
kernels.  Loading fails loudly when the library has not been built.
"""

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librrf.so")

RRF_F32, RRF_F64 = 0, 1
RRF_OK = 0
RRF_WARN_KMAX = 1
RRF_ERR_INVALID_ARG = -1
RRF_ERR_SHAPE = -2
RRF_ERR_NONFINITE = -3
RRF_ERR_NOMEM = -4
RRF_ERR_HIP = -5
RRF_ERR_INTERNAL = -6
RRF_STOP_TRAILING, RRF_STOP_SUBTRACT, RRF_STOP_SPECTRAL = 0, 1, 2
STAGES = ["sketch", "sample", "panel", "reduce", "formw", "update",
          "finalize", "orgqr"]
RRF_NUM_STAGES = len(STAGES)

_i64 = ctypes.c_int64
_u64 = ctypes.c_uint64
_vp = ctypes.c_void_p
_pvp = ctypes.POINTER(ctypes.c_void_p)
_pi64 = ctypes.POINTER(ctypes.c_int64)
_pd = ctypes.POINTER(ctypes.c_double)
_int = ctypes.c_int

# name: (restype, argtypes)
SIGNATURES = {
    "rrf_plan_create": (_int, [_pvp, _int, _i64, _i64, _i64, _i64, _vp]),
    "rrf_plan_create_in": (_int, [_pvp, _int, _i64, _i64, _i64, _i64, _vp, _vp,
                                  ctypes.c_size_t]),
    "rrf_run": (_int, [_vp, _vp, _i64, _i64, _i64, ctypes.c_double, _i64, _u64,
                       _pvp, _pi64, _pi64, _pvp, _pi64]),
    "rrf_destroy": (_int, [_vp]),
    "rrf_status_string": (ctypes.c_char_p, [_int]),
    "rrf_workspace_size": (_int, [_int, _i64, _i64, _i64, _i64,
                                  ctypes.POINTER(ctypes.c_size_t)]),
    "rrf_set_stop_mode": (_int, [_vp, _int]),
    "rrf_set_timing": (_int, [_vp, _int]),
    "rrf_get_trace": (_int, [_vp, _i64, _pi64, _pd, _pd, _pd, _pd, _pd]),
    "rrf_set_power_iterations": (_int, [_vp, _int]),
    "rrf_get_stage_stats": (_int, [_vp, _pd, _pi64, _pd, _pd]),
    "rrf_get_reflectors": (_int, [_vp, _pvp, _pi64, _pvp, _pi64, _pvp]),
    "rrf_sketch": (_int, [_int, _u64, _i64, _i64, _i64, _vp, _i64, _vp]),
    "rrf_panel_qr": (_int, [_vp, _vp, _i64, _i64, _i64, _vp, _i64, _vp, _i64,
                            _vp]),
    "rrf_apply_block_reflector": (_int, [_vp, _int, _vp, _i64, _vp, _i64, _i64,
                                         _vp, _i64, _i64, _i64]),
    "rrf_copy_matrix": (_int, [_int, _vp, _i64, _vp, _i64, _i64, _i64, _vp]),
    "rrf_panel_qr_noalloc": (_int, [_int, _vp, _i64, _i64, _i64, _vp, _i64, _vp, _i64,
                                    _vp, _vp, _vp]),
    "rrf_subspace_map": (_int, [_vp, _vp, _i64, _i64, _vp, _i64, _i64, _vp, _i64,
                                _i64, _i64, _vp, _i64]),
}

_lib = None


class RRFError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


def load():
    """The loaded librrf (ctypes.CDLL); raises if it was not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2608_28941_amd.build` (no CPU fallback exists)")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def status_string(status):
    return load().rrf_status_string(int(status)).decode()


def check(status, where, allow_warn=True):
    if status < 0 or (status > 0 and not allow_warn):
        raise RRFError(status, where)
    return status
