"""ctypes binding of libsoftneuro.so (the C ABI in include/softneuro.h).

Argument marshalling only: every step of the path runs inside the library.
The library is loaded from this package directory; if it is missing the
import fails loudly (there is no fallback implementation).
"""

from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsoftneuro.so")

# enums of softneuro.h
F32, F16, BF16 = 0, 1, 2
DTYPE = {"f32": F32, "f16": F16, "bf16": BF16}
NCHW, NHWC, NC8HW8 = 0, 1, 2
LAYOUT = {"NCHW": NCHW, "NHWC": NHWC, "NC8HW8": NC8HW8}
LAYOUT_NAME = {v: k for k, v in LAYOUT.items()}
DIRECT, IGEMM, WINOGRAD = 0, 1, 2
ALGO = {"direct": DIRECT, "igemm": IGEMM, "winograd": WINOGRAD}
ALGO_NAME = {v: k for k, v in ALGO.items()}
L_INPUT, L_CONV2D, L_MAXPOOL, L_GAP, L_ADD, L_FC, L_OUTPUT = range(7)
ACT = {"none": 0, "relu": 1, "relu6": 2}
SELECT_DPRS, SELECT_FIXED = 0, 1
OPT_LAYOUTS, OPT_ALGOS, OPT_PARAMS, OPT_HIPGRAPH, OPT_SEED, OPT_FLUSH, OPT_KEEP, OPT_DTYPES, OPT_WS_LIMIT = range(9)
DTYPE_NAME = {v: k for k, v in DTYPE.items()}

STATUS = {0: "SN_OK", -1: "SN_E_INVALID", -2: "SN_E_SHAPE", -3: "SN_E_STATE",
          -4: "SN_E_UNSUPPORTED", -5: "SN_E_DEVICE", -6: "SN_E_NOMEM", -7: "SN_E_INTERNAL"}


class SNError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


class LayerDesc(ctypes.Structure):
    _fields_ = [("type", ctypes.c_int32), ("k", ctypes.c_int32), ("r", ctypes.c_int32),
                ("s", ctypes.c_int32), ("stride", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("groups", ctypes.c_int32), ("act", ctypes.c_int32)]


class RoutineDesc(ctypes.Structure):
    _fields_ = [("id", ctypes.c_int32), ("layout", ctypes.c_int32), ("algo", ctypes.c_int32),
                ("param", ctypes.c_int32), ("dtype", ctypes.c_int32), ("schema", ctypes.c_int32),
                ("cost_ns", ctypes.c_int64), ("ws_bytes", ctypes.c_int64), ("name", ctypes.c_char * 64)]


# exported functions: name -> (restype, argtypes)
_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I32P = ctypes.POINTER(ctypes.c_int32)
_I64P = ctypes.POINTER(ctypes.c_int64)
SIGNATURES = {
    "sn_graph_create": (ctypes.c_int, [_I32, _I32, _I32, _I32, _I32, _I32, ctypes.POINTER(_P)]),
    "sn_set_option": (ctypes.c_int, [_P, _I32, ctypes.c_int64]),
    "sn_add_layer": (ctypes.c_int, [_P, ctypes.POINTER(LayerDesc), _I32P, _I32, _P,
                                    ctypes.POINTER(ctypes.c_float), _I32P]),
    "sn_add_input": (ctypes.c_int, [_P, _I32, _I32, _I32, _I32P]),
    "sn_add_projected_conv": (ctypes.c_int, [_P, ctypes.POINTER(LayerDesc), _I32, _I32, _I32, _P,
                                             ctypes.POINTER(ctypes.c_float), _P, ctypes.POINTER(ctypes.c_float),
                                             _I32P]),
    "sn_mark_output": (ctypes.c_int, [_P, _I32]),
    "sn_num_io": (ctypes.c_int, [_P, _I32P, _I32P]),
    "sn_run_mimo": (ctypes.c_int, [_P, ctypes.POINTER(_P), _I32, ctypes.POINTER(_P), _I32, _P]),
    "sn_profile": (ctypes.c_int, [_P, _I32, _I32, _P]),
    "sn_select_path": (ctypes.c_int, [_P, _I32, _I32, _I32]),
    "sn_set_path": (ctypes.c_int, [_P, _I32P, _I32]),
    "sn_run": (ctypes.c_int, [_P, _P, _P, _P]),
    "sn_run_noalloc": (ctypes.c_int, [_P, _P, _P, _P]),
    "sn_run_timed": (ctypes.c_int, [_P, _P, _P, _P, _I32, ctypes.POINTER(ctypes.c_float), _I32]),
    "sn_layer_output": (ctypes.c_int, [_P, _I32, _P, ctypes.c_size_t, ctypes.POINTER(ctypes.c_size_t),
                                       _I32P, _P]),
    "sn_plan_launches": (ctypes.c_int, [_P, _I32P, _I32, _I32P]),
    "sn_profile_integrated": (ctypes.c_int, [_P, _I32, _I32, _P, _I32P]),
    "sn_integrated_candidate": (ctypes.c_int, [_P, _I32, _I32P, _I32, _I64P, _I64P, _I32P]),
    "sn_refine_in_path": (ctypes.c_int, [_P, _I32, _I32, _I32, _P, _I32P]),
    "sn_get_costs": (ctypes.c_int, [_P, ctypes.c_char_p, ctypes.c_size_t,
                                    ctypes.POINTER(ctypes.c_size_t)]),
    "sn_set_costs": (ctypes.c_int, [_P, ctypes.c_char_p]),
    "sn_get_path": (ctypes.c_int, [_P, _I32P, _I32, _I64P]),
    "sn_num_layers": (ctypes.c_int, [_P, _I32P]),
    "sn_num_routines": (ctypes.c_int, [_P, _I32, _I32P]),
    "sn_routine_info": (ctypes.c_int, [_P, _I32, _I32, ctypes.POINTER(RoutineDesc)]),
    "sn_layer_shape": (ctypes.c_int, [_P, _I32, _I32P]),
    "sn_dp_stats": (ctypes.c_int, [_P, _I32, _I64P, _I64P]),
    "sn_graph_destroy": (None, [_P]),
    "sn_last_error": (ctypes.c_char_p, []),
}

_lib = None


def lib():
    """Load the library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run paper_2110_06037_amd/build.py "
                              "(or __graft_entry__.build()) first")
        # torch (device memory and streams) must load its HIP runtime first:
        # loaded after the library it would bind to the runtime the library
        # pulled in and find no GPU; loaded before, both share one device view
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def check(rc):
    if rc != 0:
        msg = lib().sn_last_error()
        raise SNError(rc, msg.decode() if msg else "")
    return rc
