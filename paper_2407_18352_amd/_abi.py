"""ctypes declarations of the C ABI in ``include/hpacml.h`` (argument
marshalling only: every step of the region runs in the HIP library)."""
from __future__ import annotations

import ctypes as C
import os

MAX_RANK = 4
OK, E_INVAL, E_SHAPE, E_RANGE, E_ALIAS, E_UNSUPPORTED, E_NOMEM, E_DEVICE = range(8)
TO, FROM = 0, 1
BND_NONE, BND_PERIODIC, BND_CLAMP = 0, 1, 2
F32, BF16 = 0, 1
ACT_IDENTITY, ACT_RELU = 0, 1
LAYER_CONV2D, LAYER_MAXPOOL2D, LAYER_LINEAR = 0, 1, 2
MODE_INFER, MODE_COLLECT, MODE_PREDICATED = 0, 1, 2
PAD_VALID, PAD_SAME = 0, 1
PADMODE_ZEROS, PADMODE_CIRCULAR, PADMODE_REPLICATE = 0, 1, 2

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhpacml.so")


class Slice(C.Structure):
    _fields_ = [("lo", C.c_int32 * MAX_RANK), ("count", C.c_int32 * MAX_RANK)]


class Functor(C.Structure):
    _fields_ = [("rank", C.c_int32), ("n_slices", C.c_int32),
                ("slices", C.POINTER(Slice)), ("n_features", C.c_int32)]


class Array(C.Structure):
    _fields_ = [("data", C.c_void_p), ("dtype", C.c_int32), ("reserved", C.c_int32),
                ("extent", C.c_int64 * MAX_RANK), ("stride", C.c_int64 * MAX_RANK)]


class Sweep(C.Structure):
    _fields_ = [("start", C.c_int64 * MAX_RANK), ("stop", C.c_int64 * MAX_RANK),
                ("step", C.c_int64 * MAX_RANK)]


class Layer(C.Structure):
    _fields_ = [("kind", C.c_int32), ("out_channels", C.c_int32), ("kernel", C.c_int32 * 2),
                ("stride", C.c_int32 * 2), ("padding", C.c_int32), ("pad_mode", C.c_int32), ("act", C.c_int32)]


# hpacml_accurate_fn: void (*)(void *user, void *stream)
ACCURATE_FN = C.CFUNCTYPE(None, C.c_void_p, C.c_void_p)

# every symbol the header declares, with (restype, argtypes)
_P = C.POINTER
SIGNATURES = {
    "hpacml_abi_version": (C.c_int32, []),
    "hpacml_status_string": (C.c_char_p, [C.c_int]),
    "hpacml_map_validate": (C.c_int, [_P(Functor), C.c_int32, _P(Array), C.c_int32, _P(Sweep),
                                      _P(C.c_int32), _P(C.c_int64), _P(C.c_int32)]),
    "hpacml_map_create": (C.c_int, [_P(Functor), C.c_int32, _P(Array), C.c_int32, _P(Sweep),
                                    _P(C.c_int32), _P(C.c_void_p)]),
    "hpacml_map_shape": (C.c_int, [C.c_void_p, _P(C.c_int64), _P(C.c_int32)]),
    "hpacml_map_destroy": (None, [C.c_void_p]),
    "hpacml_model_validate": (C.c_int, [C.c_int32, _P(C.c_int32), _P(C.c_int32), C.c_int32]),
    "hpacml_model_create": (C.c_int, [C.c_int32, _P(C.c_int32), _P(_P(C.c_float)), _P(_P(C.c_float)),
                                      _P(C.c_int32), C.c_int32, _P(C.c_void_p)]),
    "hpacml_model_destroy": (None, [C.c_void_p]),
    "hpacml_infer": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]),
    "hpacml_infer_noalloc": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]),
    "hpacml_collect": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p]),
    "hpacml_collect_pair": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p, C.c_int64,
                                      C.c_void_p]),
    "hpacml_infer_variant": (C.c_char_p, [C.c_void_p, C.c_void_p, C.c_void_p]),
    "hpacml_cnn_validate": (C.c_int, [C.c_int32, C.c_int32, C.c_int32, C.c_int32, _P(Layer), _P(C.c_int32)]),
    "hpacml_cnn_param_counts": (C.c_int, [C.c_int32, C.c_int32, C.c_int32, C.c_int32, _P(Layer), _P(C.c_int64),
                                          _P(C.c_int64)]),
    "hpacml_cnn_create": (C.c_int, [C.c_int32, C.c_int32, C.c_int32, C.c_int32, _P(Layer), _P(_P(C.c_float)),
                                    _P(_P(C.c_float)), C.c_int32, _P(C.c_void_p)]),
    "hpacml_region_create": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32, C.c_int64,
                                       _P(C.c_void_p)]),
    "hpacml_region_run": (C.c_int, [C.c_void_p, C.c_int32, C.c_int32, ACCURATE_FN, C.c_void_p, C.c_void_p]),
    "hpacml_region_samples": (C.c_int, [C.c_void_p, _P(C.c_int64)]),
    "hpacml_region_read": (C.c_int, [C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p, C.c_void_p]),
    "hpacml_region_save": (C.c_int, [C.c_void_p, C.c_char_p, C.c_char_p]),
    "hpacml_region_reset": (C.c_int, [C.c_void_p]),
    "hpacml_region_destroy": (None, [C.c_void_p]),
}

_lib = None


def lib():
    """Load the built library; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libhpacml.so is not built: run `python -m paper_2407_18352_amd.build` "
                               "(or __graft_entry__.build())")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


class HpacmlError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        msg = lib().hpacml_status_string(status).decode()
        super().__init__("%s failed: %s (status %d)" % (what, msg, status))


def check(status: int, what: str) -> None:
    if status != OK:
        raise HpacmlError(status, what)
