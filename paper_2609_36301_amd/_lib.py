"""ctypes declarations for libmore.so (argument marshalling only).

The library is loaded from this package directory.  If it has not been built the import
of any router function fails loudly; there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmore.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = range(5)
K_MAX = 32
LOWRANK_K_MAX = 32
LOWRANK_TRAIN_K_MAX = 16
ROUTE_WIDE = 4
NOALLOC_SCRATCH_BYTES = 256 << 20

# (name, restype, argtypes) for every symbol declared in include/more.h
_P = ctypes.c_void_p
_I64, _I32, _SZ = ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
_PSZ = ctypes.POINTER(ctypes.c_size_t)
_PI32 = ctypes.POINTER(ctypes.c_int32)
SIGNATURES = {
    "more_route_lowrank": (_I32, [_P, _P, _P, _I64, _I32, _I32, _I32, _I32, _P, _P, _P, _P, _P,
                                  _SZ, _P]),
    "more_route_lowrank_workspace_size": (_I32, [_I64, _I32, _I32, _I32, _I32, _PSZ]),
    "more_route_lowrank_ex": (_I32, [_P, _P, _P, _I64, _I32, _I32, _I32, _I32, _I32, _P, _P, _P,
                                     _P, _P, _SZ, _P]),
    "more_route_lowrank_workspace_size_ex": (_I32, [_I64, _I32, _I32, _I32, _I32, _I32, _PSZ]),
    "more_route_lowrank_plan": (_I32, [_I64, _I32, _I32, _I32, _I32, _PI32]),
    "more_route_lowrank_route": (_I32, [_I64, _I32, _I32, _I32, _I32, _PI32]),
    "more_route_lowrank_train": (_I32, [_P, _P, _P, _I64, _I32, _I32, _I32, _I32, _P, _P, _P,
                                        _P, _P, _P, _P, _P, _SZ, _P]),
    "more_route_lowrank_train_workspace_size": (_I32, [_I64, _I32, _I32, _I32, _I32, _PSZ]),
    "more_route_lowrank_backward": (_I32, [_P, _P, _P, _I64, _I32, _I32, _I32, _I32, _P, _P,
                                           _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "more_route_lowrank_backward_workspace_size": (_I32, [_I64, _I32, _I32, _I32, _I32, _I32,
                                                          _PSZ]),
    "more_route_fullrank": (_I32, [_P, _P, _I64, _I32, _I32, _I32, _I32, _P, _P, _P, _P, _SZ,
                                   _P]),
    "more_route_fullrank_workspace_size": (_I32, [_I64, _I32, _I32, _I32, _I32, _PSZ]),
    "more_route_fullrank_fused": (_I32, [_P, _P, _I64, _I32, _I32, _I32, _P, _P, _P, _P, _SZ,
                                         _P]),
    "more_route_fullrank_fused_workspace_size": (_I32, [_I64, _I32, _I32, _I32, _PSZ]),
    "more_expert_histogram": (_I32, [_P, _I64, _I32, _I32, _P, _P]),
    "more_dispatch_sort": (_I32, [_P, _I64, _I32, _I32, _P, _P, _P, _SZ, _P]),
    "more_dispatch_sort_workspace_size": (_I32, [_I64, _I32, _I32, _PSZ]),
    "more_route_lowrank_noalloc": (_I32, [_P, _P, _P, _I64, _I32, _I32, _I32, _I32, _P, _P, _P,
                                          _P, _P]),
    "more_status_string": (ctypes.c_char_p, [_I32]),
    "more_version": (ctypes.c_char_p, []),
}

_lib = None


class MoreError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s: %s" % (where, status_string(status)))


def load():
    """Load libmore.so (once).  Raises ImportError if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("%s is missing: build it with `python -m paper_2609_36301_amd.build`"
                          % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().more_status_string(status).decode()


def check(status: int, where: str):
    if status != OK:
        raise MoreError(status, where)
