"""ctypes loader for ``libpulsar.so`` (the C ABI declared in include/pulsar.h).

Loading never falls back to anything: if the library is missing the call
raises, so no result can silently come from another implementation.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpulsar.so")

_c_int, _c_i64, _c_size, _c_float, _vp = (ctypes.c_int, ctypes.c_int64, ctypes.c_size_t,
                                         ctypes.c_float, ctypes.c_void_p)

# name -> (restype, argtypes); mirrors include/pulsar.h
SIGNATURES = {
    "pulsar_status_string": (ctypes.c_char_p, [_c_int]),
    "pulsar_version": (_c_int, []),
    "pulsar_maxidf_summaries": (_c_int, [_vp, _c_int, _c_i64, _c_int, _c_int, _c_int, _c_int,
                                         _vp, _vp, _vp, _vp, _c_size, _vp]),
    "pulsar_maxidf_workspace_bytes": (_c_size, [_c_int, _c_i64, _c_int, _c_int, _c_int]),
    "pulsar_chunk_summaries": (_c_int, [_vp, _c_int, _c_i64, _c_int, _c_int, _c_int, _c_int,
                                        _c_int, _vp, _vp, _vp, _c_size, _vp]),
    "pulsar_chunk_workspace_bytes": (_c_size, [_c_int, _c_i64, _c_int, _c_int, _c_int, _c_int]),
    "pulsar_phase1_len": (_c_i64, [_c_i64, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int]),
    "pulsar_phase1_positions": (_c_int, [_vp, _c_int, _c_i64, _c_int, _c_int, _c_int, _c_int,
                                         _c_int, _c_int, _vp, _vp]),
    "pulsar_phase1_gather": (_c_int, [_vp, _c_int, _c_i64, _c_int, _c_int, _c_int, _c_int, _c_int,
                                      _c_int, _c_int, _vp, _c_int, _c_int, _vp, ctypes.c_double,
                                      _vp, _vp]),
    "pulsar_phase1_attn": (_c_int, [_vp, _vp, _vp, _c_int, _c_i64, _c_int, _c_int, _c_int,
                                    _c_int, _c_int, _c_int, _c_int, _c_int, _vp, _c_int,
                                    _c_float, _vp, _c_int, _vp, _vp, _vp, _vp]),
    "pulsar_phase2_workspace_bytes": (_c_size, [_c_int, _c_int, _c_i64, _c_int, _c_int, _c_int]),
    "pulsar_phase2_partial": (_c_int, [_vp, _vp, _vp, _c_int, _c_int, _c_i64, _c_int, _c_int,
                                       _c_int, _c_float, _vp, _vp, _vp, _c_size, _vp]),
    "pulsar_lse_merge": (_c_int, [_vp, _vp, _c_int, _c_int, _c_int, _c_int, _vp, _vp, _vp]),
    "pulsar_phase2_query_workspace_bytes": (_c_size, [_c_int, _c_int, _c_i64, _c_i64, _c_int,
                                                       _c_int, _c_int]),
    "pulsar_phase2_query": (_c_int, [_vp, _vp, _vp, _c_i64, _vp, _vp, _c_int, _c_int, _c_i64,
                                     _c_int, _c_int, _c_int, _c_float, _vp, _vp, _vp, _c_size,
                                     _vp]),
    "pulsar_phase2_query_noalloc": (_c_int, [_vp, _vp, _vp, _c_i64, _vp, _vp, _c_int, _c_int,
                                             _c_i64, _c_int, _c_int, _c_int, _c_float, _vp, _vp,
                                             _vp]),
    "pulsar_rope": (_c_int, [_vp, _c_int, _c_i64, _c_int, _c_int, _vp, _c_i64, _vp,
                             ctypes.c_double, _vp]),
}

_lib = None


class PulsarError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what} failed: {status_string(status)} ({status})")


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2607_20457_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def status_string(status: int) -> str:
    return lib().pulsar_status_string(status).decode()


def check(status: int, what: str) -> None:
    if status != 0:
        raise PulsarError(status, what)
