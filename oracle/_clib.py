"""Loader for the oracle's plain-C selection routine (oracle/select.c).

TEST INFRASTRUCTURE ONLY.  The shared object is built with gcc by
the repository's build step (``build()`` below); this
module builds it on first use if it is missing.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liborderoracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile select.c with gcc (no HIP headers, no library sources)."""
    src = os.path.join(_HERE, "select.c")
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(src):
        tmp = _SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                               "-ffp-contract=off", "-fno-fast-math", src, "-o", tmp, "-lm"])
        os.replace(tmp, _SO)
    return _SO


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_SO)
        P = ctypes.c_void_p
        L.orc_select.restype = ctypes.c_int
        L.orc_select.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                 P, P, P, P, ctypes.c_float, P, ctypes.c_float, ctypes.c_float,
                                 ctypes.c_int32, ctypes.c_int32, P, P, P, P, P, P, P]
        _lib = L
    return _lib
