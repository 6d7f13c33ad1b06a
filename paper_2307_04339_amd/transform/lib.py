"""ctypes binding of libmiriam_elastified.so: the plain kernels of transform/plain and their
elastic forms, with argument types derived from the plain kernels' parameter lists."""
from __future__ import annotations

import ctypes
import os
import re

from . import elastify

PKG = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB_PATH = os.path.join(PKG, "libmiriam_elastified.so")

_CTYPE = {"int": ctypes.c_int, "unsigned": ctypes.c_uint, "float": ctypes.c_float, "long long": ctypes.c_longlong,
          "double": ctypes.c_double}

_lib = None
_kernels = None


def _argtype(param: str):
    p = param.strip()
    if "*" in p:
        return ctypes.c_void_p
    base = re.sub(r"\bconst\b", "", p).strip().rsplit(None, 1)[0].strip()
    if base not in _CTYPE:
        raise TypeError(f"no ctypes mapping for parameter {param!r}")
    return _CTYPE[base]


def kernels() -> dict:
    """Plain kernels by name (elastify.Kernel)."""
    global _kernels
    if _kernels is None:
        ks = {}
        for f in sorted(os.listdir(elastify.PLAIN_DIR)):
            if f.endswith(".hip"):
                with open(os.path.join(elastify.PLAIN_DIR, f)) as fh:
                    for k in elastify.parse(fh.read()):
                        ks[k.name] = k
        _kernels = ks
    return _kernels


def load():
    """Load the library (raises if it has not been built) and set every launcher's signature."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run python -m paper_2307_04339_amd.build")
    lib = ctypes.CDLL(LIB_PATH)
    for name, k in kernels().items():
        args = [_argtype(p) for p in k.params.split(",")]
        fp = getattr(lib, f"{name}_plain_launch")
        fp.argtypes = args + [ctypes.c_int, ctypes.c_int, ctypes.c_void_p]  # grid_x, grid_y, stream
        fp.restype = ctypes.c_int
        fe = getattr(lib, f"{name}_elastic_launch")
        # grid_x, grid_y, begin, len, grid, block, stream
        fe.argtypes = args + [ctypes.c_int, ctypes.c_int, ctypes.c_longlong, ctypes.c_longlong, ctypes.c_int,
                              ctypes.c_int, ctypes.c_void_p]
        fe.restype = ctypes.c_int
    _lib = lib
    return lib
