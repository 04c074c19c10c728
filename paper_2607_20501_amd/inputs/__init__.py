"""Seeded synthetic inputs (definition in include/mkgen.h).

This module produces the raw storage bytes of module inputs.  It holds none of
the modules' arithmetic; both the HIP library and the oracle consume the same
bytes.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libmkgen.so")
_lib = None

NORMAL, UNIFORM = 0, 1
_DT = {"f32": 0, "bf16": 1}


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(_LIB_PATH)
        lib.mkgen_fill.restype = ctypes.c_int
        lib.mkgen_fill.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32,
                                   ctypes.c_double, ctypes.c_double, ctypes.c_int32,
                                   ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        _lib = lib
    return _lib


def fill(seed, tensor_id, dist, p0, p1, dtype, n, first=0):
    """Elements [first, first+n) of tensor `tensor_id` as a numpy array
    (float32, or uint16 bfloat16 bit patterns)."""
    lib = _load()
    out = np.empty(n, dtype=np.float32 if dtype == "f32" else np.uint16)
    rc = lib.mkgen_fill(seed, tensor_id, dist, p0, p1, _DT[dtype], first, n,
                        out.ctypes.data_as(ctypes.c_void_p))
    if rc != 0:
        raise ValueError("mkgen_fill rejected its arguments")
    return out


def make_inputs(module, seed):
    """Generate every module input of `module` (see workloads.py) under `seed`;
    returns a list of flat numpy arrays in input order."""
    out = []
    for tid, (shape, recipe) in enumerate(zip(module["inputs"], module["recipes"])):
        n = int(np.prod(shape))
        dist, p0, p1 = recipe
        out.append(fill(seed, tid, dist, p0, p1, module["dtype"], n))
    return out


def bf16_bits_to_f32(bits):
    """Widen bfloat16 bit patterns to float32 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
