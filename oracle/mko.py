"""ctypes wrapper of the oracle library (mko.c).  Test infrastructure only.

A module is a plain dict {"dtype": "f32"|"bf16", "inputs": [shape, ...],
"ops": [{"kind": name, "in": [...], "ip": [...], "fp": [...]}, ...]}; inputs
are flat numpy arrays of the storage type (float32, or uint16 bfloat16 bits).
"""
import contextlib
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# MKO_LIBRARY names another build of the oracle (the sanitized build).
_LIB = os.environ.get("MKO_LIBRARY") or os.path.join(_HERE, "libmko.so")
_lib = None

KINDS = ["GEMM", "BIAS", "BIAS_CHANNEL", "RELU", "GELU_ERF", "GELU_TANH", "SCALE", "ADD",
         "ROWSUM", "SOFTMAX", "LAYERNORM", "CONV2D", "GAP", "QK", "CAUSAL_MASK", "PV",
         "GMP", "LPPOOL"]
MAX_OPS = 64


class _Shape(ctypes.Structure):
    _fields_ = [("ndim", ctypes.c_int32), ("dims", ctypes.c_int64 * 4)]


class _Op(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("in_", ctypes.c_int32 * 3),
                ("ip", ctypes.c_int64 * 4), ("fp", ctypes.c_double * 2)]


class _Desc(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("n_inputs", ctypes.c_int32),
                ("input_shapes", ctypes.POINTER(_Shape)), ("n_ops", ctypes.c_int32),
                ("ops", ctypes.POINTER(_Op))]


class _Group(ctypes.Structure):
    _fields_ = [("op_begin", ctypes.c_int32), ("op_end", ctypes.c_int32),
                ("out_value", ctypes.c_int32), ("out_shape", _Shape),
                ("out_bytes", ctypes.c_int64), ("ws_offset", ctypes.c_int64),
                ("flops", ctypes.c_int64), ("alg_bytes", ctypes.c_int64)]


class _Plan(ctypes.Structure):
    _fields_ = [("n_groups", ctypes.c_int32), ("g", _Group * MAX_OPS),
                ("value_shapes", _Shape * (2 * MAX_OPS)),
                ("ws_intermediate_bytes", ctypes.c_int64), ("flops", ctypes.c_int64),
                ("alg_bytes", ctypes.c_int64)]


SOURCE = os.path.join(_HERE, "mko.c")


def build(src=SOURCE, out=None):
    """Compile the oracle with gcc (plain C99, OpenMP): libmko.so from mko.c by
    default; tests that plant a mistake in a copy of mko.c build that copy."""
    out = out or _LIB
    tmp = out + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=c99", "-D_DEFAULT_SOURCE", "-fPIC", "-shared",
                           "-fopenmp", "-Wall", "-I", _HERE, "-o", tmp, src, "-lm"])
    os.replace(tmp, out)


@contextlib.contextmanager
def library(path):
    """Evaluate with another build of the oracle inside the block (used by the
    tests that show a pin rejects a planted mistake)."""
    global _lib, _LIB
    saved = (_lib, _LIB)
    _lib, _LIB = None, path
    try:
        yield
    finally:
        _lib, _LIB = saved


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        lib.mko_plan.restype = ctypes.c_int
        lib.mko_plan.argtypes = [ctypes.POINTER(_Desc), ctypes.POINTER(ctypes.c_int32),
                                 ctypes.POINTER(_Plan)]
        lib.mko_run.restype = ctypes.c_int
        lib.mko_run.argtypes = [ctypes.POINTER(_Desc), ctypes.POINTER(ctypes.c_int32),
                                ctypes.POINTER(ctypes.c_void_p),
                                ctypes.POINTER(ctypes.POINTER(ctypes.c_double)),
                                ctypes.c_int, ctypes.c_int]
        for name in ("mko_round_bf16", "mko_round_f32", "mko_gelu_erf", "mko_gelu_tanh"):
            f = getattr(lib, name)
            f.restype = ctypes.c_double
            f.argtypes = [ctypes.c_double]
        _lib = lib
    return _lib


def _marshal(module):
    shapes = (_Shape * max(1, len(module["inputs"])))()
    for i, s in enumerate(module["inputs"]):
        shapes[i].ndim = len(s)
        for k, v in enumerate(s):
            shapes[i].dims[k] = int(v)
    ops = (_Op * len(module["ops"]))()
    for i, o in enumerate(module["ops"]):
        ops[i].kind = KINDS.index(o["kind"])
        ins = list(o["in"]) + [-1] * (3 - len(o["in"]))
        for k in range(3):
            ops[i].in_[k] = ins[k]
        for k, v in enumerate(o.get("ip", [])):
            ops[i].ip[k] = int(v)
        for k, v in enumerate(o.get("fp", [])):
            ops[i].fp[k] = float(v)
    d = _Desc(0 if module["dtype"] == "f32" else 1, len(module["inputs"]), shapes,
              len(module["ops"]), ops)
    return d, (shapes, ops)


def _groups(module, groups):
    g = (ctypes.c_int32 * len(module["ops"]))(*[int(x) for x in groups])
    return g


def _shape_tuple(s):
    return tuple(int(s.dims[k]) for k in range(s.ndim))


def plan(module, groups):
    """Bookkeeping of a grouping; returns a dict, or raises ValueError with the
    oracle's code (-1 argument, -2 shape, -3 grouping)."""
    lib = _load()
    d, keep = _marshal(module)
    p = _Plan()
    rc = lib.mko_plan(ctypes.byref(d), _groups(module, groups), ctypes.byref(p))
    if rc != 0:
        raise ValueError(rc)
    gs = []
    for i in range(p.n_groups):
        G = p.g[i]
        gs.append({"op_begin": G.op_begin, "op_end": G.op_end, "out_value": G.out_value,
                   "out_shape": _shape_tuple(G.out_shape), "out_bytes": G.out_bytes,
                   "ws_offset": G.ws_offset, "flops": G.flops, "alg_bytes": G.alg_bytes})
    nv = len(module["inputs"]) + len(module["ops"])
    return {"groups": gs, "ws_intermediate_bytes": p.ws_intermediate_bytes,
            "flops": p.flops, "alg_bytes": p.alg_bytes,
            "value_shapes": [_shape_tuple(p.value_shapes[i]) for i in range(nv)]}


def run(module, groups, inputs, ideal=False, nthreads=0, keep=None):
    """Evaluate; returns a list with op i's fp64 output (shaped) for every op
    (or only for the op indices in `keep`, None elsewhere)."""
    lib = _load()
    info = plan(module, groups)
    d, hold = _marshal(module)
    nin = len(module["inputs"])
    arrs = []
    for i, x in enumerate(inputs):
        want = np.float32 if module["dtype"] == "f32" else np.uint16
        a = np.ascontiguousarray(np.asarray(x).reshape(-1), dtype=want)
        if a.size != int(np.prod(module["inputs"][i])):
            raise ValueError(f"input {i} has {a.size} elements")
        arrs.append(a)
    ptrs = (ctypes.c_void_p * max(1, nin))(*[a.ctypes.data for a in arrs])
    outs = []
    optrs = (ctypes.POINTER(ctypes.c_double) * len(module["ops"]))()
    for i in range(len(module["ops"])):
        if keep is None or i in keep:
            shp = info["value_shapes"][nin + i]
            o = np.empty(shp, dtype=np.float64)
            outs.append(o)
            optrs[i] = o.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
        else:
            outs.append(None)
    rc = lib.mko_run(ctypes.byref(d), _groups(module, groups), ptrs, optrs,
                     1 if ideal else 0, int(nthreads))
    if rc != 0:
        raise ValueError(rc)
    return outs


def round_bf16(v):
    return _load().mko_round_bf16(float(v))


def round_f32(v):
    return _load().mko_round_f32(float(v))


def gelu_erf(v):
    return _load().mko_gelu_erf(float(v))


def gelu_tanh(v):
    return _load().mko_gelu_tanh(float(v))
