"""Python binding of libmk (include/mk.h).

Argument marshalling only: every step of a module runs in the HIP library.
PyTorch provides device memory and streams.  The functions keep the C names;
`Module` is a small convenience wrapper over them.
"""
import ctypes
import os
import warnings

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# MK_LIBRARY names another build of the same library (the sanitized host
# build that a CPU test runs the host-side tests against).
LIB_PATH = os.environ.get("MK_LIBRARY") or os.path.join(_HERE, "libmk.so")

KINDS = ["GEMM", "BIAS", "BIAS_CHANNEL", "RELU", "GELU_ERF", "GELU_TANH", "SCALE", "ADD",
         "ROWSUM", "SOFTMAX", "LAYERNORM", "CONV2D", "GAP", "QK", "CAUSAL_MASK", "PV",
         "GMP", "LPPOOL"]
FAMILIES = ["GEMM", "CONV", "EW", "ROW", "ATTN"]
# mk_tuned_limit: why the tuned implementation of a contraction subkernel
# runs the simple kernels ("none": it does not).
TUNED_LIMITS = ["none", "dtype", "align", "shape", "range"]
STATUS = ["MK_OK", "MK_E_INVALID_ARG", "MK_E_SHAPE", "MK_E_DTYPE", "MK_E_DECOMP",
          "MK_E_UNSUPPORTED", "MK_E_WORKSPACE", "MK_E_HIP", "MK_E_INTERNAL"]
IMPL_TUNED, IMPL_SIMPLE = 0, 1
MAX_CHECKS = 64


class MkError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS[status] if 0 <= status < len(STATUS) else status}: {msg}")
        self.status = status


class TunedLimitWarning(UserWarning):
    """The tuned implementation of a subkernel runs the simple kernels on
    these shapes (mk_tuned_limit); results are unaffected, speed is not."""


class mk_shape(ctypes.Structure):
    _fields_ = [("ndim", ctypes.c_int32), ("dims", ctypes.c_int64 * 4)]


class mk_op(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("in_", ctypes.c_int32 * 3),
                ("ip", ctypes.c_int64 * 4), ("fp", ctypes.c_double * 2)]


class mk_module_desc(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("n_inputs", ctypes.c_int32),
                ("input_shapes", ctypes.POINTER(mk_shape)), ("n_ops", ctypes.c_int32),
                ("ops", ctypes.POINTER(mk_op))]


class mk_module_info_t(ctypes.Structure):
    _fields_ = [("n_subkernels", ctypes.c_int32), ("n_ops", ctypes.c_int32),
                ("out_shape", mk_shape), ("ws_bytes", ctypes.c_int64),
                ("ws_intermediate_bytes", ctypes.c_int64), ("flops", ctypes.c_int64),
                ("alg_bytes", ctypes.c_int64)]


class mk_subkernel_info_t(ctypes.Structure):
    _fields_ = [("op_begin", ctypes.c_int32), ("op_end", ctypes.c_int32),
                ("out_value", ctypes.c_int32), ("out_shape", mk_shape),
                ("out_bytes", ctypes.c_int64), ("ws_offset", ctypes.c_int64),
                ("flops", ctypes.c_int64), ("alg_bytes", ctypes.c_int64),
                ("family", ctypes.c_int32), ("impl", ctypes.c_int32),
                ("n_launches", ctypes.c_int32), ("scratch_bytes", ctypes.c_int64),
                ("uses_mfma", ctypes.c_int32), ("tuned_limit", ctypes.c_int32)]


class mk_check(ctypes.Structure):
    _fields_ = [("stage", ctypes.c_int32), ("n", ctypes.c_int64),
                ("index", ctypes.POINTER(ctypes.c_int64)),
                ("expect", ctypes.POINTER(ctypes.c_double)),
                ("rtol", ctypes.c_double), ("atol", ctypes.c_double)]


class mk_check_result(ctypes.Structure):
    _fields_ = [("stage", ctypes.c_int32), ("pass_", ctypes.c_int32),
                ("n_checked", ctypes.c_int64), ("n_violations", ctypes.c_int64),
                ("n_nonfinite", ctypes.c_int64), ("max_abs_err", ctypes.c_double),
                ("max_rel_err", ctypes.c_double), ("worst_ratio", ctypes.c_double),
                ("worst_index", ctypes.c_int64), ("got_at_worst", ctypes.c_double),
                ("expect_at_worst", ctypes.c_double)]


class mk_verify_report(ctypes.Structure):
    _fields_ = [("pass_", ctypes.c_int32), ("first_failing_stage", ctypes.c_int32),
                ("n_results", ctypes.c_int32), ("results", mk_check_result * MAX_CHECKS)]


EXPORTS = ["mk_decomposition_preset", "mk_module_create", "mk_module_destroy", "mk_module_info",
           "mk_subkernel_info", "mk_subkernel_select", "mk_workspace_size", "mk_run",
           "mk_verify", "mk_status_str", "mk_last_error", "mk_profile_begin", "mk_profile_end",
           "mk_swap_decide", "mk_swap", "mk_budget_shares", "mk_gen_fill", "mk_run_noalloc"]
NOALLOC_WS_BYTES = 64 << 20   # MK_NOALLOC_WS_BYTES

_lib = None


def load():
    """Load libmk.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    # torch carries its own copy of the HIP runtime under the same soname;
    # loaded first, it is the one libmk binds to.  Loaded after libmk, it
    # would be a second runtime in the process, and libmk's own calls (device
    # queries, events) would not see the devices torch's memory lives on.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    vp = ctypes.c_void_p
    lib.mk_decomposition_preset.argtypes = [P(mk_module_desc), ctypes.c_int32, P(ctypes.c_int32)]
    lib.mk_module_create.argtypes = [P(mk_module_desc), P(ctypes.c_int32), P(vp)]
    lib.mk_module_destroy.argtypes = [vp]
    lib.mk_module_destroy.restype = None
    lib.mk_module_info.argtypes = [vp, P(mk_module_info_t)]
    lib.mk_subkernel_info.argtypes = [vp, ctypes.c_int32, P(mk_subkernel_info_t)]
    lib.mk_subkernel_select.argtypes = [vp, ctypes.c_int32, ctypes.c_int32]
    lib.mk_workspace_size.argtypes = [vp, P(ctypes.c_int64)]
    lib.mk_run.argtypes = [vp, P(vp), vp, vp, ctypes.c_int64, vp, P(ctypes.c_float)]
    lib.mk_run_noalloc.argtypes = [vp, P(vp), vp, vp]
    lib.mk_verify.argtypes = [vp, P(vp), vp, vp, ctypes.c_int64, vp, ctypes.c_int32,
                              P(mk_check), P(mk_verify_report)]
    for f in ("mk_decomposition_preset", "mk_module_create", "mk_module_info",
              "mk_subkernel_info", "mk_subkernel_select", "mk_workspace_size", "mk_run",
              "mk_run_noalloc", "mk_verify"):
        getattr(lib, f).restype = ctypes.c_int
    lib.mk_profile_begin.argtypes = [vp, ctypes.c_int32, ctypes.c_int32]
    lib.mk_profile_end.argtypes = [vp, P(ctypes.c_float), ctypes.c_int32, P(ctypes.c_int32)]
    lib.mk_profile_begin.restype = ctypes.c_int
    lib.mk_profile_end.restype = ctypes.c_int
    fp, ip = P(ctypes.c_float), P(ctypes.c_int32)
    lib.mk_swap_decide.argtypes = [ctypes.c_int32, fp, fp, ctypes.c_float, ip, ip]
    lib.mk_swap.argtypes = [vp, P(vp), vp, vp, ctypes.c_int64, vp, ctypes.c_int32,
                            ctypes.c_float, ctypes.c_int32, fp, fp, ip, ip]
    lib.mk_budget_shares.argtypes = [ctypes.c_int32, fp, ip, fp]
    for f in ("mk_swap_decide", "mk_swap", "mk_budget_shares"):
        getattr(lib, f).restype = ctypes.c_int
    lib.mk_gen_fill.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32,
                                ctypes.c_double, ctypes.c_double, ctypes.c_int32, vp,
                                ctypes.c_int64]
    lib.mk_gen_fill.restype = ctypes.c_int
    lib.mk_status_str.argtypes = [ctypes.c_int]
    lib.mk_status_str.restype = ctypes.c_char_p
    lib.mk_last_error.argtypes = []
    lib.mk_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(rc):
    if rc != 0:
        raise MkError(rc, load().mk_last_error().decode())


def marshal(module):
    """Module dict (see workloads.py) -> (mk_module_desc, keep-alive tuple)."""
    n_in = len(module["inputs"])
    shapes = (mk_shape * max(1, n_in))()
    for i, s in enumerate(module["inputs"]):
        shapes[i].ndim = len(s)
        for k, v in enumerate(s):
            shapes[i].dims[k] = int(v)
    ops = (mk_op * len(module["ops"]))()
    for i, o in enumerate(module["ops"]):
        ops[i].kind = KINDS.index(o["kind"])
        ins = list(o["in"]) + [-1] * (3 - len(o["in"]))
        for k in range(3):
            ops[i].in_[k] = int(ins[k])
        for k, v in enumerate(o.get("ip", [])):
            ops[i].ip[k] = int(v)
        for k, v in enumerate(o.get("fp", [])):
            ops[i].fp[k] = float(v)
    dt = {"f32": 0, "bf16": 1}.get(module["dtype"], module["dtype"])
    desc = mk_module_desc(dt, n_in, shapes, len(module["ops"]), ops)
    return desc, (shapes, ops)


def _shape(s):
    return tuple(int(s.dims[k]) for k in range(s.ndim))


def mk_decomposition_preset(module, preset):
    """preset: 0/'split' or 1/'fused' -> list of group ids."""
    preset = {"split": 0, "fused": 1}.get(preset, preset)
    desc, keep = marshal(module)
    g = (ctypes.c_int32 * len(module["ops"]))()
    _check(load().mk_decomposition_preset(ctypes.byref(desc), int(preset), g))
    return list(g)


def mk_module_create(module, groups):
    desc, keep = marshal(module)
    g = (ctypes.c_int32 * len(module["ops"]))(*[int(x) for x in groups])
    h = ctypes.c_void_p()
    _check(load().mk_module_create(ctypes.byref(desc), g, ctypes.byref(h)))
    return h


def mk_module_destroy(h):
    load().mk_module_destroy(h)


def mk_module_info(h):
    i = mk_module_info_t()
    _check(load().mk_module_info(h, ctypes.byref(i)))
    return {"n_subkernels": i.n_subkernels, "n_ops": i.n_ops, "out_shape": _shape(i.out_shape),
            "ws_bytes": i.ws_bytes, "ws_intermediate_bytes": i.ws_intermediate_bytes,
            "flops": i.flops, "alg_bytes": i.alg_bytes}


def mk_subkernel_info(h, i):
    s = mk_subkernel_info_t()
    _check(load().mk_subkernel_info(h, int(i), ctypes.byref(s)))
    return {"op_begin": s.op_begin, "op_end": s.op_end, "out_value": s.out_value,
            "out_shape": _shape(s.out_shape), "out_bytes": s.out_bytes,
            "ws_offset": s.ws_offset, "flops": s.flops, "alg_bytes": s.alg_bytes,
            "family": FAMILIES[s.family], "impl": s.impl, "n_launches": s.n_launches,
            "scratch_bytes": s.scratch_bytes, "uses_mfma": bool(s.uses_mfma),
            "tuned_limit": TUNED_LIMITS[s.tuned_limit]}


def mk_subkernel_select(h, i, impl):
    _check(load().mk_subkernel_select(h, int(i), int(impl)))


def mk_workspace_size(h):
    b = ctypes.c_int64()
    _check(load().mk_workspace_size(h, ctypes.byref(b)))
    return b.value


def mk_run(h, dev_inputs, dev_out, dev_ws, ws_bytes, stream, n_subkernels=None):
    """dev_* are device addresses (ints); stream a hipStream_t address or 0.
    With n_subkernels given, returns per-subkernel milliseconds (synchronises)."""
    ptrs = (ctypes.c_void_p * max(1, len(dev_inputs)))(*dev_inputs)
    ms = (ctypes.c_float * n_subkernels)() if n_subkernels else None
    _check(load().mk_run(h, ptrs, dev_out, dev_ws, int(ws_bytes), stream, ms))
    return list(ms) if ms is not None else None


def mk_run_noalloc(h, dev_inputs, dev_out, stream):
    """mk_run on the library's static workspace (no workspace argument)."""
    ptrs = (ctypes.c_void_p * max(1, len(dev_inputs)))(*dev_inputs)
    _check(load().mk_run_noalloc(h, ptrs, dev_out, stream))


def mk_profile_begin(h, max_launches, only_launch=-1):
    _check(load().mk_profile_begin(h, int(max_launches), int(only_launch)))


def mk_profile_end(h, capacity):
    """Returns the list of recorded per-launch milliseconds."""
    buf = (ctypes.c_float * max(1, capacity))()
    n = ctypes.c_int32()
    _check(load().mk_profile_end(h, buf, int(capacity), ctypes.byref(n)))
    return list(buf[:min(n.value, capacity)])


def mk_verify(h, dev_inputs, dev_out, dev_ws, ws_bytes, stream, checks):
    """checks: list of dicts {stage, expect (float64 array), index (int64 array
    or None), rtol, atol}.  Returns the report as a dict."""
    if len(checks) > MAX_CHECKS:
        raise ValueError("too many checks")
    arr = (mk_check * max(1, len(checks)))()
    keep = []
    for i, c in enumerate(checks):
        e = np.ascontiguousarray(c["expect"], dtype=np.float64).reshape(-1)
        keep.append(e)
        arr[i].stage = int(c["stage"])
        arr[i].n = e.size
        arr[i].expect = e.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
        if c.get("index") is not None:
            ix = np.ascontiguousarray(c["index"], dtype=np.int64).reshape(-1)
            if ix.size != e.size:
                raise ValueError("index and expect sizes differ")
            keep.append(ix)
            arr[i].index = ix.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))
        arr[i].rtol = float(c["rtol"])
        arr[i].atol = float(c["atol"])
    ptrs = (ctypes.c_void_p * max(1, len(dev_inputs)))(*dev_inputs)
    rep = mk_verify_report()
    _check(load().mk_verify(h, ptrs, dev_out, dev_ws, int(ws_bytes), stream, len(checks), arr,
                            ctypes.byref(rep)))
    res = []
    for i in range(rep.n_results):
        r = rep.results[i]
        res.append({"stage": r.stage, "pass": bool(r.pass_), "n_checked": r.n_checked,
                    "n_violations": r.n_violations, "n_nonfinite": r.n_nonfinite,
                    "max_abs_err": r.max_abs_err, "max_rel_err": r.max_rel_err,
                    "worst_ratio": r.worst_ratio, "worst_index": r.worst_index,
                    "got_at_worst": r.got_at_worst, "expect_at_worst": r.expect_at_worst})
    return {"pass": bool(rep.pass_), "first_failing_stage": rep.first_failing_stage,
            "results": res}


def mk_gen_fill(seed, tensor_id, dist, p0, p1, dtype, n):
    """Elements 0..n-1 of seeded input tensor `tensor_id` (numpy float32, or
    uint16 bfloat16 bit patterns for dtype 'bf16')."""
    bf = dtype in ("bf16", 1)
    out = np.empty(int(n), dtype=np.uint16 if bf else np.float32)
    _check(load().mk_gen_fill(int(seed), int(tensor_id), int(dist), float(p0), float(p1),
                              1 if bf else 0, out.ctypes.data_as(ctypes.c_void_p), int(n)))
    return out


def mk_swap_decide(ms_selected, ms_reference, tau):
    """-> (swap flags, triggered) for per-subkernel times (host lists)."""
    n = len(ms_selected)
    a = (ctypes.c_float * max(1, n))(*ms_selected)
    b = (ctypes.c_float * max(1, n))(*ms_reference)
    sw = (ctypes.c_int32 * max(1, n))()
    trig = ctypes.c_int32()
    _check(load().mk_swap_decide(n, a, b, float(tau), sw, ctypes.byref(trig)))
    return [int(x) for x in sw[:n]], bool(trig.value)


def mk_budget_shares(ms, needs_work=None):
    n = len(ms)
    a = (ctypes.c_float * max(1, n))(*ms)
    w = (ctypes.c_int32 * max(1, n))(*(needs_work or [0] * n)) if needs_work is not None else None
    out = (ctypes.c_float * max(1, n))()
    _check(load().mk_budget_shares(n, a, w, out))
    return list(out[:n])


# ------------------------------------------------------------------ convenience

class Module:
    """A created module plus its device buffers (torch tensors)."""

    def __init__(self, module, groups, strict=False):
        """strict: raise instead of warning when the tuned implementation of
        a subkernel cannot use its matrix-core kernels on these shapes."""
        if isinstance(groups, str):
            groups = mk_decomposition_preset(module, groups)
        self.desc = module
        self.groups = list(groups)
        self.h = mk_module_create(module, self.groups)
        self.info = mk_module_info(self.h)
        self.n = self.info["n_subkernels"]
        limited = [(i, s["family"], s["tuned_limit"]) for i, s in enumerate(self.subkernels())
                   if s["tuned_limit"] != "none"]
        if limited:
            msg = (f"module {module.get('name', '?')}: the tuned implementation runs the simple "
                   "kernels for " + ", ".join(f"subkernel {i} ({f}, limit '{lim}')"
                                              for i, f, lim in limited))
            if strict:
                raise MkError(STATUS.index("MK_E_UNSUPPORTED"), msg)
            warnings.warn(msg, TunedLimitWarning, stacklevel=2)

    def __del__(self):
        h = getattr(self, "h", None)
        if h is not None and _lib is not None:
            _lib.mk_module_destroy(h)
            self.h = None

    def subkernels(self):
        return [mk_subkernel_info(self.h, i) for i in range(self.n)]

    def select(self, i, impl):
        mk_subkernel_select(self.h, i, impl)

    def workspace_size(self):
        return mk_workspace_size(self.h)

    def launches_per_run(self):
        return sum(s["n_launches"] for s in self.subkernels())

    def profile_begin(self, max_launches, only_launch=-1):
        mk_profile_begin(self.h, max_launches, only_launch)

    def profile_end(self, capacity):
        return mk_profile_end(self.h, capacity)

    @staticmethod
    def _ptrs(tensors):
        return [t.data_ptr() for t in tensors]

    def run(self, dev_inputs, out, ws, stream=None, timing=False):
        st = stream.cuda_stream if stream is not None else _current_stream()
        return mk_run(self.h, self._ptrs(dev_inputs), out.data_ptr(),
                      ws.data_ptr() if ws is not None and ws.numel() else None,
                      ws.numel() * ws.element_size() if ws is not None else 0, st,
                      self.n if timing else None)

    def run_noalloc(self, dev_inputs, out, stream=None):
        st = stream.cuda_stream if stream is not None else _current_stream()
        mk_run_noalloc(self.h, self._ptrs(dev_inputs), out.data_ptr(), st)

    def swap(self, dev_inputs, out, ws, reference_impl=IMPL_SIMPLE, tau=0.9, n_runs=5,
             stream=None):
        """Apply the swap policy (mk_swap); returns the per-subkernel times and
        decision."""
        st = stream.cuda_stream if stream is not None else _current_stream()
        n = self.n
        t_sel, t_ref = (ctypes.c_float * n)(), (ctypes.c_float * n)()
        sw, trig = (ctypes.c_int32 * n)(), ctypes.c_int32()
        ptrs = (ctypes.c_void_p * max(1, len(dev_inputs)))(*self._ptrs(dev_inputs))
        _check(load().mk_swap(self.h, ptrs, out.data_ptr(),
                              ws.data_ptr() if ws is not None and ws.numel() else None,
                              ws.numel() * ws.element_size() if ws is not None else 0, st,
                              int(reference_impl), float(tau), int(n_runs), t_sel, t_ref, sw,
                              ctypes.byref(trig)))
        return {"ms_selected": list(t_sel), "ms_reference": list(t_ref),
                "swapped": [int(x) for x in sw], "triggered": bool(trig.value)}

    def verify(self, dev_inputs, out, ws, checks, stream=None):
        st = stream.cuda_stream if stream is not None else _current_stream()
        return mk_verify(self.h, self._ptrs(dev_inputs), out.data_ptr(),
                         ws.data_ptr() if ws is not None and ws.numel() else None,
                         ws.numel() * ws.element_size() if ws is not None else 0, st, checks)


def _current_stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


def device_buffers(module, host_inputs, ws_bytes, device="cuda"):
    """Copy host inputs (numpy storage arrays) to device tensors and allocate the
    output and a workspace.  Returns (inputs, out, ws)."""
    import torch
    bf = module["dtype"] == "bf16"
    dt = torch.bfloat16 if bf else torch.float32
    ins = []
    for a, shape in zip(host_inputs, module["inputs"]):
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16) if bf else
                             np.ascontiguousarray(a, dtype=np.float32))
        if bf:
            t = t.view(torch.bfloat16)
        ins.append(t.reshape(shape).to(device))
    return ins, None, torch.empty(max(1, int(ws_bytes)), dtype=torch.uint8, device=device)


def out_tensor(module, out_shape, device="cuda"):
    """Output buffer filled with NaN, so elements a run leaves unwritten show."""
    import torch
    dt = torch.bfloat16 if module["dtype"] == "bf16" else torch.float32
    return torch.full(out_shape, float("nan"), dtype=dt, device=device)


def to_float64(t):
    """Device or host tensor in the module dtype -> numpy float64 (exact)."""
    import torch
    return t.detach().to("cpu").to(torch.float64).numpy()
