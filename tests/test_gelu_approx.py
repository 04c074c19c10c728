"""The GEMM epilogue's GELU (erf form) for bf16 results evaluates the normal
CDF in logistic form, Phi(x) ~= sigmoid(x (c0 + c1 x^2 + c2 x^4)) with x^2
capped at 49.  Its constants are read from the device header and the form is
evaluated in fp32 (exp2, reciprocal) against x Phi(x) from scipy in fp64: the
stated bound of 2.6e-5 must hold everywhere, and the form must keep GELU's
limits and the symmetry Phi(-x) = 1 - Phi(x)."""
import pathlib
import re

import numpy as np
from scipy.special import ndtr

HDR = pathlib.Path(__file__).resolve().parents[1] / "paper_2607_20501_amd" / "csrc" / "dev.hpp"


def _constants():
    src = HDR.read_text()
    body = src[src.index("float gelu_erf_bf16out(float x)"):]
    body = body[:body.index("}")]
    cap = float(re.search(r"fminf\(x \* x, ([0-9.]+)f\)", body).group(1))
    k2, k1, k0 = (float(v) for v in re.search(
        r"fmaf\(fmaf\(([-0-9.e]+)f, x2, ([-0-9.e]+)f\), x2, ([-0-9.e]+)f\)", body).groups())
    return cap, np.float32(k0), np.float32(k1), np.float32(k2)


def _gelu_fp32(x):
    cap, k0, k1, k2 = _constants()
    x = x.astype(np.float32)
    with np.errstate(over="ignore"):   # x * x may overflow to inf; the cap takes it
        x2 = np.minimum(x * x, np.float32(cap))
        p = (k2 * x2 + k1) * x2 + k0
        e = np.exp2(x * p).astype(np.float32)
        return x * (np.float32(1) / (np.float32(1) + e))


def test_bound_everywhere():
    x = np.concatenate([np.linspace(-12, 12, 480001), np.linspace(12, 1e4, 10001),
                        -np.linspace(12, 1e4, 10001)])
    err = np.abs(_gelu_fp32(x).astype(np.float64) - x.astype(np.float32) * ndtr(x.astype(np.float32)))
    assert err.max() <= 2.6e-5, err.max()


def test_limits_and_symmetry():
    big = np.array([30.0, 1e3, 3e38], dtype=np.float32)
    assert np.array_equal(_gelu_fp32(big), big)
    assert np.all(np.abs(_gelu_fp32(-big)) <= 1e-6)
    x = np.linspace(0, 8, 8001).astype(np.float32)
    s = _gelu_fp32(x)[1:] / x[1:] + _gelu_fp32(-x)[1:] / (-x[1:])
    assert np.max(np.abs(s - 1)) <= 2e-7
