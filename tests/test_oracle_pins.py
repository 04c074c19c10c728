"""Pins of the oracle against facts fixed outside it: closed forms, special
cases, brute force on tiny inputs, and independent library routines (numpy,
scipy, torch CPU in float64).  No value here comes from the HIP path."""
import math

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from oracle import mko

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def f32_inputs(*arrays):
    return [np.ascontiguousarray(a, dtype=np.float32).reshape(-1) for a in arrays]


def module(dtype, inputs, ops):
    return {"dtype": dtype, "inputs": [list(s) for s in inputs], "ops": ops}


def op(kind, ins, ip=(), fp=()):
    return {"kind": kind, "in": list(ins), "ip": list(ip), "fp": list(fp)}


def run1(m, inputs, ideal=True, groups=None):
    g = groups if groups is not None else [0] * len(m["ops"])
    return oracle.run(m, g, inputs, ideal=ideal)


# --------------------------------------------------------------------------- rounding

def test_bf16_rne_bit_patterns():
    # 0x3F808000 = 1 + 2^-8: exact tie between 0x3F80 and 0x3F81 -> even 0x3F80.
    assert oracle.round_bf16(1 + 2 ** -8) == 1.0
    # 0x3F818000 = 1 + 3 * 2^-8: tie between 0x3F81 and 0x3F82 -> even 0x3F82.
    assert oracle.round_bf16(1 + 3 * 2 ** -8) == 1 + 2 * 2 ** -7
    assert oracle.round_bf16(1 + 2 ** -8 + 2 ** -30) == 1 + 2 ** -7   # above the tie
    assert oracle.round_bf16(-(1 + 3 * 2 ** -8)) == -(1 + 2 * 2 ** -7)
    for v in (0.0, math.inf, -math.inf):
        assert oracle.round_bf16(v) == v
    assert math.copysign(1.0, oracle.round_bf16(-0.0)) == -1.0
    assert math.isnan(oracle.round_bf16(math.nan))
    # Largest finite bf16 is (2 - 2^-7) 2^127; the halfway point rounds to inf.
    mx = (2 - 2 ** -7) * 2.0 ** 127
    assert oracle.round_bf16(mx) == mx
    assert oracle.round_bf16(mx * (1 + 2 ** -10)) == mx
    assert oracle.round_bf16((2 - 2 ** -8) * 2.0 ** 127) == math.inf
    # Subnormal quantum 2^-133.
    assert oracle.round_bf16(2.0 ** -133) == 2.0 ** -133
    assert oracle.round_bf16(1.5 * 2.0 ** -133) == 2.0 ** -132
    assert oracle.round_bf16(0.5 * 2.0 ** -133) == 0.0


def test_bf16_rne_matches_torch_on_float32_values():
    rng = np.random.default_rng(1)
    vals = np.concatenate([rng.standard_normal(4000) * 10.0 ** rng.integers(-30, 30, 4000),
                           rng.standard_normal(1000)]).astype(np.float32)
    ref = torch.from_numpy(vals).to(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([oracle.round_bf16(float(v)) for v in vals])
    np.testing.assert_array_equal(got, ref)


def test_f32_rounding_matches_numpy():
    rng = np.random.default_rng(2)
    vals = rng.standard_normal(2000) * 10.0 ** rng.integers(-20, 20, 2000)
    got = np.array([oracle.round_f32(v) for v in vals])
    np.testing.assert_array_equal(got, vals.astype(np.float32).astype(np.float64))


# --------------------------------------------------------------------------- activations

def test_gelu_known_points():
    assert oracle.gelu_erf(1.0) == pytest.approx(0.8413447460685429, abs=1e-15)
    assert oracle.gelu_erf(-1.0) == pytest.approx(-0.15865525393145707, abs=1e-15)
    assert oracle.gelu_tanh(1.0) == pytest.approx(0.8411919906082768, abs=1e-15)
    assert oracle.gelu_tanh(-1.0) == pytest.approx(-0.15880800939172324, abs=1e-15)
    assert oracle.gelu_erf(0.0) == 0.0 and oracle.gelu_tanh(0.0) == 0.0
    # The sigmoid approximation x * sigmoid(1.702 x) (an injected bug in App. D)
    # differs from exact GELU at x = 1 by far more than 1e-3.
    assert abs(1.0 / (1.0 + math.exp(-1.702)) - oracle.gelu_erf(1.0)) > 1e-3
    for x in np.linspace(-6, 6, 61):
        # Both forms are x * (odd-symmetric CDF): GELU(x) - GELU(-x) = x.
        assert oracle.gelu_erf(x) - oracle.gelu_erf(-x) == pytest.approx(x, abs=1e-13)
        assert oracle.gelu_tanh(x) - oracle.gelu_tanh(-x) == pytest.approx(x, abs=1e-13)


def test_gelu_against_libraries():
    xs = np.linspace(-8, 8, 1601)
    got_erf = np.array([oracle.gelu_erf(x) for x in xs])
    np.testing.assert_allclose(got_erf, xs * scipy.special.ndtr(xs), rtol=1e-14, atol=1e-15)
    ref_tanh = torch.nn.functional.gelu(torch.from_numpy(xs), approximate="tanh").numpy()
    got_tanh = np.array([oracle.gelu_tanh(x) for x in xs])
    np.testing.assert_allclose(got_tanh, ref_tanh, rtol=1e-14, atol=1e-15)


def test_elementwise_ops_in_a_module():
    xs = np.linspace(-4, 4, 24).reshape(4, 6)
    r = np.arange(24, dtype=np.float64).reshape(4, 6) / 7
    m = module("f32", [(4, 6), (4, 6)],
               [op("RELU", [0]), op("GELU_ERF", [0]), op("GELU_TANH", [0]),
                op("SCALE", [0], fp=[-0.25]), op("ADD", [0, 1])])
    x32 = xs.astype(np.float32).astype(np.float64)
    r32 = r.astype(np.float32).astype(np.float64)
    out = run1(m, f32_inputs(xs, r))
    np.testing.assert_array_equal(out[0], np.maximum(x32, 0))
    np.testing.assert_allclose(out[1], x32 * scipy.special.ndtr(x32), rtol=1e-14, atol=1e-15)
    np.testing.assert_array_equal(out[3], x32 * -0.25)
    np.testing.assert_array_equal(out[4], x32 + r32)


# --------------------------------------------------------------------------- GEMM

def test_gemm_identity_and_zero():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, 8)).astype(np.float32)
    b = rng.standard_normal(8).astype(np.float32)
    eye = np.eye(8, dtype=np.float32)
    zero = np.zeros((8, 8), dtype=np.float32)
    for layout in (0, 1):
        m = module("f32", [(5, 8), (8, 8), (8,)], [op("GEMM", [0, 1], [layout]),
                                                   op("BIAS", [3, 2])])
        out = run1(m, f32_inputs(x, eye, b), ideal=False)
        np.testing.assert_array_equal(out[0], x.astype(np.float64))
        out = run1(m, f32_inputs(x, zero, b), ideal=False)
        np.testing.assert_array_equal(out[1], np.broadcast_to(b.astype(np.float64), (5, 8)))


def test_gemm_brute_force_integers_both_layouts():
    rng = np.random.default_rng(4)
    A = rng.integers(-9, 10, (3, 7)).astype(np.float64)
    W = rng.integers(-9, 10, (5, 7)).astype(np.float64)     # [N, K]
    expect = np.zeros((3, 5))
    for i in range(3):
        for j in range(5):
            for k in range(7):
                expect[i, j] += A[i, k] * W[j, k]
    m0 = module("f32", [(3, 7), (5, 7)], [op("GEMM", [0, 1], [0])])
    m1 = module("f32", [(3, 7), (7, 5)], [op("GEMM", [0, 1], [1])])
    np.testing.assert_array_equal(run1(m0, f32_inputs(A, W))[0], expect)
    np.testing.assert_array_equal(run1(m1, f32_inputs(A, W.T.copy()))[0], expect)


def test_gemm_against_numpy_batched_rows():
    rng = np.random.default_rng(5)
    A = rng.standard_normal((2, 3, 33)).astype(np.float32)
    W = rng.standard_normal((17, 33)).astype(np.float32)
    m = module("f32", [(2, 3, 33), (17, 33)], [op("GEMM", [0, 1], [0])])
    got = run1(m, f32_inputs(A, W))[0]
    assert got.shape == (2, 3, 17)
    np.testing.assert_allclose(got, A.astype(np.float64) @ W.T.astype(np.float64),
                               rtol=1e-13, atol=1e-13)


# --------------------------------------------------------------------------- row ops

def test_softmax_closed_forms():
    x = np.array([[0.0, math.log(2.0)], [1000.0, 0.0], [3.0, 3.0]])
    m = module("f32", [(3, 2)], [op("SOFTMAX", [0])])
    xin = x.astype(np.float32)
    got = run1(m, f32_inputs(xin))[0]
    ln2 = float(np.float32(math.log(2.0)))
    np.testing.assert_allclose(got[0], [1 / (1 + math.exp(ln2)), math.exp(ln2) / (1 + math.exp(ln2))],
                               rtol=1e-15)
    assert got[0][0] == pytest.approx(1 / 3, abs=1e-7)
    np.testing.assert_array_equal(got[1], [1.0, math.exp(-1000.0)])   # no overflow
    np.testing.assert_array_equal(got[2], [0.5, 0.5])


def test_softmax_invariants_and_scipy():
    rng = np.random.default_rng(6)
    # multiples of 2^-10 below 2^8 in magnitude: adding 64 is exact in fp32
    x = (np.round(rng.standard_normal((7, 129)) * 5 * 1024) / 1024).astype(np.float32)
    m = module("f32", [(7, 129)], [op("SOFTMAX", [0])])
    got = run1(m, f32_inputs(x))[0]
    np.testing.assert_allclose(got.sum(-1), 1.0, atol=1e-14)
    np.testing.assert_allclose(got, scipy.special.softmax(x.astype(np.float64), axis=-1),
                               rtol=1e-13, atol=1e-300)
    shifted = run1(m, f32_inputs(x + np.float32(64.0)))[0]   # exact shift in fp32
    np.testing.assert_allclose(shifted, got, rtol=1e-12)
    const = run1(module("f32", [(2, 10)], [op("SOFTMAX", [0])]),
                 f32_inputs(np.full((2, 10), 3.5)))[0]
    np.testing.assert_array_equal(const, np.full((2, 10), 0.1))


def test_rowsum_and_gap():
    m = module("f32", [(3, 11)], [op("ROWSUM", [0])])
    np.testing.assert_array_equal(run1(m, f32_inputs(np.ones((3, 11))))[0], [11.0] * 3)
    rng = np.random.default_rng(7)
    x = rng.standard_normal((2, 3, 5, 4)).astype(np.float32)
    g = run1(module("f32", [(2, 3, 5, 4)], [op("GAP", [0])]), f32_inputs(x))[0]
    np.testing.assert_allclose(g, x.astype(np.float64).mean(axis=(2, 3)), rtol=1e-14)
    c = np.full((1, 2, 3, 3), 2.5, dtype=np.float32)
    np.testing.assert_array_equal(
        run1(module("f32", [(1, 2, 3, 3)], [op("GAP", [0])]), f32_inputs(c))[0], [[2.5, 2.5]])


def test_global_max_and_lp_pool():
    """GMP and LPPOOL (pooling variants of Sec. 4): hand values, the torch CPU
    pooling routines in float64, and p = 1 / p = 2 special cases."""
    x = np.array([[[[1.0, -2.0], [5.0, 0.5]], [[-3.0, -1.0], [-7.0, -2.0]]]])   # [1,2,2,2]
    m = module("f32", [x.shape], [op("GMP", [0])])
    assert run1(m, f32_inputs(x))[-1].tolist() == [[5.0, -1.0]]
    m = module("f32", [x.shape], [op("LPPOOL", [0], fp=[2.0])])
    np.testing.assert_allclose(run1(m, f32_inputs(x))[-1],
                               [[math.sqrt(1 + 4 + 25 + 0.25), math.sqrt(9 + 1 + 49 + 4)]],
                               rtol=1e-15)
    # odd p keeps the sign of the sum: channel 1 sums to -(27 + 1 + 343 + 8)
    m = module("f32", [x.shape], [op("LPPOOL", [0], fp=[3.0])])
    got = run1(m, f32_inputs(x))[-1]
    np.testing.assert_allclose(got[0, 1], -(379.0 ** (1 / 3)), rtol=1e-14)
    np.testing.assert_allclose(got[0, 0], (1 - 8 + 125 + 0.125) ** (1 / 3), rtol=1e-14)
    rng = np.random.default_rng(5)
    x = rng.standard_normal((3, 4, 6, 5)).astype(np.float32)
    xt = torch.from_numpy(x.astype(np.float64))
    m = module("f32", [x.shape], [op("GMP", [0])])
    ref = torch.nn.functional.max_pool2d(xt, (6, 5)).reshape(3, 4).numpy()
    np.testing.assert_array_equal(run1(m, f32_inputs(x))[-1], ref)
    xr = np.maximum(x, 0)
    for p in (1.0, 2.0, 3.0):
        m = module("f32", [x.shape], [op("LPPOOL", [0], fp=[p])])
        ref = torch.nn.functional.lp_pool2d(torch.from_numpy(xr.astype(np.float64)), p,
                                            (6, 5)).reshape(3, 4).numpy()
        np.testing.assert_allclose(run1(m, f32_inputs(xr))[-1], ref, rtol=1e-12)
    m = module("f32", [x.shape], [op("LPPOOL", [0], fp=[1.0])])
    np.testing.assert_allclose(run1(m, f32_inputs(xr))[-1], xr.astype(np.float64).sum((2, 3)),
                               rtol=1e-12)
    with pytest.raises(ValueError):
        oracle.plan(module("f32", [x.shape], [op("LPPOOL", [0], fp=[0.0])]), [0])


def test_layernorm_closed_form():
    eps = 1e-5
    m = module("f32", [(2, 4), (4,), (4,)], [op("LAYERNORM", [0, 1, 2], fp=[eps])])
    x = np.array([[1, 2, 3, 4], [7, 7, 7, 7]], dtype=np.float32)
    g = np.ones(4, np.float32)
    b = np.array([0.5, -1, 2, 0], np.float32)
    got = run1(m, f32_inputs(x, g, b))[0]
    np.testing.assert_allclose(got[0], (np.array([1, 2, 3, 4]) - 2.5) / math.sqrt(1.25 + eps) + b,
                               rtol=1e-15)
    np.testing.assert_array_equal(got[1], b.astype(np.float64))   # constant row -> beta


def test_layernorm_moments_and_torch():
    eps = 1e-5
    rng = np.random.default_rng(8)
    x = (rng.standard_normal((6, 257)) * 3 + 1).astype(np.float32)
    g = rng.standard_normal(257).astype(np.float32)
    b = rng.standard_normal(257).astype(np.float32)
    m = module("f32", [(6, 257), (257,), (257,)], [op("LAYERNORM", [0, 1, 2], fp=[eps])])
    plain = run1(m, f32_inputs(x, np.ones(257), np.zeros(257)))[0]
    var = x.astype(np.float64).var(axis=-1)
    np.testing.assert_allclose(plain.mean(-1), 0.0, atol=1e-14)
    np.testing.assert_allclose(plain.var(-1), var / (var + eps), rtol=1e-12)
    got = run1(m, f32_inputs(x, g, b))[0]
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x.astype(np.float64)), (257,),
                                         torch.from_numpy(g.astype(np.float64)),
                                         torch.from_numpy(b.astype(np.float64)), eps).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------- conv

def conv_module(N, C, H, W, K, R, stride=1, pad=1):
    return module("f32", [(N, C, H, W), (K, C, R, R)], [op("CONV2D", [0, 1], [stride, pad])])


def test_conv_center_tap_identity_and_ones():
    rng = np.random.default_rng(9)
    x = rng.standard_normal((1, 2, 4, 5)).astype(np.float32)
    w = np.zeros((2, 2, 3, 3), np.float32)
    w[0, 0, 1, 1] = 1.0
    w[1, 1, 1, 1] = 1.0
    np.testing.assert_array_equal(run1(conv_module(1, 2, 4, 5, 2, 3), f32_inputs(x, w))[0],
                                  x.astype(np.float64))
    C = 3
    ones = run1(conv_module(1, C, 5, 5, 1, 3), f32_inputs(np.ones((1, C, 5, 5)),
                                                          np.ones((1, C, 3, 3))))[0][0, 0]
    assert ones[2, 2] == 9 * C and ones[0, 2] == 6 * C and ones[0, 0] == 4 * C
    assert ones[4, 4] == 4 * C and ones[2, 4] == 6 * C


def test_conv_brute_force_im2col_and_torch():
    rng = np.random.default_rng(10)
    x = rng.integers(-3, 4, (1, 2, 4, 4)).astype(np.float32)
    w = rng.integers(-3, 4, (3, 2, 3, 3)).astype(np.float32)
    got = run1(conv_module(1, 2, 4, 4, 3, 3), f32_inputs(x, w))[0]
    xp = np.pad(x.astype(np.float64), ((0, 0), (0, 0), (1, 1), (1, 1)))
    cols = np.array([[xp[0, c, p + r, q + s] for c in range(2) for r in range(3) for s in range(3)]
                     for p in range(4) for q in range(4)])             # [PQ, CRS]
    ref = (w.reshape(3, -1).astype(np.float64) @ cols.T).reshape(1, 3, 4, 4)
    np.testing.assert_array_equal(got, ref)
    x2 = rng.standard_normal((2, 3, 7, 6)).astype(np.float32)
    w2 = rng.standard_normal((4, 3, 3, 3)).astype(np.float32)
    for stride, pad in ((1, 1), (2, 1), (1, 0)):
        got = run1(conv_module(2, 3, 7, 6, 4, 3, stride, pad), f32_inputs(x2, w2))[0]
        ref = torch.nn.functional.conv2d(torch.from_numpy(x2.astype(np.float64)),
                                         torch.from_numpy(w2.astype(np.float64)),
                                         stride=stride, padding=pad).numpy()
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------- attention

def attn_module(B, S, H, dh, causal=True):
    ops = [op("QK", [1], [B, H, dh, S], [1 / math.sqrt(dh)])]
    v = 2
    if causal:
        ops.append(op("CAUSAL_MASK", [v]))
        v += 1
    ops.append(op("SOFTMAX", [v]))
    ops.append(op("PV", [v + 1, 1], [B, H, dh, S]))
    # input 0 is an unused placeholder so that qkv is value 1
    return module("f32", [(1,), (B * S, 3 * H * dh)], ops)


def test_attention_first_row_and_prefix_mean():
    B, S, H, dh = 2, 6, 2, 4
    rng = np.random.default_rng(11)
    qkv = rng.standard_normal((B * S, 3 * H * dh)).astype(np.float32)
    out = run1(attn_module(B, S, H, dh), f32_inputs(np.zeros(1), qkv))[-1]
    v = qkv.astype(np.float64)[:, 2 * H * dh:].reshape(B, S, H, dh)
    np.testing.assert_array_equal(out[:, 0, :].reshape(B, H, dh), v[:, 0])   # row 0 -> v_0
    # Identical keys: every kept score is equal, so o_i is the mean of v_0..v_i.
    same = qkv.copy()
    same[:, H * dh:2 * H * dh] = 0.37
    out = run1(attn_module(B, S, H, dh), f32_inputs(np.zeros(1), same))[-1]
    pref = np.cumsum(v, axis=1) / np.arange(1, S + 1)[None, :, None, None]
    np.testing.assert_allclose(out.reshape(B, S, H, dh), pref, rtol=1e-13, atol=1e-14)


def test_causal_mask_keeps_diagonal():
    m = module("f32", [(1, 1, 3, 3)], [op("CAUSAL_MASK", [0])])
    x = np.arange(9, dtype=np.float32).reshape(1, 1, 3, 3)
    got = run1(m, f32_inputs(x))[0][0, 0]
    ninf = -math.inf
    np.testing.assert_array_equal(got, [[0, ninf, ninf], [3, 4, ninf], [6, 7, 8]])


def test_attention_against_torch_sdpa():
    B, S, H, dh = 2, 9, 3, 8
    rng = np.random.default_rng(12)
    qkv = rng.standard_normal((B * S, 3 * H * dh)).astype(np.float32)
    t = torch.from_numpy(qkv.astype(np.float64)).reshape(B, S, 3, H, dh)
    q, k, v = (t[:, :, i].permute(0, 2, 1, 3).contiguous() for i in range(3))
    for causal in (True, False):
        got = run1(attn_module(B, S, H, dh, causal), f32_inputs(np.zeros(1), qkv))[-1]
        ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=causal)
        ref = ref.permute(0, 2, 1, 3).reshape(B, S, H * dh).numpy()
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)


# --------------------------------------------------------------------------- modules

def mlp(M, D, F):
    return module("f32", [(M, D), (D,), (D,), (F, D), (D, F)],
                  [op("LAYERNORM", [0, 1, 2], fp=[1e-5]), op("GEMM", [5, 3], [0]),
                   op("GELU_ERF", [6]), op("GEMM", [7, 4], [0]), op("ADD", [8, 0])])


def test_mlp_zero_weights_give_identity():
    rng = np.random.default_rng(13)
    x = rng.standard_normal((4, 8)).astype(np.float32)
    ones, zeros = np.ones(8), np.zeros(8)
    W1 = rng.standard_normal((16, 8)).astype(np.float32)
    for w1, w2 in ((W1, np.zeros((8, 16))), (np.zeros((16, 8)), rng.standard_normal((8, 16)))):
        out = oracle.run(mlp(4, 8, 16), [0, 0, 0, 1, 1], f32_inputs(x, ones, zeros, w1, w2))[-1]
        np.testing.assert_array_equal(out, x.astype(np.float64))


def test_mlp_against_torch():
    rng = np.random.default_rng(14)
    M, D, F = 5, 16, 24
    arrs = [rng.standard_normal(s).astype(np.float32) * sc
            for s, sc in (((M, D), 1), ((D,), 1), ((D,), 1), ((F, D), 0.2), ((D, F), 0.2))]
    got = oracle.run(mlp(M, D, F), [0, 1, 2, 3, 3], f32_inputs(*arrs), ideal=True)[-1]
    x, g, b, w1, w2 = (torch.from_numpy(a.astype(np.float64)) for a in arrs)
    ref = x + torch.nn.functional.gelu(
        torch.nn.functional.layer_norm(x, (D,), g, b, 1e-5) @ w1.T) @ w2.T
    np.testing.assert_allclose(got, ref.numpy(), rtol=1e-12, atol=1e-12)


def test_rounding_model_boundaries():
    """bf16 module: a materialised group output is the bf16 rounding of the
    unrounded value, and a group-internal value is not rounded."""
    rng = np.random.default_rng(15)
    m = mlp(3, 8, 12)
    m["dtype"] = "bf16"
    xs = [rng.standard_normal(s) for s in ((3, 8), (8,), (8,), (12, 8), (8, 12))]
    bits = [torch.from_numpy(a.astype(np.float32)).to(torch.bfloat16).view(torch.int16)
            .numpy().view(np.uint16).reshape(-1) for a in xs]
    split = oracle.run(m, [0, 1, 2, 3, 3], bits)
    ideal = oracle.run(m, [0, 1, 2, 3, 3], bits, ideal=True)
    rb = np.vectorize(oracle.round_bf16)
    np.testing.assert_array_equal(split[0], rb(ideal[0]))          # LN output materialised
    fused = oracle.run(m, [0, 0, 0, 1, 1], bits)
    np.testing.assert_array_equal(fused[0], rb(ideal[0]))          # LN prologue operand
    np.testing.assert_array_equal(fused[2], rb(fused[2]))          # group output
    assert not np.array_equal(fused[1], rb(fused[1]))              # GEMM inside a group: fp64


# --------------------------------------------------------------------------- bookkeeping

def test_plan_hand_computed_integers():
    conv = {"dtype": "bf16", "inputs": [[64, 128, 56, 56], [256, 128, 3, 3], [256]],
            "ops": [op("CONV2D", [0, 1], [1, 1]), op("BIAS_CHANNEL", [3, 2]), op("RELU", [4]),
                    op("GAP", [5])]}
    p = oracle.plan(conv, [0, 0, 1, 2])
    assert p["flops"] == 2 * 200704 * 256 * 1152 == 118380036096
    y = 64 * 256 * 56 * 56 * 2
    assert [g["ws_offset"] for g in p["groups"]] == [0, y, -1]
    assert p["ws_intermediate_bytes"] == 2 * y
    assert p["groups"][0]["alg_bytes"] == (64 * 128 * 56 * 56 + 256 * 128 * 9 + 256) * 2 + y
    assert p["groups"][2]["out_shape"] == (64, 256)
    attn = attn_module(1, 2048, 16, 128)
    q = oracle.plan(attn, [0, 1, 2, 3])
    causal = 2 * 16 * 128 * 2048 * 2049 // 2
    assert q["groups"][0]["flops"] == causal and q["groups"][3]["flops"] == causal
    assert q["flops"] == 2 * causal
    p = oracle.plan(attn_module(1, 2048, 16, 128, causal=False), [0, 1, 2])
    assert p["flops"] == 2 * 2 * 16 * 128 * 2048 * 2048


def test_plan_materialisation_rule():
    m = mlp(4, 8, 16)
    assert oracle.plan(m, [0, 1, 1, 2, 2])["groups"][1]["op_begin"] == 1
    oracle.plan(m, [0, 0, 1, 1, 1])
    # Non-contiguous / not starting at 0 groupings are rejected.
    for bad in ([1, 1, 1, 1, 1], [0, 2, 2, 2, 2], [0, 1, 0, 1, 1]):
        with pytest.raises(ValueError):
            oracle.plan(m, bad)
    # Transformer: h (op 7) feeds op 12; a group that hides op 7 inside is invalid.
    x = {"dtype": "bf16", "inputs": [[2, 4], [4, 4]],
         "ops": [op("GEMM", [0, 1], [0]), op("RELU", [2]), op("ADD", [3, 2])]}
    with pytest.raises(ValueError):
        oracle.plan(x, [0, 0, 1])          # op 0's output read by op 2 outside its group
    oracle.plan(x, [0, 1, 2])
    oracle.plan(x, [0, 0, 0])


# --------------------------------------------------------------------------- channel bias

def check_bias_channel():
    """Per-channel bias of an NCHW tensor: on a zero input every position of
    channel c holds b[c] (a non-square image with three distinct biases, so a
    bias indexed by position or by the flat index modulo C differs), and the
    conv + channel bias chain equals torch's conv2d with its own bias argument
    in float64, grouped with the conv and split from it."""
    N, C, H, W = 2, 3, 2, 5
    b = np.array([1.0, 10.0, 100.0])
    m = module("f32", [(N, C, H, W), (C,)], [op("BIAS_CHANNEL", [0, 1])])
    got = run1(m, f32_inputs(np.zeros((N, C, H, W)), b))[0]
    for c in range(C):
        assert (got[:, c] == b[c]).all(), (c, got[:, c])
    rng = np.random.default_rng(21)
    n, ci, h, w_, k = 2, 3, 5, 7, 4
    x = rng.standard_normal((n, ci, h, w_)).astype(np.float32)
    wt = rng.standard_normal((k, ci, 3, 3)).astype(np.float32)
    bias = (rng.standard_normal(k) * 3).astype(np.float32)
    conv = module("f32", [(n, ci, h, w_), (k, ci, 3, 3), (k,)],
                  [op("CONV2D", [0, 1], [1, 1]), op("BIAS_CHANNEL", [3, 2])])
    ref = torch.nn.functional.conv2d(torch.from_numpy(x.astype(np.float64)),
                                     torch.from_numpy(wt.astype(np.float64)),
                                     torch.from_numpy(bias.astype(np.float64)),
                                     stride=1, padding=1).numpy()
    for groups in ([0, 0], [0, 1]):
        y = oracle.run(conv, groups, f32_inputs(x, wt, bias), ideal=True)[-1]
        np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_bias_channel_hand_values_and_torch_conv_bias():
    check_bias_channel()


# --------------------------------------------------------------------------- composition

def tiny_modules(dtype):
    from paper_2607_20501_amd import workloads
    return [
        workloads.linear_relu_rowsum(M=5, K=7, N=6, dtype=dtype),
        workloads.gemm_gelu_softmax(M=4, K=6, N=9, dtype=dtype),
        workloads.conv_relu_gap(N=2, C=3, H=5, W=4, K=4, dtype=dtype),
        workloads.mlp_block(M=3, D=8, F=12, dtype=dtype),
        workloads.transformer_layer(B=2, S=5, D=8, H=2, F=12, dtype=dtype),
    ]


def all_groupings(n):
    for cuts in range(1 << (n - 1)):
        g = [0]
        for i in range(n - 1):
            g.append(g[-1] + ((cuts >> i) & 1))
        yield g


def check_composition(dtype):
    """Sec. 3 / App. H.1: a top-level module that chains subproblem kernels
    computes the module itself, whatever the grouping.  For every contiguous
    grouping the oracle accepts (brute force over all 2^(n-1)), the output
    equals the all-split grouping's within the dtype tolerance (plus the
    row-scaled softmax check), and without the rounding model the output does
    not depend on the grouping at all."""
    from paper_2607_20501_amd import inputs
    rtol, atol = {"f32": (1e-4, 1e-5), "bf16": (2e-2, 2e-2)}[dtype]
    for m in tiny_modules(dtype):
        n = len(m["ops"])
        host = inputs.make_inputs(m, 3)
        split = list(range(n))
        ref = oracle.run(m, split, host, keep={n - 1})[-1]
        ideal = oracle.run(m, split, host, ideal=True, keep={n - 1})[-1]
        atol_out = atol / ref.shape[-1] if m["ops"][-1]["kind"] == "SOFTMAX" else atol
        accepted = 0
        for g in all_groupings(n):
            try:
                oracle.plan(m, g)
            except ValueError:
                continue
            accepted += 1
            got = oracle.run(m, g, host, keep={n - 1})[-1]
            np.testing.assert_allclose(got, ref, rtol=rtol, atol=atol_out,
                                       err_msg=f"{m['name']} grouping {g}")
            np.testing.assert_array_equal(
                oracle.run(m, g, host, ideal=True, keep={n - 1})[-1], ideal)
        assert accepted >= n, (m["name"], accepted)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_every_grouping_agrees_with_all_split(dtype):
    check_composition(dtype)


# --------------------------------------------------------------------------- planted mistakes

def planted(tmp_path, old, new):
    """A copy of the oracle with one plausible mistake planted in its source
    (CPU only); returns the context that evaluates with it."""
    src = open(mko.SOURCE).read()
    assert src.count(old) == 1, old
    path = tmp_path / "mko_planted.c"
    path.write_text(src.replace(old, new))
    so = str(tmp_path / "libmko_planted.so")
    mko.build(str(path), so)
    return oracle.library(so)


def test_bias_channel_pin_rejects_flat_index_bias(tmp_path):
    with planted(tmp_path, "b[(k / hw) % C]", "b[k % C]"):
        with pytest.raises(AssertionError):
            check_bias_channel()


def test_bias_channel_pin_rejects_position_index_bias(tmp_path):
    with planted(tmp_path, "b[(k / hw) % C]", "b[(k % hw) % C]"):
        with pytest.raises(AssertionError):
            check_bias_channel()


def test_composition_pin_rejects_rounding_to_the_wrong_dtype(tmp_path):
    # Group outputs of an fp32 module rounded to bfloat16: the result then
    # depends on where the groups end.
    with planted(tmp_path, "if (is_last || ln_prologue) round_to(y, n, d->dtype);",
                 "if (is_last || ln_prologue) round_to(y, n, MKO_BF16);"):
        with pytest.raises(AssertionError):
            check_composition("f32")

