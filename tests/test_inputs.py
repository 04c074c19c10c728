"""The seeded input generator: determinism, slicing, distribution moments and
the float32 -> bfloat16 rounding of its output."""
import numpy as np
import torch

from paper_2607_20501_amd import inputs, workloads


def test_deterministic_and_sliceable():
    a = inputs.fill(7, 3, inputs.NORMAL, 0.0, 1.0, "f32", 10000)
    b = inputs.fill(7, 3, inputs.NORMAL, 0.0, 1.0, "f32", 10000)
    np.testing.assert_array_equal(a, b)
    part = inputs.fill(7, 3, inputs.NORMAL, 0.0, 1.0, "f32", 500, first=1234)
    np.testing.assert_array_equal(part, a[1234:1734])
    c = inputs.fill(8, 3, inputs.NORMAL, 0.0, 1.0, "f32", 10000)
    d = inputs.fill(7, 4, inputs.NORMAL, 0.0, 1.0, "f32", 10000)
    assert not np.array_equal(a, c) and not np.array_equal(a, d)


def test_moments_and_bounds():
    n = 1_000_000
    x = inputs.fill(0, 0, inputs.NORMAL, 0.0, 0.02, "f32", n).astype(np.float64)
    assert abs(x.mean()) < 3 * 0.02 / np.sqrt(n)
    # std of the sample std is about sigma / sqrt(2n)
    assert abs(x.std() - 0.02) < 3 * 0.02 / np.sqrt(2 * n)
    u = inputs.fill(0, 1, inputs.UNIFORM, -0.1, 0.1, "f32", n).astype(np.float64)
    assert u.min() >= -0.1 and u.max() <= 0.1
    assert abs(u.mean()) < 3 * (0.2 / np.sqrt(12)) / np.sqrt(n)
    one = inputs.fill(0, 2, inputs.UNIFORM, 1.0, 1.0, "bf16", 100)
    assert (one == 0x3F80).all()


def test_bf16_output_is_rne_of_f32_output():
    f = inputs.fill(3, 5, inputs.NORMAL, 0.0, 3.0, "f32", 100000)
    b = inputs.fill(3, 5, inputs.NORMAL, 0.0, 3.0, "bf16", 100000)
    ref = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(b, ref)


def test_make_inputs_shapes():
    m = workloads.linear_relu_rowsum()
    xs = inputs.make_inputs(m, 0)
    assert [a.size for a in xs] == [128 * 256, 256 * 256, 256]
    assert all(a.dtype == np.float32 for a in xs)


def test_library_mk_gen_fill_gives_the_generator_bytes():
    """libmk's mk_gen_fill is the same generator the tests feed to the oracle."""
    from paper_2607_20501_amd import mk
    for dtype in ("f32", "bf16"):
        for dist, p0, p1 in ((inputs.NORMAL, 0.0, 0.02), (inputs.UNIFORM, -0.1, 0.1)):
            a = mk.mk_gen_fill(5, 2, dist, p0, p1, dtype, 4097)
            b = inputs.fill(5, 2, dist, p0, p1, dtype, 4097)
            np.testing.assert_array_equal(a, b)
    assert mk.mk_gen_fill(0, 0, inputs.NORMAL, 0.0, 1.0, "f32", 0).size == 0
    import pytest
    with pytest.raises(mk.MkError) as e:
        mk.mk_gen_fill(0, 0, 7, 0.0, 1.0, "f32", 4)
    assert e.value.status == 1
