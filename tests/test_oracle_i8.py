"""Pins for the oracle's integer-activation variant (Eq. 1 with the input replaced by
s * q, q int8 codes), all on the CPU.

The activation codes are pinned to hand-worked values at every rounding and clamping
boundary (including a case where rounding the product to fp32 first changes the code)
and to numpy's fp32 arithmetic.  The exact integer sums are pinned to torch's fp64 CPU
conv2d on the same integer tensors (exact: every partial sum is far below 2^53), to numpy
integer matmul for 1x1 layers and to a hand-worked layer; the scaled output is tied to the
fp64 two-bit forward pass of the dequantised input (Eq. 1) within fp32 rounding.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth

GEOMS = [
    # n, h, w, c, k, r, s, stride, pad
    (2, 7, 6, 16, 3, 5, 5, 1, 2),
    (1, 9, 9, 32, 5, 3, 3, 2, 1),
    (2, 8, 5, 4, 6, 3, 3, 1, 0),
    (1, 11, 10, 2, 4, 7, 7, 2, 3),
    (3, 5, 5, 48, 7, 1, 1, 1, 0),
    (1, 4, 4, 16, 2, 4, 4, 1, 0),
    (2, 6, 6, 3, 4, 3, 2, 3, 2),
]


def test_act_codes_hand_values():
    # inv = 1: the codes are the inputs rounded half to even and limited to [-127, 127]
    x = np.array([0.0, -0.0, 0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 0.49999997, 126.5, 127.49998, 127.5,
                  1e9, -1e9, np.inf, -np.inf, np.nan, 3.0], np.float32)
    want = [0, 0, 0, 2, 2, 0, -2, -2, 0, 126, 127, 127, 127, -127, 127, -127, 0, 3]
    assert oracle.quantize_act_i8(x, 1.0).tolist() == want


def test_act_codes_round_the_product_to_fp32_first():
    # 25 * fp32(0.1) = 2.50000003725... exactly, which would round to 3; rounded to fp32
    # the product is 2.5, a tie, so the code is 2
    inv = np.float32(0.1)
    exact = Fraction(25) * Fraction(float(inv))
    assert exact > Fraction(5, 2)
    assert float(np.float32(25) * inv) == 2.5
    assert oracle.quantize_act_i8(np.float32([25.0]), inv).tolist() == [2]
    # 35 * fp32(0.1) rounds to 3.5: a tie, to the even 4
    assert oracle.quantize_act_i8(np.float32([35.0]), inv).tolist() == [4]


def test_act_codes_match_numpy_fp32():
    x = synth.normal(0, "i8-act", (20000,), 3.0).astype(np.float32)
    x[::97] = np.float32(0.5) * np.arange(x[::97].size, dtype=np.float32)  # many exact ties
    inv = np.float32(127.0) / np.float32(np.abs(x).max())
    v = x * inv
    want = np.clip(np.rint(v), -127, 127).astype(np.int8)
    got = oracle.quantize_act_i8(x, inv)
    assert np.array_equal(got, want)
    assert got.min() >= -127 and got.max() <= 127


def _int_problem(g, name):
    n, h, w, c, k, r, s, st, pd = g
    desc = oracle.ConvDesc(n, h, w, c, k, r, s, st, pd)
    rng = synth.rng(0, name)
    xq = rng.integers(-127, 128, size=(n, h, w, c)).astype(np.int8)
    codes = rng.choice(np.array([-2, -1, 1, 2], np.int8), size=(k, r, s, c))
    alpha = (rng.random(k).astype(np.float32) + np.float32(0.25)).astype(np.float32)
    return desc, xq, codes, alpha


@pytest.mark.parametrize("g", GEOMS)
def test_i8_sums_equal_torch_conv(g):
    desc, xq, codes, alpha = _int_problem(g, "i8-sum%s" % (g,))
    _, acc = oracle.conv_fwd_i8(desc, xq, codes, alpha, 0.5)
    xt = torch.from_numpy(xq.astype(np.float64)).permute(0, 3, 1, 2)
    wt = torch.from_numpy(codes.astype(np.float64)).permute(0, 3, 1, 2)
    ref = F.conv2d(xt, wt, stride=(desc.stride_h, desc.stride_w), padding=(desc.pad_h, desc.pad_w))
    ref = ref.permute(0, 2, 3, 1).numpy()
    assert np.array_equal(acc.astype(np.float64), ref)


def test_i8_one_by_one_is_integer_matmul():
    desc, xq, codes, alpha = _int_problem((3, 4, 5, 40, 9, 1, 1, 1, 0), "i8-mm")
    _, acc = oracle.conv_fwd_i8(desc, xq, codes, alpha, 1.0)
    ref = xq.reshape(-1, 40).astype(np.int64) @ codes.reshape(9, 40).astype(np.int64).T
    assert np.array_equal(acc.reshape(-1, 9), ref)


def test_i8_hand_worked_layer():
    # one pixel, two channels: q = (3, -5), W~ = (2, -1): sum = 6 + 5 = 11;
    # alpha = 0.5, s = 0.25: y = 11 * 0.125 = 1.375 (exact); a second filter (-2, -1) gives
    # -6 + 5 = -1 -> -0.125, which ReLU maps to 0
    desc = oracle.ConvDesc(1, 1, 1, 2, 2, 1, 1)
    xq = np.array([3, -5], np.int8)
    codes = np.array([[2, -1], [-2, -1]], np.int8)
    alpha = np.float32([0.5, 0.5])
    y, acc = oracle.conv_fwd_i8(desc, xq, codes, alpha, 0.25)
    assert acc.ravel().tolist() == [11, -1]
    assert y.ravel().tolist() == [1.375, -0.125]
    y, _ = oracle.conv_fwd_i8(desc, xq, codes, alpha, 0.25, relu=True)
    assert y.ravel().tolist() == [1.375, 0.0]


@pytest.mark.parametrize("g", GEOMS[:4])
def test_i8_output_is_eq1_on_the_dequantised_input(g):
    """y equals the fp64 two-bit forward pass of x = s * q (Eq. 1) within the two fp32
    roundings of the scale and the product."""
    desc, xq, codes, alpha = _int_problem(g, "i8-eq1%s" % (g,))
    s = np.float32(0.0371)
    y, _ = oracle.conv_fwd_i8(desc, xq, codes, alpha, s)
    ref = oracle.conv_fwd(desc, xq.astype(np.float64) * float(s), codes.reshape(desc.k, -1),
                          alpha.astype(np.float64))
    err = np.abs(y.astype(np.float64) - ref)
    assert np.all(err <= 2.5 * 2.0 ** -24 * np.abs(ref) + 1e-30)
    assert np.abs(ref).max() > 0


def test_i8_relu_only_clears_negatives():
    desc, xq, codes, alpha = _int_problem((2, 6, 6, 16, 5, 3, 3, 1, 1), "i8-relu")
    y, _ = oracle.conv_fwd_i8(desc, xq, codes, alpha, 0.01)
    yr, _ = oracle.conv_fwd_i8(desc, xq, codes, alpha, 0.01, relu=True)
    assert np.array_equal(yr, np.where(y > 0, y, 0.0).astype(np.float32))
    assert (y < 0).any() and (y > 0).any()


@pytest.mark.parametrize("relu", [False, True])
def test_i8_sampled_equals_full(relu):
    desc, xq, codes, alpha = _int_problem((2, 9, 7, 32, 11, 3, 3, 2, 1), "i8-sampled")
    y, _ = oracle.conv_fwd_i8(desc, xq, codes, alpha, 0.02, relu=relu)
    idx = synth.sample_indices(0, "i8-sampled-idx", y.size, 300)
    ys = oracle.conv_fwd_i8_sampled(desc, xq, codes, alpha, 0.02, idx, relu=relu)
    assert np.array_equal(ys, y.ravel()[idx])
