"""Pins for the oracle's fp8-activation variant (Eq. 1 with the input replaced by s * f,
f an E4M3 value), all on the CPU.

The E4M3 decode is pinned to torch's float8_e4m3fn on all 256 codes; the encoder to torch's
conversion (nearest, ties to even) on every exact value, every midpoint between neighbours
and random fp32 values in the range where neither saturates, and to hand-worked values for
saturation, NaN and signed zero.  The forward pass is pinned to torch's fp64 CPU conv2d on
the dequantised activations and the two-bit filter values (exact: every product is a
multiple of 2^-9 below 2^10, so the sums are exact in fp64), to numpy matmul for 1x1 layers
and to the closed form of an all-ones input.
"""
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
    (3, 5, 5, 48, 7, 1, 1, 1, 0),
    (2, 6, 6, 3, 4, 3, 2, 3, 2),
]


def torch_codes(v: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.asarray(v, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_decode_matches_torch_e4m3fn():
    codes = np.arange(256, dtype=np.uint8)
    got = oracle.fp8_value(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).double().numpy()
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok])
    assert np.array_equal(np.signbit(got[ok]), np.signbit(ref[ok]))
    # hand values: smallest subnormal, smallest normal, one, largest finite
    assert got[0x01] == 2.0 ** -9 and got[0x08] == 2.0 ** -6 and got[0x38] == 1.0 and got[0x7E] == 448.0


def test_encode_matches_torch_on_exact_values_and_midpoints():
    vals = oracle.fp8_value(np.arange(0x7F, dtype=np.uint8))  # every finite non-negative value
    mids = (vals[:-1] + vals[1:]) / 2                          # exact in fp32
    probes = np.concatenate([vals, mids, np.nextafter(mids.astype(np.float32), 0),
                             np.nextafter(mids.astype(np.float32), np.float32(1000))]).astype(np.float32)
    probes = np.concatenate([probes, -probes])
    probes = probes[np.abs(probes) <= 464.0]
    got = np.array([oracle.fp8_encode_one(v) for v in probes], np.uint8)
    assert np.array_equal(got, torch_codes(probes))


def test_encode_matches_torch_on_random_values():
    rng = np.random.default_rng(1701)
    v = np.concatenate([rng.normal(0, 1, 3000), rng.normal(0, 100, 3000), rng.normal(0, 0.01, 3000),
                        rng.uniform(-464, 464, 3000)]).astype(np.float32)
    got = oracle.quantize_act_fp8(v, 1.0)
    assert np.array_equal(got, torch_codes(v))


def test_encode_saturation_nan_and_signed_zero():
    x = np.array([448.0, 449.0, 464.0, 465.0, 1e30, np.inf, -449.0, -np.inf, np.nan, -0.0, 0.0,
                  -2.0 ** -11, 2.0 ** -10, 3 * 2.0 ** -10], np.float32)
    want = [0x7E, 0x7E, 0x7E, 0x7E, 0x7E, 0x7E, 0xFE, 0xFE, 0x00, 0x80, 0x00, 0x80, 0x00, 0x02]
    assert oracle.quantize_act_fp8(x, 1.0).tolist() == want


def test_quantize_rounds_the_product_to_fp32_first():
    rng = np.random.default_rng(7)
    x = rng.normal(0, 3, 4000).astype(np.float32)
    inv = np.float32(0.37)
    prod = (x * inv).astype(np.float32)  # numpy fp32 product
    assert np.array_equal(oracle.quantize_act_fp8(x, inv), torch_codes(prod))


def _inputs(g, seed):
    n, h, w, c, k, r, s, st, pd = g
    xv = synth.normal(seed, "fp8x", (n, h, w, c), 2.0).astype(np.float32)
    xq = oracle.quantize_act_fp8(xv, 1.0)
    wr = synth.normal(seed, "fp8w", (k, r * s * c), 1.0)
    q = oracle.quantize(wr)
    return xq, q


@pytest.mark.parametrize("g", GEOMS)
def test_conv_matches_torch_conv2d(g):
    n, h, w, c, k, r, s, st, pd = g
    d = oracle.ConvDesc(*g)
    xq, q = _inputs(g, 3)
    x_scale = 0.75
    y = oracle.conv_fwd_fp8(d, xq, q.codes, q.alpha, x_scale)
    xt = torch.from_numpy(oracle.fp8_value(xq)).permute(0, 3, 1, 2)
    wt = torch.from_numpy(q.codes.astype(np.float64).reshape(k, r, s, c)).permute(0, 3, 1, 2)
    acc = F.conv2d(xt, wt, stride=st, padding=pd).permute(0, 2, 3, 1).numpy()
    ref = acc * q.alpha.astype(np.float64) * np.float64(np.float32(x_scale))
    assert np.array_equal(y, ref)
    yr = oracle.conv_fwd_fp8(d, xq, q.codes, q.alpha, x_scale, relu=True)
    assert np.array_equal(yr, np.maximum(ref, 0.0))
    idx = np.arange(0, y.size, 7, dtype=np.int64)
    assert np.array_equal(oracle.conv_fwd_fp8_sampled(d, xq, q.codes, q.alpha, x_scale, idx), y.reshape(-1)[idx])


def test_conv_1x1_is_a_matmul():
    g = (2, 3, 4, 24, 5, 1, 1, 1, 0)
    d = oracle.ConvDesc(*g)
    xq, q = _inputs(g, 4)
    y = oracle.conv_fwd_fp8(d, xq, q.codes, q.alpha, 2.0)
    ref = (oracle.fp8_value(xq).reshape(-1, 24) @ q.codes.astype(np.float64).T) * q.alpha.astype(np.float64) * 2.0
    assert np.array_equal(y.reshape(-1, 5), ref)


def test_conv_all_ones_input_closed_form():
    # f = 1 everywhere (code 0x38), 3x3 pad 1: an interior output is alpha_k * s * sum of the
    # filter's codes; a corner output sums only the four in-image taps
    g = (1, 5, 5, 8, 3, 3, 3, 1, 1)
    d = oracle.ConvDesc(*g)
    xq = np.full((1, 5, 5, 8), 0x38, np.uint8)
    wr = synth.normal(5, "fp8ones", (3, 72), 1.0)
    q = oracle.quantize(wr)
    y = oracle.conv_fwd_fp8(d, xq, q.codes, q.alpha, 1.0)
    cw = q.codes.astype(np.float64).reshape(3, 3, 3, 8)
    a = q.alpha.astype(np.float64)
    assert np.array_equal(y[0, 2, 2], a * cw.sum(axis=(1, 2, 3)))
    assert np.array_equal(y[0, 0, 0], a * cw[:, 1:, 1:, :].sum(axis=(1, 2, 3)))
