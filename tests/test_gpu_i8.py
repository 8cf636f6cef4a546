"""GPU parity of the integer-activation variant (int8 activation codes, two-bit filters on
the int8 matrix cores) against the oracle on the same seeded inputs.

Bars: activation codes bit-exact (the decision is one fp32 product and a round-half-even on
both sides); convolution outputs exact, because the integer sums are exact on both sides
and both apply the same two fp32 roundings (the scale product, then the scaling): fp32
outputs equal the oracle's value for value (-0 and +0 compare equal), bf16 outputs equal
the oracle's fp32 output rounded to nearest even.  Layer-sized cases compare sampled outputs
computed one by one by the oracle.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


SPECIAL = np.array([0.5, 1.5, 2.5, -2.5, -0.5, 126.5, 127.5, 300.0, -300.0, np.inf, -np.inf, np.nan, -0.0, 0.0],
                   np.float32)

ACT_CASES = [(1, "f32", 1.0), (15, "bf16", 1.0), (17, "f32", 1.0), (4097, "bf16", 0.73),
             (1 << 20, "f32", 0.73), (3 * 1048576 + 5, "bf16", 1.27)]


@pytest.mark.parametrize("count,dt,inv", ACT_CASES)
def test_quantize_act_parity(tbn, count, dt, inv):
    log("quantize_act_i8 count=%d %s inv=%g" % (count, dt, inv))
    x = synth.normal(3, "act%d" % count, (count,), 60.0).astype(np.float32)
    m = min(count, SPECIAL.size)
    x[:m] = SPECIAL[:m]
    inv = np.float32(inv)
    if dt == "bf16":
        bits = synth.bf16_bits(x)
        xv = synth.bf16_values(bits)
        xd = to_dev(bits.view(np.int16)).view(torch.bfloat16)
    else:
        xv = x
        xd = to_dev(x)
    q = tbn.quantize_act_i8(xd, float(inv))
    torch.cuda.synchronize()
    ref = oracle.quantize_act_i8(xv, inv)
    got = q.cpu().numpy()
    assert np.array_equal(got, ref), "mismatches: %d" % int((got != ref).sum())


def _problem(g, stream, full_range=False):
    n, h, w, c, k, r, s, st, pd = g
    d = oracle.ConvDesc(*g)
    if full_range:
        xq = synth.rng(stream, "xq%s" % (g,)).integers(-127, 128, size=(n, h, w, c)).astype(np.int8)
        x_scale = np.float32(0.01)
    else:
        x = synth.normal(stream, "x%s" % (g,), (n, h, w, c)).astype(np.float32)
        amax = np.float32(np.abs(x).max())
        inv = np.float32(127.0) / amax
        x_scale = amax / np.float32(127.0)
        xq = oracle.quantize_act_i8(x, inv)
    wr = synth.normal(stream, "w%s" % (g,), (k, r * s * c), 1.0)
    qz = oracle.quantize(wr)
    words = oracle.pack(qz.codes)
    return d, xq, qz.codes, qz.alpha, words, x_scale


def _run(tbn, g, xq, words, alpha, x_scale, out, relu):
    desc = tbn.ConvDesc(*g)
    y = tbn.conv2d_fwd_i8(desc, to_dev(xq), to_dev(words.view(np.int32)), to_dev(alpha), float(x_scale),
                          out_dtype=torch.float32 if out == "f32" else torch.bfloat16, relu=relu)
    torch.cuda.synchronize()
    return y.float().cpu().numpy()


def _expect(ref32, out):
    return ref32.astype(np.float64) if out == "f32" else oracle.round_bf16(ref32)


CONV_CASES = [
    # n, h, w, c, k, r, s, stride, pad
    (2, 9, 9, 16, 24, 3, 3, 1, 1),       # 16 channels: per-lane taps, ragged filter tile
    (1, 12, 12, 32, 70, 3, 3, 2, 1),     # stride 2, K % 8 != 0
    (2, 7, 7, 128, 256, 3, 3, 1, 1),     # 128 channels: one tap per stage
    (3, 6, 6, 256, 300, 3, 3, 1, 1),     # one tap per stage, two filter tiles, ragged
    (2, 14, 14, 64, 128, 1, 1, 1, 0),    # 1x1
    (1, 8, 8, 48, 64, 5, 5, 1, 2),       # 1200-element filters: odd code-chunk count
    (4, 4, 4, 512, 10, 4, 4, 1, 0),      # full-map "valid" layer (fully-connected form)
    (1, 1, 1, 16, 1, 1, 1, 1, 0),        # smallest layer
    (2, 17, 19, 16, 33, 7, 7, 2, 3),     # 7x7 stride 2, ragged everywhere
    (1, 30, 30, 144, 136, 3, 3, 1, 1),   # C % 128 != 0 above 128 channels
]


@pytest.mark.parametrize("g", CONV_CASES)
@pytest.mark.parametrize("out,relu", [("f32", False), ("bf16", True)])
def test_conv_i8_parity(tbn, g, out, relu):
    log("conv_fwd_i8 %s out=%s relu=%d" % (g, out, relu))
    d, xq, codes, alpha, words, x_scale = _problem(g, 4)
    ref, _ = oracle.conv_fwd_i8(d, xq, codes, alpha, x_scale, relu=relu)
    got = _run(tbn, g, xq, words, alpha, x_scale, out, relu)
    want = _expect(ref, out)
    assert np.array_equal(got.astype(np.float64), want.reshape(got.shape)), \
        "mismatches: %d" % int((got.astype(np.float64) != want.reshape(got.shape)).sum())


@pytest.mark.parametrize("tile", [1, 2, 3, 4])
def test_conv_i8_every_tile_shape(tbn, tile, knobs):
    g = (3, 10, 11, 128, 200, 3, 3, 1, 1)
    knobs(i8_tile=tile)
    log("conv_fwd_i8 tile %d %s" % (tile, g))
    d, xq, codes, alpha, words, x_scale = _problem(g, 5, full_range=True)
    ref, _ = oracle.conv_fwd_i8(d, xq, codes, alpha, x_scale)
    got = _run(tbn, g, xq, words, alpha, x_scale, "f32", False)
    assert np.array_equal(got.astype(np.float64), ref.astype(np.float64))


@pytest.mark.parametrize("g", [(128, 56, 56, 256, 256, 3, 3, 1, 1),   # the training layer's shape
                               (64, 14, 14, 256, 256, 3, 3, 1, 1),    # a ResNet-18 layer-3 shape
                               (64, 56, 56, 64, 64, 3, 3, 1, 1)])     # a ResNet-18 layer-1 shape
def test_conv_i8_layer_sized_sampled(tbn, g):
    """Full layer on the GPU (the launch configuration the benchmark times); 3000 sampled
    outputs computed one by one by the oracle, full-range activation codes."""
    log("conv_fwd_i8 layer-sized %s" % (g,))
    n, h, w, c, k, r, s, st, pd = g
    d = oracle.ConvDesc(*g)
    xq = synth.rng(6, "xqL%s" % (g,)).integers(-127, 128, size=(n, h, w, c)).astype(np.int8)
    wr = synth.normal(6, "wL%s" % (g,), (k, r * s * c), 1.0)
    qz = oracle.quantize(wr)
    words = oracle.pack(qz.codes)
    x_scale = np.float32(0.013)
    got = _run(tbn, g, xq, words, qz.alpha, x_scale, "f32", False).ravel()
    idx = synth.sample_indices(6, "idxL%s" % (g,), got.size, 3000)
    ref = oracle.conv_fwd_i8_sampled(d, xq, qz.codes, qz.alpha, x_scale, idx)
    assert np.array_equal(got[idx].astype(np.float64), ref.astype(np.float64))
    assert np.isfinite(got).all()
