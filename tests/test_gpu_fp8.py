"""GPU parity of the fp8-activation variant (E4M3 activation codes, two-bit filters as E2M1
values on the scaled fp8 x fp4 matrix cores) against the oracle on the same seeded inputs.

Bars: activation codes bit-exact (the decision is one fp32 product and a nearest-even
choice among the E4M3 values on both sides); the E2M1 repack of the codes equal to the
layout written out below.  Convolution outputs: the oracle's sums are exact, while the
matrix core forms each 64-element step's dot product in a fixed-point window that keeps
the products only down to 2^(e - 14), e the exponent of the step's largest product
(measured: 448 + 63 x 2^-9 gives 448 + 56 x 2^-9), before adding it to the fp32 sum.  So
an output may differ from the exact one by up to n * 2^(e_max - 14) (n = R*S*C terms, e_max
the exponent of the largest |f W~| in the layer) times alpha_k * s, plus fp32 rounding of
the running sum; the bar below takes one more bit, n * 2^(e_max - 13), plus 2^-20 of the
sum of |terms| (bound via n * max|term|), and bf16 outputs one bf16 rounding (2^-8 relative)
more.  Layer-sized cases compare sampled outputs computed one by one by the oracle.
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


def nerr(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-300))


# values at the format's edges: subnormal steps, ties between neighbours, the largest
# finite value and beyond, NaN and both zeros
SPECIAL = np.array([2.0 ** -10, 3 * 2.0 ** -10, 2.0 ** -9, 2.0 ** -6, 1.0625, 1.1875, 448.0, 464.0, 465.0, 1e30,
                    -1e30, np.inf, -np.inf, np.nan, -0.0, 0.0, -2.0 ** -11, 0.0150], np.float32)

ACT_CASES = [(1, "f32", 1.0), (15, "bf16", 1.0), (17, "f32", 1.0), (4097, "bf16", 0.73),
             (1 << 20, "f32", 3.1), (3 * 1048576 + 5, "bf16", 1.27)]


@pytest.mark.parametrize("count,dt,inv", ACT_CASES)
def test_quantize_act_fp8_parity(tbn, count, dt, inv):
    log("quantize_act_fp8 count=%d %s inv=%g" % (count, dt, inv))
    x = synth.normal(3, "f8act%d" % count, (count,), 40.0).astype(np.float32)
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
    q = tbn.quantize_act_fp8(xd, float(inv))
    torch.cuda.synchronize()
    ref = oracle.quantize_act_fp8(xv, inv)
    got = q.cpu().numpy()
    assert np.array_equal(got, ref), "mismatches: %d" % int((got != ref).sum())


@pytest.mark.parametrize("inv", [1.0, 0.37, 448.0 / 3.0])
def test_quantize_act_fp8_every_bf16_value(tbn, inv):
    # all 65536 bf16 bit patterns (NaNs, infinities, subnormals included)
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    xv = synth.bf16_values(bits)
    q = tbn.quantize_act_fp8(to_dev(bits.view(np.int16)).view(torch.bfloat16), float(inv))
    torch.cuda.synchronize()
    ref = oracle.quantize_act_fp8(xv, np.float32(inv))
    got = q.cpu().numpy()
    assert np.array_equal(got, ref), "mismatches: %d" % int((got != ref).sum())


def e2m1_layout(words: np.ndarray) -> np.ndarray:
    """The E2M1 operand layout of packed words, written out from its definition: element
    e = 8 r + j of a word (magnitude bit 16 (e % 2) + e / 2, sign bit 8 above it) goes to
    magnitude bit 4 j + 1 - r and sign bit 4 j + 3 - r."""
    w = words.astype(np.uint64)
    out = np.zeros_like(w)
    for e in range(16):
        m = (w >> np.uint64(16 * (e % 2) + e // 2)) & np.uint64(1)
        s = (w >> np.uint64(16 * (e % 2) + 8 + e // 2)) & np.uint64(1)
        j, r = e % 8, e // 8
        out |= (m << np.uint64(4 * j + 1 - r)) | (s << np.uint64(4 * j + 3 - r))
    return out.astype(np.uint32)


def test_repack_codes_fp4_layout(tbn):
    wr = synth.normal(8, "f4pack", (300, 777), 1.0)
    words = oracle.pack(oracle.quantize(wr).codes)
    got = tbn.repack_codes_fp4(to_dev(words.view(np.int32)))
    torch.cuda.synchronize()
    assert np.array_equal(got.cpu().numpy().view(np.uint32), e2m1_layout(words))


def _problem(g, stream):
    n, h, w, c, k, r, s, st, pd = g
    d = oracle.ConvDesc(*g)
    # full-range finite E4M3 codes (NaN codes 0x7F and 0xFF left out)
    raw = synth.rng(stream, "f8xq%s" % (g,)).integers(0, 254, size=(n, h, w, c))
    xq = (raw + (raw >= 0x7F)).astype(np.uint8)
    x_scale = np.float32(0.01)
    wr = synth.normal(stream, "f8w%s" % (g,), (k, r * s * c), 1.0)
    qz = oracle.quantize(wr)
    words = oracle.pack(qz.codes)
    return d, xq, qz.codes, qz.alpha, words, x_scale


def _run(tbn, g, xq, words, alpha, x_scale, out, relu):
    desc = tbn.ConvDesc(*g)
    f4 = tbn.repack_codes_fp4(to_dev(words.view(np.int32)))
    y = tbn.conv2d_fwd_fp8(desc, to_dev(xq), f4, to_dev(alpha), float(x_scale),
                           out_dtype=torch.float32 if out == "f32" else torch.bfloat16, relu=relu)
    torch.cuda.synchronize()
    return y.float().cpu().numpy()


def check(got, ref, d, xq, alpha_k, x_scale, out):
    """|got - ref| within the bound of the module docstring, per output (alpha_k broadcasts
    over the last axis, or is given per sampled output)."""
    n = d.r * d.s * d.c
    fmax = float(np.nanmax(np.abs(oracle.fp8_value(xq))))
    tmax = 2.0 * fmax  # largest |f W~|: |W~| <= 2
    e_max = np.floor(np.log2(tmax)) if tmax > 0 else -30
    per_unit = n * 2.0 ** (e_max - 13) + 2.0 ** -20 * n * tmax
    scale = np.abs(np.asarray(alpha_k, np.float64)) * float(np.float32(x_scale))
    bound = per_unit * scale
    if out != "f32":
        bound = bound + 2.0 ** -8 * np.abs(ref)
    err = np.abs(np.asarray(got, np.float64) - ref)
    log("  max error %.3e, max error / bound %.3f, normalised max error %.3e"
        % (err.max(), float(np.max(err / bound)), nerr(got, ref)))
    assert np.all(err <= bound)


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
def test_conv_fp8_parity(tbn, g, out, relu):
    log("conv_fwd_fp8 %s out=%s relu=%d" % (g, out, relu))
    d, xq, codes, alpha, words, x_scale = _problem(g, 4)
    ref = oracle.conv_fwd_fp8(d, xq, codes, alpha, x_scale, relu=relu)
    got = _run(tbn, g, xq, words, alpha, x_scale, out, relu)
    check(got, ref.reshape(got.shape), d, xq, alpha, x_scale, out)


@pytest.mark.parametrize("tile", [1, 2, 3, 4])
def test_conv_fp8_every_tile_shape(tbn, tile, knobs):
    g = (3, 10, 11, 128, 200, 3, 3, 1, 1)
    knobs(fp8_tile=tile)
    log("conv_fwd_fp8 tile %d %s" % (tile, g))
    d, xq, codes, alpha, words, x_scale = _problem(g, 5)
    ref = oracle.conv_fwd_fp8(d, xq, codes, alpha, x_scale)
    got = _run(tbn, g, xq, words, alpha, x_scale, "f32", False)
    check(got, ref.reshape(got.shape), d, xq, alpha, x_scale, "f32")


@pytest.mark.parametrize("g", [(128, 56, 56, 256, 256, 3, 3, 1, 1),   # the training layer's shape
                               (64, 14, 14, 256, 256, 3, 3, 1, 1),    # a ResNet-18 layer-3 shape
                               (64, 56, 56, 64, 64, 3, 3, 1, 1)])     # a ResNet-18 layer-1 shape
def test_conv_fp8_layer_sized_sampled(tbn, g):
    """Full layer on the GPU (the launch configuration the benchmark times); 3000 sampled
    outputs computed one by one by the oracle, full-range activation codes."""
    log("conv_fwd_fp8 layer-sized %s" % (g,))
    n, h, w, c, k, r, s, st, pd = g
    d = oracle.ConvDesc(*g)
    raw = synth.rng(6, "f8xqL%s" % (g,)).integers(0, 254, size=(n, h, w, c))
    xq = (raw + (raw >= 0x7F)).astype(np.uint8)
    wr = synth.normal(6, "f8wL%s" % (g,), (k, r * s * c), 1.0)
    qz = oracle.quantize(wr)
    words = oracle.pack(qz.codes)
    x_scale = np.float32(0.013)
    got = _run(tbn, g, xq, words, qz.alpha, x_scale, "f32", False).ravel()
    idx = synth.sample_indices(6, "f8idxL%s" % (g,), got.size, 3000)
    ref = oracle.conv_fwd_fp8_sampled(d, xq, qz.codes, qz.alpha, x_scale, idx)
    k_of = idx % k
    check(got[idx], ref, d, xq, qz.alpha[k_of], x_scale, "f32")
    assert np.isfinite(got).all()
