"""GPU parity: every call of the C ABI against the fp64 oracle on the same seeded inputs.

Bars (from the method's arithmetic):
  * codes, packed words and B1/B2 counts: bit-exact;
  * alpha: within 1 fp32 ulp (both sides sum in fp64 and round once; only the order of
    the fp64 sums differs);
  * convolution outputs and gradients: normalised max error max|g - r| / max|r| <= 1e-2
    (bf16 operands, fp32 accumulation; fwd with fp32 output is in fact ~1e-6);
  * SGD: fp32 element-wise arithmetic, relative 1e-6 of the largest value.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

TOL = 1e-2


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def nerr(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.max(np.abs(ref)) if ref.size else 0.0
    if scale == 0.0:
        return float(np.max(np.abs(got))) if got.size else 0.0
    return float(np.max(np.abs(got - ref)) / scale)


def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.to(dtype)


def bf16_dev(bits):
    return to_dev(bits.view(np.int16)).view(torch.bfloat16)


def words_np(codes_t):
    return codes_t.cpu().numpy().view(np.uint32)


def ulp_diff(a, b):
    a = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    b = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    return np.abs(a - b)


# ---------------------------------------------------------------------------------------
# Quantiser (Sec. 2 Eq. 3-5)
# ---------------------------------------------------------------------------------------
def _boundary_weights(K, n, name):
    g = synth.rng(0, name)
    base = np.array([-1.0, 0.0, -0.0, 1.0, 2.0, -2.0, 1e-40, -1e-40, 3.4e38, -3.4e38], np.float32)
    vals = base[g.integers(0, base.size, size=(K, n))]
    steps = g.integers(-2, 3, size=(K, n))
    out = vals.copy()
    for s in (-2, -1, 1, 2):
        m = steps == s
        v = out[m]
        for _ in range(abs(s)):
            v = np.nextafter(v, np.float32(np.sign(s) * np.inf))
        out[m] = v
    return out.astype(np.float32)


def test_codes_of_every_fp32_bit_pattern(tbn):
    """Eq. 3 on all 2^32 fp32 bit patterns (16 chunks of 2^28 weights, quantised as 65536
    filters of 4096): the GPU's codes equal the oracle's for every non-NaN value, and a NaN
    gets -1 (the documented choice; NaN is outside the method)."""
    CH = 1 << 28
    K, n = CH // 4096, 4096
    for c in range(16):
        start = c * CH
        v = torch.arange(start, start + CH, dtype=torch.int64, device="cuda")
        v = torch.where(v >= 2 ** 31, v - 2 ** 32, v).to(torch.int32)
        w = v.view(torch.float32).view(K, n)
        codes, _, _ = tbn.quantize(w, want_counts=False)
        torch.cuda.synchronize()
        del v, w
        got = oracle.unpack(words_np(codes), K, n).ravel()
        ref = oracle.codes_of_bits(start, CH)
        nan = ref == 0
        bad = int(np.count_nonzero(got[~nan] != ref[~nan]))
        log("bit patterns 0x%08x..0x%08x: %d NaN, %d mismatches" % (start, start + CH - 1, int(nan.sum()), bad))
        assert bad == 0
        assert np.all(got[nan] == -1)
        del codes, got, ref, nan


QCASES = [
    # K, n, distribution
    (1, 1, "n1"), (32, 25, "n0.05"), (64, 800, "n0.05"), (10, 512, "n1"), (130, 2304, "n1"),
    (512, 3136, "n0.05"), (7, 4608, "n3"), (65, 129, "boundary"), (200, 64, "boundary"),
    (3, 100, "zeros"), (1000, 512, "n1"),
]


@pytest.mark.parametrize("K,n,dist", QCASES)
def test_quantize_parity(tbn, K, n, dist):
    log("quantize K=%d n=%d %s" % (K, n, dist))
    if dist == "boundary":
        w = _boundary_weights(K, n, "qb%d_%d" % (K, n))
    elif dist == "zeros":
        w = np.zeros((K, n), np.float32)
        w[1, :] = -0.0
        w[2, 5] = 1e-45
    else:
        w = synth.normal(1, "q%d_%d_%s" % (K, n, dist), (K, n), float(dist[1:]))
    q = oracle.quantize(w)
    codes, alpha, counts = tbn.quantize(to_dev(w))
    torch.cuda.synchronize()
    assert np.array_equal(words_np(codes), oracle.pack(q.codes)), "packed codes differ"
    assert np.array_equal(counts.cpu().numpy(), np.stack([q.b1_size, q.b2_size], 1)), "B1/B2 counts differ"
    d = ulp_diff(alpha.cpu().numpy(), q.alpha)
    assert d.max() <= 1, "alpha differs by %d ulp" % d.max()
    log("  alpha ulp max %d, exact %d/%d" % (d.max(), int((d == 0).sum()), K))


SQCASES = [(1, 1), (3, 5), (70, 2341), (256, 2304), (512, 3136)]


@pytest.mark.parametrize("K,n", SQCASES)
def test_sgd_step_quantize_parity(tbn, K, n):
    """Update fused with the next quantisation: the weights and momentum equal the
    standalone SGD call and the fp32 oracle bit for bit; codes, counts and alpha equal the
    standalone quantiser and the oracle's quantisation of the updated weights."""
    log("sgd_step_quantize K=%d n=%d" % (K, n))
    w = synth.normal(1, "sq_w%d_%d" % (K, n), (K, n), 1.0)
    v = synth.normal(1, "sq_v%d_%d" % (K, n), (K, n), 0.5)
    g = synth.normal(1, "sq_g%d_%d" % (K, n), (K, n), 1.0)
    lr, mu, wd = 0.5, 0.5, 0.25
    if K * n >= 4:
        # elements whose exact update lands on the thresholds of Eq. (3): w_new = 1, 0, -1
        w.flat[:3] = [1.5, 0.5, -0.5]
        v.flat[:3] = [0.25, 0.25, 0.25]
        g.flat[:3] = [0.5, 0.75, 1.0]
    wf, vf = to_dev(w), to_dev(v)
    gd = to_dev(g)
    codes_f, alpha_f, counts_f = tbn.sgd_step_quantize(wf, vf, gd, lr, mu, wd)
    ws, vs = to_dev(w), to_dev(v)
    tbn.sgd_step(ws, vs, gd, lr, mu, wd)
    codes_s, alpha_s, counts_s = tbn.quantize(ws)
    torch.cuda.synchronize()
    w_new, v_new = wf.cpu().numpy(), vf.cpu().numpy()
    assert np.array_equal(w_new.view(np.int32), ws.cpu().numpy().view(np.int32)), "w differs from sgd_step"
    assert np.array_equal(v_new.view(np.int32), vs.cpu().numpy().view(np.int32)), "v differs from sgd_step"
    assert np.array_equal(words_np(codes_f), words_np(codes_s))
    assert np.array_equal(alpha_f.cpu().numpy().view(np.int32), alpha_s.cpu().numpy().view(np.int32))
    assert np.array_equal(counts_f.cpu().numpy(), counts_s.cpu().numpy())
    w_o, v_o = oracle.sgd_f32(w, v, g, lr, mu, wd)
    assert np.array_equal(w_new.ravel().view(np.int32), w_o.view(np.int32)), "w differs from the fp32 oracle"
    assert np.array_equal(v_new.ravel().view(np.int32), v_o.view(np.int32)), "v differs from the fp32 oracle"
    if K * n >= 4:
        assert list(w_o[:3]) == [1.0, 0.0, -1.0]
    q = oracle.quantize(w_o.reshape(K, n))
    assert np.array_equal(words_np(codes_f), oracle.pack(q.codes)), "packed codes differ"
    assert np.array_equal(counts_f.cpu().numpy(), np.stack([q.b1_size, q.b2_size], 1))
    d = ulp_diff(alpha_f.cpu().numpy(), q.alpha)
    assert d.max() <= 1, "alpha differs by %d ulp" % d.max()
    w64, _ = oracle.sgd(w, v, g, lr, mu, wd)
    assert nerr(w_new.ravel(), w64) <= 1e-6


VARIANT_CASES = [
    # K, n, weight std, threshold, stochastic
    (32, 25, 0.05, 0.05, False), (130, 2304, 1.0, 0.5, False), (7, 4608, 1.0, 2.0, False),
    (65, 129, 1.0, 1.0, True), (256, 2304, 1.0, 1.0, True), (3, 5, 3.0, 1.0, True), (1, 1, 1.0, 0.7, False),
]


@pytest.mark.parametrize("K,n,std,t,stoch", VARIANT_CASES)
def test_quantize_variant_parity(tbn, K, n, std, t, stoch):
    """Discretisation variants against the oracle: codes and counts bit-exact, alpha within
    1 ulp.  Threshold cases include weights exactly at +-t and one ulp either side."""
    log("quantize_variant K=%d n=%d std=%g t=%g stochastic=%s" % (K, n, std, t, stoch))
    w = synth.normal(1, "qv_w%d_%d" % (K, n), (K, n), std)
    if not stoch and K * n >= 6:
        tt = np.float32(t)
        w.flat[:6] = [tt, -tt, np.nextafter(tt, np.float32(9)), np.nextafter(-tt, np.float32(-9)),
                      np.nextafter(tt, np.float32(0)), 0.0]
    u = np.minimum(synth.uniform(1, "qv_u%d_%d" % (K, n), (K, n)), np.float32(1 - 2 ** -24)) if stoch else None
    q = oracle.quantize_variant(w, t, u)
    codes, alpha, counts = tbn.quantize_variant(to_dev(w), t, None if u is None else to_dev(u))
    torch.cuda.synchronize()
    assert np.array_equal(words_np(codes), oracle.pack(q.codes)), "packed codes differ"
    assert np.array_equal(counts.cpu().numpy(), np.stack([q.b1_size, q.b2_size], 1)), "counts differ"
    d = ulp_diff(alpha.cpu().numpy(), q.alpha)
    assert d.max() <= 1, "alpha differs by %d ulp" % d.max()
    if not stoch and t == 1.0:
        c2, a2, _ = tbn.quantize(to_dev(w))
        assert torch.equal(c2, codes) and torch.equal(a2, alpha)


def test_quantize_bit_pattern_sweep(tbn):
    # Every fp32 sign/exponent/top-7-fraction pattern with 16 low-fraction variants:
    # 2^16 * 16 values, finite ones compared with the oracle; NaN -> code -1 by contract.
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lo = np.array([0, 1, 2, 3, 0x7FFF, 0x8000, 0x8001, 0xFFFE, 0xFFFF, 0x1234, 0x4000, 0xC000,
                   0x00FF, 0xFF00, 0x5555, 0xAAAA], np.uint32)
    bits = (hi[:, None] | lo[None, :]).ravel()
    w = bits.view(np.float32)
    finite = np.isfinite(w)
    wf = w[finite]
    n = 4096
    wf = wf[: wf.size // n * n].reshape(-1, n)
    q = oracle.quantize(wf)
    codes, _, _ = tbn.quantize(to_dev(wf))
    torch.cuda.synchronize()
    assert np.array_equal(words_np(codes), oracle.pack(q.codes))
    # non-finite inputs: +-inf behave as |W| > 1; NaN takes code -1
    special = np.array([[np.inf, -np.inf, np.nan, -np.nan, 0.5, -0.5, 2.0, -2.0]], np.float32)
    codes, _, _ = tbn.quantize(to_dev(special))
    torch.cuda.synchronize()
    got = oracle.unpack(words_np(codes), 1, 8)[0].tolist()
    assert got == [2, -2, -1, -1, 1, -1, 2, -2]


# ---------------------------------------------------------------------------------------
# Convolutions (Sec. 2 Eq. 1; Sec. 3)
# ---------------------------------------------------------------------------------------
CONV_CASES = [
    # n, h, w, c, k, r, s, stride, pad
    (16, 28, 28, 1, 32, 5, 5, 1, 2),        # single two-bit layer, MNIST-shaped
    (4, 14, 14, 32, 64, 5, 5, 1, 2),        # LeNet conv2 shape, small batch
    (2, 9, 9, 3, 5, 3, 3, 2, 1),            # tiny, ragged everything
    (2, 16, 16, 64, 64, 3, 3, 1, 1),
    (2, 15, 13, 64, 96, 3, 3, 1, 1),        # ragged pixels and filters
    (3, 12, 12, 128, 130, 3, 3, 2, 1),      # stride 2, filters beyond two 64-blocks
    (2, 14, 14, 256, 256, 3, 3, 1, 1),
    (4, 1, 1, 512, 10, 1, 1, 1, 0),         # FC 512 -> 10 as a 1x1 conv
    (8, 7, 7, 64, 512, 7, 7, 1, 0),         # FC 3136 -> 512 as a 7x7 "valid" conv
    (2, 16, 16, 64, 128, 1, 1, 2, 0),       # 1x1 stride-2 projection
    (1, 33, 31, 3, 64, 7, 7, 2, 3),         # stem-like, C = 3
    (2, 10, 10, 40, 24, 3, 3, 1, 1),        # C = 40 (not a multiple of 64), K = 24
    (3, 40, 70, 3, 64, 7, 7, 2, 3),         # stem 7x7/2 over RGB: several row and column tiles
    (2, 11, 13, 7, 72, 3, 3, 1, 1),         # 7 channels (padded to 8), two filter blocks
    (1, 19, 23, 4, 64, 5, 5, 2, 2),         # 4 channels, stride 2
    (2, 9, 9, 2, 16, 3, 3, 1, 0),           # 2 channels, no padding
    (1, 1, 1, 16, 8, 3, 3, 1, 1),           # 1x1 image under a 3x3 window: only the centre tap
    (2, 5, 5, 8, 1, 3, 3, 1, 1),            # a single filter
    (2, 20, 24, 3, 20, 5, 11, 1, 2),        # C = 3, 11 taps per filter row (64-element rows)
    (1, 12, 12, 7, 16, 3, 9, 1, 1),         # C = 7, 9 taps per row (128-element rows)
]


def _conv_inputs(g, stream, wstd=1.0):
    n, h, w, c, k, r, s, st, pd = g
    d = oracle.ConvDesc(*g)
    P, Q = d.out_dims()
    xb = synth.normal_bf16(stream, "x%s" % (g,), (n, h, w, c))
    dyb = synth.normal_bf16(stream, "dy%s" % (g,), (n, P, Q, k))
    wr = synth.normal(stream, "w%s" % (g,), (k, r * s * c), wstd)
    return d, P, Q, xb, dyb, wr


@pytest.mark.parametrize("g", CONV_CASES)
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_fwd_parity(tbn, g, out):
    log("fwd %s out=%s" % (g, out))
    d, P, Q, xb, _, wr = _conv_inputs(g, 2)
    q = oracle.quantize(wr)
    ref = oracle.conv_fwd(d, oracle.bf16_bits_to_f64(xb), q.codes, q.alpha.astype(np.float64))
    codes, alpha, _ = tbn.quantize(to_dev(wr))
    desc = tbn.ConvDesc(*g)
    y = tbn.conv2d_fwd(desc, bf16_dev(xb), codes, alpha,
                       out_dtype=torch.float32 if out == "f32" else torch.bfloat16)
    torch.cuda.synchronize()
    e = nerr(y.float().cpu().numpy(), ref)
    log("  normalised max error %.3e" % e)
    assert e <= (1e-4 if out == "f32" else TOL)


@pytest.mark.parametrize("g,xdt", [((8, 224, 224, 3, 64, 7, 7, 2, 3), "bf16"),   # ResNet stem, batch 8
                                    ((7, 224, 224, 3, 40, 7, 7, 2, 3), "f32"),    # fp32 input, ragged filters
                                    ((16, 256, 256, 1, 32, 5, 5, 1, 2), "bf16"),  # one channel
                                    ((4, 257, 263, 5, 24, 3, 3, 2, 1), "bf16")])  # 5 channels, odd sizes
def test_fwd_thin_bordered_copy(tbn, g, xdt, knobs):
    """Inputs of 2^20 elements and more with fewer than 8 channels: the input is first written
    into workspace as a zero-bordered copy and the patches are copied from it (the thin-input
    kernel forced, as small filters would otherwise take the direct kernel)."""
    knobs(conv_tile=20)
    log("fwd thin bordered copy %s %s" % (g, xdt))
    n, h, w, c, k, r, s, st, pd = g
    assert n * h * w * c >= 1 << 20
    desc = tbn.ConvDesc(*g)
    assert tbn.workspace_size(tbn.OP_FWD, desc) > 0
    d = oracle.ConvDesc(*g)
    wr = synth.normal(2, "bw%s" % (g,), (k, r * s * c), 1.0)
    q = oracle.quantize(wr)
    codes, alpha, _ = tbn.quantize(to_dev(wr))
    if xdt == "f32":
        x = synth.normal(2, "bx%s" % (g,), (n, h, w, c))
        xin, xref = to_dev(x), oracle.round_bf16(x)
    else:
        xb = synth.normal_bf16(2, "bx%s" % (g,), (n, h, w, c))
        xin, xref = bf16_dev(xb), oracle.bf16_bits_to_f64(xb)
    y = tbn.conv2d_fwd(desc, xin, codes, alpha, out_dtype=torch.float32)
    torch.cuda.synchronize()
    imgs = [0, n - 1]
    ref = oracle.conv_fwd(oracle.ConvDesc(len(imgs), h, w, c, k, r, s, st, pd), xref[imgs], q.codes,
                          q.alpha.astype(np.float64))
    e = nerr(y.cpu().numpy()[imgs], ref)
    log("  images %s: normalised max error %.3e" % (imgs, e))
    assert e <= 1e-4


@pytest.mark.parametrize("g,xdt", [((16, 28, 28, 1, 32, 5, 5, 1, 2), "f32"),   # the single-layer workload
                                    ((3, 28, 28, 1, 20, 5, 5, 1, 0), "bf16"),   # LeNet conv1 shape, ragged K
                                    ((2, 9, 9, 3, 72, 3, 3, 2, 1), "f32"),      # RGB 3x3 stride 2, two filter blocks
                                    ((1, 13, 11, 7, 40, 3, 3, 1, 1), "bf16"),   # 7 channels (63 elements)
                                    ((2, 10, 9, 1, 8, 7, 7, 1, 3), "bf16"),     # 7x7, one filter group
                                    ((5, 6, 7, 4, 33, 1, 1, 1, 0), "f32"),      # 1x1, K one past 32
                                    ((1, 37, 35, 3, 64, 7, 7, 2, 3), "bf16")])  # the 7x7 RGB stem, 147 elements
def test_fwd_direct_small_layers(tbn, g, xdt):
    """The direct fp32-FMA kernel (few channels, at most 147 filter elements): fused epilogue
    (scale, bias, residual, ReLU) with bf16 output and plain fp32 output against the oracle."""
    log("fwd direct %s %s" % (g, xdt))
    n, h, w, c, k, r, s, st, pd = g
    d = oracle.ConvDesc(*g)
    P, Q = d.out_dims()
    wr = synth.normal(11, "dw%s" % (g,), (k, r * s * c), 1.0)
    q = oracle.quantize(wr)
    codes, alpha, _ = tbn.quantize(to_dev(wr))
    if xdt == "f32":
        x = synth.normal(11, "dx%s" % (g,), (n, h, w, c))
        xin, xref = to_dev(x), oracle.round_bf16(x)
    else:
        xb = synth.normal_bf16(11, "dx%s" % (g,), (n, h, w, c))
        xin, xref = bf16_dev(xb), oracle.bf16_bits_to_f64(xb)
    scale = synth.uniform(11, "dsc", (k,), 0.5, 1.5)
    bias = synth.normal(11, "dbi", (k,), 0.1)
    resb = synth.normal_bf16(11, "dres", (n, P, Q, k))
    acc = oracle.conv_fwd(d, xref, q.codes, q.alpha.astype(np.float64))
    desc = tbn.ConvDesc(*g)
    y32 = tbn.conv2d_fwd(desc, xin, codes, alpha, out_dtype=torch.float32)
    y = tbn.conv2d_fwd(desc, xin, codes, alpha, out_dtype=torch.bfloat16, scale=to_dev(scale), bias=to_dev(bias),
                       residual=bf16_dev(resb), relu=True)
    torch.cuda.synchronize()
    e = nerr(y32.cpu().numpy(), acc)
    assert e <= 1e-4, "fwd %s: %.3e" % (g, e)
    ref = np.maximum(acc * scale.astype(np.float64) + bias + oracle.bf16_bits_to_f64(resb), 0.0)
    e = nerr(y.float().cpu().numpy(), ref)
    assert e <= TOL, "fwd epilogue %s: %.3e" % (g, e)


def test_fwd_fp32_input_single_layer(tbn):
    # 16 x 1 x 28 x 28 fp32 uniform[0,1) input, 32 filters 5x5, pad 2, N(0, 0.05) masters.
    g = (16, 28, 28, 1, 32, 5, 5, 1, 2)
    d = oracle.ConvDesc(*g)
    x = synth.uniform(0, "x", (16, 28, 28, 1))
    wr = synth.normal(0, "w", (32, 25), 0.05)
    q = oracle.quantize(wr)
    ref = oracle.conv_fwd(d, oracle.round_bf16(x), q.codes, q.alpha.astype(np.float64))
    codes, alpha, _ = tbn.quantize(to_dev(wr))
    y = tbn.conv2d_fwd(tbn.ConvDesc(*g), to_dev(x), codes, alpha, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert np.array_equal(words_np(codes), oracle.pack(q.codes))
    e = nerr(y.cpu().numpy(), ref)
    log("single layer fp32 input: normalised max error %.3e" % e)
    assert e <= 1e-4


@pytest.mark.parametrize("g", [(2, 16, 16, 64, 64, 3, 3, 1, 1), (2, 15, 13, 64, 96, 3, 3, 1, 1),
                               (3, 12, 12, 128, 130, 3, 3, 2, 1), (2, 10, 10, 40, 24, 3, 3, 1, 1)])
def test_fwd_epilogue(tbn, g):
    log("fwd epilogue %s" % (g,))
    d, P, Q, xb, _, wr = _conv_inputs(g, 3)
    k = g[4]
    q = oracle.quantize(wr)
    scale = synth.uniform(3, "sc", (k,), 0.5, 1.5)
    bias = synth.normal(3, "bi", (k,), 0.1)
    resb = synth.normal_bf16(3, "res", (g[0], P, Q, k))
    acc = oracle.conv_fwd(d, oracle.bf16_bits_to_f64(xb), q.codes, q.alpha.astype(np.float64))
    ref = np.maximum(acc * scale.astype(np.float64) + bias + oracle.bf16_bits_to_f64(resb), 0.0)
    codes, alpha, _ = tbn.quantize(to_dev(wr))
    y = tbn.conv2d_fwd(tbn.ConvDesc(*g), bf16_dev(xb), codes, alpha, out_dtype=torch.bfloat16,
                       scale=to_dev(scale), bias=to_dev(bias), residual=bf16_dev(resb), relu=True)
    torch.cuda.synchronize()
    e = nerr(y.float().cpu().numpy(), ref)
    log("  normalised max error %.3e" % e)
    assert e <= TOL


DENSE_CASES = [(4, 32, 32, 3, 128, 3, 3, 1, 1), (2, 9, 9, 3, 5, 3, 3, 2, 1), (2, 12, 11, 40, 24, 3, 3, 1, 1),
               (1, 20, 20, 70, 16, 3, 3, 1, 1),  # reduces over 630 > one LDS fill of 512 (vector-ALU kernel)
               (2, 14, 14, 1, 32, 5, 5, 1, 2), (2, 10, 9, 7, 70, 3, 3, 1, 1)]  # thin MFMA kernel, two filter blocks


@pytest.mark.parametrize("g", DENSE_CASES)
def test_fwd_dense_parity(tbn, g):
    # the full-precision layer: filters rounded to bf16, fp32 accumulation, fused epilogue
    log("fwd dense %s" % (g,))
    d, P, Q, xb, _, _ = _conv_inputs(g, 5)
    k = g[4]
    w = synth.normal(5, "wd%s" % (g,), (k, g[5] * g[6] * g[3]), 0.3)
    scale = synth.uniform(5, "sc", (k,), 0.5, 1.5)
    bias = synth.normal(5, "bi", (k,), 0.1)
    resb = synth.normal_bf16(5, "res", (g[0], P, Q, k))
    acc = oracle.conv_fwd_dense(d, oracle.bf16_bits_to_f64(xb), oracle.round_bf16(w))
    desc = tbn.ConvDesc(*g)
    y32 = tbn.conv2d_fwd_dense(desc, bf16_dev(xb), to_dev(w), out_dtype=torch.float32)
    y = tbn.conv2d_fwd_dense(desc, bf16_dev(xb), to_dev(w), scale=to_dev(scale), bias=to_dev(bias),
                             residual=bf16_dev(resb), relu=True)
    xf = oracle.bf16_bits_to_f64(xb).astype(np.float32)  # fp32 input holding bf16 values
    yf = tbn.conv2d_fwd_dense(desc, to_dev(xf), to_dev(w), out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert nerr(y32.cpu().numpy(), acc) <= 1e-5
    assert nerr(yf.cpu().numpy(), acc) <= 1e-5
    ref = np.maximum(acc * scale.astype(np.float64) + bias + oracle.bf16_bits_to_f64(resb), 0.0)
    assert nerr(y.float().cpu().numpy(), ref) <= TOL


FC_CASES = [
    # n, h, w, c, k, r, s, stride, pad: the filter window covers the whole input map
    (1, 1, 1, 8192, 4096, 1, 1, 1, 0),      # weight streaming at batch 1
    (3, 1, 1, 100, 70, 1, 1, 1, 0),         # ragged reduction and filter count
    (16, 1, 1, 512, 1000, 1, 1, 1, 0),      # the ResNet classifier at the widest batch
    (2, 4, 4, 512, 10, 4, 4, 1, 0),         # the CIFAR classifier, 4x4 map
    (1, 7, 7, 64, 512, 7, 7, 1, 0),         # the MNIST fc1, 7x7 map
]


@pytest.mark.parametrize("g", FC_CASES)
def test_fc_stream_parity(tbn, g):
    # fully-connected layers at small batch (codes streamed into 16x16x32 MFMAs), with the
    # fused epilogue and with fp32 input
    log("fc %s" % (g,))
    d, P, Q, xb, _, wr = _conv_inputs(g, 10)
    k = g[4]
    q = oracle.quantize(wr)
    a64 = q.alpha.astype(np.float64)
    acc = oracle.conv_fwd(d, oracle.bf16_bits_to_f64(xb), q.codes, a64)
    codes, alpha, _ = tbn.quantize(to_dev(wr))
    desc = tbn.ConvDesc(*g)
    y32 = tbn.conv2d_fwd(desc, bf16_dev(xb), codes, alpha, out_dtype=torch.float32)
    scale = synth.uniform(10, "sc", (k,), 0.5, 1.5)
    bias = synth.normal(10, "bi", (k,), 0.1)
    resb = synth.normal_bf16(10, "res", (g[0], 1, 1, k))
    y = tbn.conv2d_fwd(desc, bf16_dev(xb), codes, alpha, scale=to_dev(scale), bias=to_dev(bias),
                       residual=bf16_dev(resb), relu=True)
    xf = oracle.bf16_bits_to_f64(xb).astype(np.float32)
    yf = tbn.conv2d_fwd(desc, to_dev(xf), codes, alpha, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert nerr(y32.cpu().numpy(), acc) <= 1e-4
    assert nerr(yf.cpu().numpy(), acc) <= 1e-4
    ref = np.maximum(acc * scale.astype(np.float64) + bias + oracle.bf16_bits_to_f64(resb), 0.0)
    assert nerr(y.float().cpu().numpy(), ref) <= TOL


@pytest.mark.parametrize("variant", list(range(8)))
def test_fc_stream_every_variant(tbn, variant, knobs):
    # each variant of the weight-streaming kernel (loads per buffer x buffers x wave groups)
    knobs(fc_variant=variant)
    for g in [(1, 1, 1, 8192, 200, 1, 1, 1, 0), (16, 7, 7, 64, 72, 7, 7, 1, 0), (3, 1, 1, 520, 130, 1, 1, 1, 0)]:
        d, P, Q, xb, _, wr = _conv_inputs(g, 11)
        q = oracle.quantize(wr)
        acc = oracle.conv_fwd(d, oracle.bf16_bits_to_f64(xb), q.codes, q.alpha.astype(np.float64))
        codes, alpha, _ = tbn.quantize(to_dev(wr))
        y = tbn.conv2d_fwd(tbn.ConvDesc(*g), bf16_dev(xb), codes, alpha, out_dtype=torch.float32)
        torch.cuda.synchronize()
        e = nerr(y.cpu().numpy(), acc)
        assert e <= 1e-4, "variant %d %s: %.3e" % (variant, g, e)


def test_fc_stream_weight_streaming_size(tbn):
    # 8192 -> 16384 at batch 1 (32 MiB of codes): sampled outputs against the oracle
    g = (1, 1, 1, 8192, 16384, 1, 1, 1, 0)
    d = oracle.ConvDesc(*g)
    xb = synth.normal_bf16(10, "wsx", (1, 1, 1, 8192))
    wr = synth.normal(10, "wsw", (16384, 8192), 1.0)
    codes, alpha, _ = tbn.quantize(to_dev(wr))
    y = tbn.conv2d_fwd(tbn.ConvDesc(*g), bf16_dev(xb), codes, alpha, out_dtype=torch.float32)
    torch.cuda.synchronize()
    idx = synth.sample_indices(10, "wsidx", 16384, 512)
    q = oracle.quantize(wr[idx])  # quantisation is per filter: the sampled filters alone
    sub = oracle.ConvDesc(1, 1, 1, 8192, len(idx), 1, 1, 1, 0)
    ref = oracle.conv_fwd(sub, oracle.bf16_bits_to_f64(xb), q.codes, q.alpha.astype(np.float64))
    e = nerr(y.cpu().numpy().reshape(-1)[idx], ref.reshape(-1))
    log("weight streaming 8192x16384, 512 sampled filters: %.3e" % e)
    assert e <= 1e-4


BWD_CASES = [c for c in CONV_CASES if c[7] == 1] + [(2, 8, 8, 64, 64, 3, 3, 1, 0), (2, 6, 6, 64, 64, 5, 5, 1, 4),
                                                    (4, 4, 4, 512, 10, 4, 4, 1, 0),   # 10-way classifier over 4x4
                                                    (3, 9, 9, 16, 13, 3, 3, 1, 1)]    # 13 filters: 16-channel copy


@pytest.mark.parametrize("g", BWD_CASES)
def test_bwd_data_parity(tbn, g):
    log("bwd_data %s" % (g,))
    d, P, Q, _, dyb, wr = _conv_inputs(g, 4)
    q = oracle.quantize(wr)
    ref = oracle.conv_bwd_data(d, oracle.bf16_bits_to_f64(dyb), q.codes, q.alpha.astype(np.float64))
    codes, alpha, _ = tbn.quantize(to_dev(wr))
    dx = tbn.conv2d_bwd_data(tbn.ConvDesc(*g), bf16_dev(dyb), codes, alpha, out_dtype=torch.float32)
    torch.cuda.synchronize()
    e = nerr(dx.cpu().numpy(), ref)
    log("  normalised max error %.3e" % e)
    assert e <= TOL


@pytest.mark.parametrize("g", CONV_CASES)
@pytest.mark.parametrize("accumulate", [False, True])
def test_bwd_weight_parity(tbn, g, accumulate):
    log("bwd_weight %s accumulate=%s" % (g, accumulate))
    d, P, Q, xb, dyb, _ = _conv_inputs(g, 5)
    ref = oracle.conv_bwd_weight(d, oracle.bf16_bits_to_f64(xb), oracle.bf16_bits_to_f64(dyb))
    prior = synth.normal(5, "prior%s" % (g,), ref.shape, 1.0)
    dw0 = to_dev(prior) if accumulate else None
    dw = tbn.conv2d_bwd_weight(tbn.ConvDesc(*g), bf16_dev(xb), bf16_dev(dyb), dw=dw0, accumulate=accumulate)
    torch.cuda.synchronize()
    want = ref + prior if accumulate else ref
    e = nerr(dw.cpu().numpy(), want)
    log("  normalised max error %.3e" % e)
    assert e <= 1e-4


@pytest.mark.parametrize("cfg,pix,pf", [(0, 48, 0), (1, 32, 0), (1, 48, 0), (1, 64, 0), (1, 48, 3)])
def test_bwd_weight_tile_shapes(tbn, cfg, pix, pf, knobs):
    # every tile / stage geometry of the transposing-read weight-gradient kernels (the
    # 48-pixel stages do not divide the 64-pixel split ranges: the last stage of a range is
    # partial), and the optional L2 prefetch; stride-1 same-size layers with C % 256 == 0
    # take the linear copy addressing (ragged K, a pixel count that ends inside a stage's
    # pixel pairs, 1x1 and 5x5 filters, images narrower than the filter)
    knobs(wgrad_cfg=cfg, wgrad_pix=pix, wgrad_pf=pf)
    for g in [(2, 14, 14, 256, 256, 3, 3, 1, 1), (3, 12, 12, 128, 136, 3, 3, 2, 1), (5, 9, 7, 64, 96, 3, 3, 1, 1),
              (2, 16, 16, 64, 128, 1, 1, 2, 0), (2, 6, 7, 256, 136, 3, 3, 1, 1), (1, 5, 3, 512, 256, 3, 3, 1, 1),
              (3, 4, 5, 256, 264, 1, 1, 1, 0), (2, 7, 9, 256, 128, 5, 5, 1, 2), (1, 2, 2, 256, 128, 3, 3, 1, 1)]:
        d, P, Q, xb, dyb, _ = _conv_inputs(g, 5)
        ref = oracle.conv_bwd_weight(d, oracle.bf16_bits_to_f64(xb), oracle.bf16_bits_to_f64(dyb))
        dw = tbn.conv2d_bwd_weight(tbn.ConvDesc(*g), bf16_dev(xb), bf16_dev(dyb))
        torch.cuda.synchronize()
        e = nerr(dw.cpu().numpy(), ref)
        log("bwd_weight cfg %d pix %d %s: %.3e" % (cfg, pix, g, e))
        assert e <= 1e-4


def test_sgd_parity(tbn):
    n = 1_000_003
    w = synth.normal(6, "w", (n,), 0.05)
    v = synth.normal(6, "v", (n,), 0.01)
    g = synth.normal(6, "g", (n,), 1.0)
    wr, vr = oracle.sgd(w, v, g, 0.1, 0.9, 1e-4)
    wt, vt = to_dev(w), to_dev(v)
    tbn.sgd_step(wt, vt, to_dev(g), 0.1, 0.9, 1e-4)
    torch.cuda.synchronize()
    assert nerr(wt.cpu().numpy(), wr) <= 1e-6
    assert nerr(vt.cpu().numpy(), vr) <= 1e-6


def test_repeat_runs_are_bitwise_identical(tbn):
    g = (2, 14, 14, 256, 256, 3, 3, 1, 1)
    _, _, _, xb, dyb, wr = _conv_inputs(g, 7)
    desc = tbn.ConvDesc(*g)
    codes, alpha, _ = tbn.quantize(to_dev(wr))
    x, dy = bf16_dev(xb), bf16_dev(dyb)
    outs = []
    for _ in range(3):
        outs.append((tbn.conv2d_fwd(desc, x, codes, alpha).clone(),
                     tbn.conv2d_bwd_data(desc, dy, codes, alpha).clone(),
                     tbn.conv2d_bwd_weight(desc, x, dy).clone()))
    torch.cuda.synchronize()
    for o in outs[1:]:
        for a, b in zip(o, outs[0]):
            assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a.view(torch.int32),
                               b.view(torch.int16) if b.dtype == torch.bfloat16 else b.view(torch.int32))


SPLIT_CASES = [(2, 14, 14, 256, 256, 3, 3, 1, 1), (2, 15, 13, 64, 96, 3, 3, 1, 1), (3, 12, 12, 128, 136, 3, 3, 2, 1),
               (2, 7, 7, 512, 512, 3, 3, 1, 1),
               # filter counts that are not a multiple of 8 (a 10-way classifier as a 4x4 valid
               # convolution; a ragged 13)
               (3, 4, 4, 64, 10, 4, 4, 1, 0), (2, 9, 9, 16, 13, 3, 3, 1, 1)]


@pytest.mark.parametrize("splits", [1, 2, 7, 1000])
def test_reduction_splits(tbn, splits, knobs):
    # the reduction split into ranges summed by the epilogue kernel: fused epilogue (scale,
    # bias, bf16 residual, ReLU) and fp32 output of fwd, and bwd_data, against the oracle;
    # 1000 clamps to one 64-element stage per range
    knobs(conv_splits=splits)
    for g in SPLIT_CASES:
        log("splits %d %s" % (splits, g))
        d, P, Q, xb, dyb, wr = _conv_inputs(g, 9)
        k = g[4]
        q = oracle.quantize(wr)
        a64 = q.alpha.astype(np.float64)
        scale = synth.uniform(9, "sc", (k,), 0.5, 1.5)
        bias = synth.normal(9, "bi", (k,), 0.1)
        resb = synth.normal_bf16(9, "res", (g[0], P, Q, k))
        acc = oracle.conv_fwd(d, oracle.bf16_bits_to_f64(xb), q.codes, a64)
        ref = np.maximum(acc * scale.astype(np.float64) + bias + oracle.bf16_bits_to_f64(resb), 0.0)
        codes, alpha, _ = tbn.quantize(to_dev(wr))
        desc = tbn.ConvDesc(*g)
        y = tbn.conv2d_fwd(desc, bf16_dev(xb), codes, alpha, out_dtype=torch.bfloat16, scale=to_dev(scale),
                           bias=to_dev(bias), residual=bf16_dev(resb), relu=True)
        y32 = tbn.conv2d_fwd(desc, bf16_dev(xb), codes, alpha, out_dtype=torch.float32)
        torch.cuda.synchronize()
        e = nerr(y.float().cpu().numpy(), ref)
        assert e <= TOL, "fwd epilogue splits %d %s: %.3e" % (splits, g, e)
        e = nerr(y32.cpu().numpy(), acc)
        assert e <= 1e-4, "fwd splits %d %s: %.3e" % (splits, g, e)
        if g[7] == 1:
            dx = tbn.conv2d_bwd_data(desc, bf16_dev(dyb), codes, alpha, out_dtype=torch.float32)
            torch.cuda.synchronize()
            e = nerr(dx.cpu().numpy(), oracle.conv_bwd_data(d, oracle.bf16_bits_to_f64(dyb), q.codes, a64))
            assert e <= TOL, "bwd_data splits %d %s: %.3e" % (splits, g, e)


@pytest.mark.parametrize("tile,splits", [(21, 2), (22, 3), (23, 1000), (24, 7), (25, 2)])
def test_grouped_tiles_with_splits(tbn, tile, splits, knobs):
    # blocks of several four-wave groups (each reducing its own stage range) combined with a
    # reduction split over the grid: fused epilogue and bwd_data against the oracle
    knobs(conv_tile=tile, conv_splits=splits)
    for g in SPLIT_CASES:
        log("grouped tile %d splits %d %s" % (tile, splits, g))
        d, P, Q, xb, dyb, wr = _conv_inputs(g, 10)
        k = g[4]
        q = oracle.quantize(wr)
        a64 = q.alpha.astype(np.float64)
        scale = synth.uniform(10, "sc", (k,), 0.5, 1.5)
        bias = synth.normal(10, "bi", (k,), 0.1)
        resb = synth.normal_bf16(10, "res", (g[0], P, Q, k))
        acc = oracle.conv_fwd(d, oracle.bf16_bits_to_f64(xb), q.codes, a64)
        ref = np.maximum(acc * scale.astype(np.float64) + bias + oracle.bf16_bits_to_f64(resb), 0.0)
        codes, alpha, _ = tbn.quantize(to_dev(wr))
        desc = tbn.ConvDesc(*g)
        y = tbn.conv2d_fwd(desc, bf16_dev(xb), codes, alpha, out_dtype=torch.bfloat16, scale=to_dev(scale),
                           bias=to_dev(bias), residual=bf16_dev(resb), relu=True)
        torch.cuda.synchronize()
        e = nerr(y.float().cpu().numpy(), ref)
        assert e <= TOL, "fwd epilogue tile %d splits %d %s: %.3e" % (tile, splits, g, e)
        if g[7] == 1:
            dx = tbn.conv2d_bwd_data(desc, bf16_dev(dyb), codes, alpha, out_dtype=torch.float32)
            torch.cuda.synchronize()
            e = nerr(dx.cpu().numpy(), oracle.conv_bwd_data(d, oracle.bf16_bits_to_f64(dyb), q.codes, a64))
            assert e <= TOL, "bwd_data tile %d splits %d %s: %.3e" % (tile, splits, g, e)


TILE_CASES = [(2, 14, 14, 256, 256, 3, 3, 1, 1), (2, 15, 13, 64, 96, 3, 3, 1, 1), (2, 10, 10, 40, 24, 3, 3, 1, 1),
              (3, 12, 12, 128, 130, 3, 3, 2, 1), (2, 19, 17, 3, 40, 7, 7, 2, 3), (4, 1, 1, 512, 72, 1, 1, 1, 0),
              (3, 5, 5, 64, 80, 5, 5, 1, 0)]


@pytest.mark.parametrize("tile", [0, 1, 10, 11, 12, 13, 14, 16, 17, 18, 19, 20, 21, 22, 23, 24, 25, 30, 40])
def test_every_tile_shape(tbn, tile, knobs):
    # each tile shape of the convolution kernels against the oracle (fwd and bwd_data)
    knobs(conv_tile=tile)
    for g in TILE_CASES:
        log("tile %d %s" % (tile, g))
        d, P, Q, xb, dyb, wr = _conv_inputs(g, 8)
        q = oracle.quantize(wr)
        a64 = q.alpha.astype(np.float64)
        codes, alpha, _ = tbn.quantize(to_dev(wr))
        desc = tbn.ConvDesc(*g)
        y = tbn.conv2d_fwd(desc, bf16_dev(xb), codes, alpha, out_dtype=torch.float32)
        torch.cuda.synchronize()
        e = nerr(y.cpu().numpy(), oracle.conv_fwd(d, oracle.bf16_bits_to_f64(xb), q.codes, a64))
        assert e <= 1e-4, "fwd tile %d %s: %.3e" % (tile, g, e)
        if g[7] == 1:
            dx = tbn.conv2d_bwd_data(desc, bf16_dev(dyb), codes, alpha, out_dtype=torch.float32)
            torch.cuda.synchronize()
            e = nerr(dx.cpu().numpy(), oracle.conv_bwd_data(d, oracle.bf16_bits_to_f64(dyb), q.codes, a64))
            assert e <= TOL, "bwd_data tile %d %s: %.3e" % (tile, g, e)
