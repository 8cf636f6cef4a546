"""GPU parity of the three contractions on randomly drawn small layer shapes (derandomised
hypothesis search, so every run draws the same cases): strides 1 and 2, padding 0-3, odd
channel and filter counts (C = 1 and 3 take the thin-input forward and the channel-padded
filter gradient, K % 8 != 0 the filter-padded gradients), filter and element counts that are
not multiples of 64.  Same bars as the parity suite: forward with fp32 output within 1e-4,
the backward passes within 1e-2 (normalised max error) of the fp64 oracle.
"""
import numpy as np
import pytest
import torch
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import synth
from test_gpu_parity import bf16_dev, log, nerr, to_dev

pytestmark = pytest.mark.gpu

CHANNELS = [1, 2, 3, 5, 8, 16, 24, 40, 64, 72]


@st.composite
def layer(draw):
    r = draw(st.integers(1, 5))
    s = draw(st.integers(1, 5))
    pad = draw(st.integers(0, 3))
    stride = draw(st.integers(1, 2))
    h = draw(st.integers(max(1, r - 2 * pad), 12))
    w = draw(st.integers(max(1, s - 2 * pad), 12))
    n = draw(st.integers(1, 3))
    c = draw(st.sampled_from(CHANNELS))
    k = draw(st.integers(1, 80))
    return (n, h, w, c, k, r, s, stride, pad)


_SETTINGS = settings(max_examples=30, derandomize=True, deadline=None, database=None,
                     suppress_health_check=[HealthCheck.too_slow, HealthCheck.function_scoped_fixture])


def _inputs(g):
    n, h, w, c, k, r, s, st_, pd = g
    d = oracle.ConvDesc(*g)
    P, Q = d.out_dims()
    xb = synth.normal_bf16(9, "rx%s" % (g,), (n, h, w, c))
    dyb = synth.normal_bf16(9, "rdy%s" % (g,), (n, P, Q, k))
    wr = synth.normal(9, "rw%s" % (g,), (k, r * s * c), 1.0)
    return d, xb, dyb, wr


@_SETTINGS
@given(g=layer())
def test_random_shape_forward(tbn, g):
    log("random fwd %s" % (g,))
    d, xb, _, wr = _inputs(g)
    q = oracle.quantize(wr)
    ref = oracle.conv_fwd(d, oracle.bf16_bits_to_f64(xb), q.codes, q.alpha.astype(np.float64))
    codes, alpha, _ = tbn.quantize(to_dev(wr))
    y = tbn.conv2d_fwd(tbn.ConvDesc(*g), bf16_dev(xb), codes, alpha, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert nerr(y.cpu().numpy(), ref) <= 1e-4


@_SETTINGS
@given(g=layer())
def test_random_shape_backward(tbn, g):
    log("random bwd %s" % (g,))
    d, xb, dyb, wr = _inputs(g)
    desc = tbn.ConvDesc(*g)
    x64, dy64 = oracle.bf16_bits_to_f64(xb), oracle.bf16_bits_to_f64(dyb)
    dw = tbn.conv2d_bwd_weight(desc, bf16_dev(xb), bf16_dev(dyb))
    torch.cuda.synchronize()
    assert nerr(dw.cpu().numpy(), oracle.conv_bwd_weight(d, x64, dy64)) <= 1e-2
    if g[7] == 1:  # backward-data is defined for stride 1
        q = oracle.quantize(wr)
        codes, alpha, _ = tbn.quantize(to_dev(wr))
        dx = tbn.conv2d_bwd_data(desc, bf16_dev(dyb), codes, alpha, out_dtype=torch.float32)
        torch.cuda.synchronize()
        assert nerr(dx.cpu().numpy(), oracle.conv_bwd_data(d, dy64, q.codes, q.alpha.astype(np.float64))) <= 1e-2
