"""Pins for the oracle's convolutions, bf16 rounding and update step, all on the CPU.

The convolutions are pinned to library routines on the same definition (torch's fp64 CPU
conv2d and its autograd gradients, numpy matmul for 1x1 layers), to impulse responses,
and to the adjoint identities that tie the three passes together.  The update step is
pinned to torch.optim.SGD and to a hand-worked step; bf16 rounding to torch's own
fp32 -> bfloat16 conversion.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth

GEOMS = [
    # n, h, w, c, k, r, s, stride, pad
    (2, 7, 6, 1, 3, 5, 5, 1, 2),
    (1, 9, 9, 3, 5, 3, 3, 2, 1),
    (2, 8, 5, 4, 6, 3, 3, 1, 0),
    (1, 11, 10, 2, 4, 7, 7, 2, 3),
    (3, 5, 5, 8, 7, 1, 1, 1, 0),
    (2, 6, 7, 5, 3, 1, 1, 2, 0),
    (1, 4, 4, 6, 2, 4, 4, 1, 0),      # "valid" full-map conv, the FC-as-conv form
    (2, 6, 6, 3, 4, 3, 2, 3, 2),
]


def _problem(g, name):
    n, h, w, c, k, r, s, st, pd = g
    desc = oracle.ConvDesc(n, h, w, c, k, r, s, st, pd)
    P, Q = desc.out_dims()
    x = synth.normal(0, name + "x", (n, h, w, c)).astype(np.float64)
    wr = synth.normal(0, name + "w", (k, r * s * c), 1.2)
    q = oracle.quantize(wr)
    dy = synth.normal(0, name + "dy", (n, P, Q, k)).astype(np.float64)
    return desc, x, q, dy


def _torch_weight(desc, q):
    wd = q.alpha64[:, None] * q.codes.astype(np.float64)           # W^ = alpha W~
    wd = wd.reshape(desc.k, desc.r, desc.s, desc.c)
    return torch.from_numpy(np.ascontiguousarray(wd.transpose(0, 3, 1, 2)))  # KCRS


@pytest.mark.parametrize("g", GEOMS)
def test_fwd_matches_torch_conv2d(g):
    desc, x, q, _ = _problem(g, "fwd%s" % (g,))
    y = oracle.conv_fwd(desc, x, q.codes, q.alpha64)
    xt = torch.from_numpy(np.ascontiguousarray(x.transpose(0, 3, 1, 2)))
    ref = F.conv2d(xt, _torch_weight(desc, q), stride=desc.stride_h, padding=desc.pad_h)
    ref = ref.numpy().transpose(0, 2, 3, 1)
    assert y.shape == ref.shape
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("g", GEOMS)
def test_fwd_three_forms_of_eq1_agree(g):
    desc, x, q, _ = _problem(g, "forms%s" % (g,))
    y0 = oracle.conv_fwd(desc, x, q.codes, q.alpha64, form=0)
    y1 = oracle.conv_fwd(desc, x, q.codes, q.alpha64, form=1)
    y2 = oracle.conv_fwd(desc, x, q.codes, q.alpha64, form=2)
    assert np.allclose(y0, y1, rtol=1e-12, atol=1e-12)
    assert np.allclose(y0, y2, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("g", GEOMS)
def test_backward_matches_torch_autograd(g):
    desc, x, q, dy = _problem(g, "bwd%s" % (g,))
    xt = torch.from_numpy(np.ascontiguousarray(x.transpose(0, 3, 1, 2))).requires_grad_(True)
    wt = _torch_weight(desc, q).requires_grad_(True)
    yt = F.conv2d(xt, wt, stride=desc.stride_h, padding=desc.pad_h)
    yt.backward(torch.from_numpy(np.ascontiguousarray(dy.transpose(0, 3, 1, 2))))
    dx = oracle.conv_bwd_data(desc, dy, q.codes, q.alpha64)
    dw = oracle.conv_bwd_weight(desc, x, dy)
    assert np.allclose(dx, xt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-11)
    assert np.allclose(dw, wt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-11)


@pytest.mark.parametrize("g", GEOMS)
def test_adjoint_identities(g):
    # <fwd(x), dy> = <x, bwd_data(dy)> = <W^, bwd_weight(x, dy)>
    desc, x, q, dy = _problem(g, "adj%s" % (g,))
    y = oracle.conv_fwd(desc, x, q.codes, q.alpha64)
    dx = oracle.conv_bwd_data(desc, dy, q.codes, q.alpha64)
    dw = oracle.conv_bwd_weight(desc, x, dy)
    wd = (q.alpha64[:, None] * q.codes).reshape(dw.shape)
    a, b, c = np.sum(y * dy), np.sum(x * dx), np.sum(wd * dw)
    assert a == pytest.approx(b, rel=1e-11, abs=1e-10)
    assert a == pytest.approx(c, rel=1e-11, abs=1e-10)


def test_one_by_one_conv_is_matmul():
    n, h, w, c, k = 3, 4, 5, 6, 7
    desc = oracle.ConvDesc(n, h, w, c, k, 1, 1)
    x = synth.normal(0, "mmx", (n, h, w, c)).astype(np.float64)
    q = oracle.quantize(synth.normal(0, "mmw", (k, c), 1.0))
    y = oracle.conv_fwd(desc, x, q.codes, q.alpha64)
    Wd = q.alpha64[:, None] * q.codes
    assert np.allclose(y.reshape(-1, k), x.reshape(-1, c) @ Wd.T, rtol=1e-13, atol=1e-13)
    dy = synth.normal(0, "mmdy", (n, h, w, k)).astype(np.float64)
    dw = oracle.conv_bwd_weight(desc, x, dy)
    assert np.allclose(dw.reshape(k, c), dy.reshape(-1, k).T @ x.reshape(-1, c), rtol=1e-13, atol=1e-12)
    dx = oracle.conv_bwd_data(desc, dy, q.codes, q.alpha64)
    assert np.allclose(dx.reshape(-1, c), dy.reshape(-1, k) @ Wd, rtol=1e-13, atol=1e-12)


def test_impulse_reads_back_the_filter():
    # A single 1 at (h0, w0, c0) gives y[p, q, k] = alpha_k W~[k, h0-p+pad, w0-q+pad, c0]:
    # the filter, mirrored, at the output positions that see the impulse.
    n, h, w, c, k, r, s, pad = 1, 9, 9, 3, 4, 3, 5, 1
    desc = oracle.ConvDesc(n, h, w, c, k, r, s, 1, pad, pad_w=2)
    q = oracle.quantize(synth.normal(0, "imp", (k, r * s * c), 1.0))
    codes = q.codes.reshape(k, r, s, c)
    x = np.zeros((n, h, w, c))
    h0, w0, c0 = 4, 5, 2
    x[0, h0, w0, c0] = 1.0
    y = oracle.conv_fwd(desc, x, q.codes, q.alpha64)
    P, Q = desc.out_dims()
    for p in range(P):
        for qq in range(Q):
            rr, ss = h0 - p + pad, w0 - qq + 2
            for kk in range(k):
                want = q.alpha64[kk] * codes[kk, rr, ss, c0] if (0 <= rr < r and 0 <= ss < s) else 0.0
                assert y[0, p, qq, kk] == want


def test_box_filter_with_unit_scale():
    # With every code +1 and alpha = 1 the layer is a plain box sum over the window.
    n, h, w, c, k = 1, 6, 6, 2, 1
    desc = oracle.ConvDesc(n, h, w, c, k, 3, 3, 1, 1)
    x = synth.uniform(0, "box", (n, h, w, c)).astype(np.float64)
    y = oracle.conv_fwd(desc, x, np.ones((1, 18), np.int8), np.ones(1))
    xp = np.pad(x[0].sum(axis=-1), 1)
    want = np.array([[xp[i:i + 3, j:j + 3].sum() for j in range(6)] for i in range(6)])
    assert np.allclose(y[0, :, :, 0], want, rtol=1e-14, atol=1e-14)


@pytest.mark.parametrize("g", GEOMS)
def test_sampled_forms_match_full(g):
    n, h, w, c, k, r, s, st, pd = g
    desc = oracle.ConvDesc(*g)
    P, Q = desc.out_dims()
    xb = synth.normal_bf16(0, "sx%s" % (g,), (n, h, w, c))
    dyb = synth.normal_bf16(0, "sdy%s" % (g,), (n, P, Q, k))
    q = oracle.quantize(synth.normal(0, "sw%s" % (g,), (k, r * s * c), 1.0))
    x = oracle.bf16_bits_to_f64(xb)
    dy = oracle.bf16_bits_to_f64(dyb)
    y = oracle.conv_fwd(desc, x, q.codes, q.alpha64).ravel()
    dx = oracle.conv_bwd_data(desc, dy, q.codes, q.alpha64).ravel()
    dw = oracle.conv_bwd_weight(desc, x, dy).ravel()
    iy = synth.sample_indices(0, "iy", y.size, 50)
    ix = synth.sample_indices(0, "ix", dx.size, 50)
    iw = synth.sample_indices(0, "iw", dw.size, 50)
    assert np.allclose(oracle.conv_fwd_sampled(desc, xb, q.codes, q.alpha64, iy), y[iy], rtol=1e-13, atol=1e-13)
    assert np.allclose(oracle.conv_bwd_data_sampled(desc, dyb, q.codes, q.alpha64, ix), dx[ix], rtol=1e-13, atol=1e-13)
    assert np.allclose(oracle.conv_bwd_weight_sampled(desc, xb, dyb, iw), dw[iw], rtol=1e-13, atol=1e-12)


def test_bad_geometry_rejected():
    with pytest.raises(oracle.OracleError):
        oracle.ConvDesc(1, 2, 2, 1, 1, 5, 5, 1, 0).out_dims()
    with pytest.raises(oracle.OracleError):
        oracle.ConvDesc(0, 2, 2, 1, 1, 1, 1).out_dims()


def test_round_bf16_matches_torch():
    g = synth.rng(0, "rne")
    bits = g.integers(0, 2 ** 32, size=200000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    # exact ties (dropped half = 0x8000) with both parities of the kept part
    ties = ((g.integers(0, 2 ** 16, size=1000, dtype=np.uint64).astype(np.uint32) << 16) | 0x8000).view(np.float32)
    x = np.concatenate([x, ties[np.isfinite(ties)], np.array([0.0, -0.0, 1.0, 3.14159], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(oracle.round_bf16(x), ref)


def test_sgd_matches_torch_optimizer():
    n = 1000
    w0 = synth.normal(0, "sgdw", (n,), 0.05)
    grads = [synth.normal(0, "sgdg%d" % i, (n,), 1.0) for i in range(3)]
    wt = torch.nn.Parameter(torch.from_numpy(w0.astype(np.float64)))
    opt = torch.optim.SGD([wt], lr=0.1, momentum=0.9, weight_decay=1e-4, dampening=0, nesterov=False)
    w, v = w0.astype(np.float64), np.zeros(n)
    for gr in grads:
        wt.grad = torch.from_numpy(gr.astype(np.float64))
        opt.step()
        w, v = oracle.sgd(w, v, gr, 0.1, 0.9, 1e-4)
    assert np.allclose(w, wt.detach().numpy(), rtol=1e-14, atol=1e-16)


def test_sgd_hand_step():
    # w = 1, v = 0.5, g = 2, eta = 0.1, mu = 0.9, lambda = 0.01:
    # v = 0.45 + 2.01 = 2.46; w = 1 - 0.246 = 0.754
    w, v = oracle.sgd([1.0], [0.5], [2.0], 0.1, 0.9, 0.01)
    assert v[0] == pytest.approx(2.46, abs=1e-15) and w[0] == pytest.approx(0.754, abs=1e-15)


@pytest.mark.parametrize("g", GEOMS)
def test_dense_fwd_matches_torch_conv2d(g):
    # the full-precision layer: Eq. (1) with real filters, pinned to torch's fp64 conv2d
    n, h, w, c, k, r, s, st, pd = g
    desc = oracle.ConvDesc(*g)
    x = synth.normal(0, "dx%s" % (g,), (n, h, w, c)).astype(np.float64)
    wr = synth.normal(0, "dw%s" % (g,), (k, r, s, c)).astype(np.float64)
    y = oracle.conv_fwd_dense(desc, x, wr)
    xt = torch.from_numpy(np.ascontiguousarray(x.transpose(0, 3, 1, 2)))
    wt = torch.from_numpy(np.ascontiguousarray(wr.transpose(0, 3, 1, 2)))
    ref = F.conv2d(xt, wt, stride=st, padding=pd).numpy().transpose(0, 2, 3, 1)
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_dense_fwd_with_approximate_filters_equals_two_bit_fwd():
    # real filters alpha W~ give exactly the two-bit layer (dense form of Eq. 1)
    g = (2, 9, 8, 5, 6, 3, 3, 1, 1)
    desc, x, q, _ = _problem(g, "dense2bit")
    wd = q.alpha64[:, None] * q.codes.astype(np.float64)
    y = oracle.conv_fwd_dense(desc, x, wd)
    assert np.allclose(y, oracle.conv_fwd(desc, x, q.codes, q.alpha64, form=2), rtol=0, atol=1e-13)


def test_sgd_f32_hand_step_exact():
    # every product and sum below is exact in fp32, so the fused form must land on it:
    # v = 0.5 * 0.25 + (0.5 + 0.25 * 1.5) = 1.0;  w = 1.5 - 0.5 * 1.0 = 1.0
    w, v = oracle.sgd_f32([1.5], [0.25], [0.5], 0.5, 0.5, 0.25)
    assert v[0] == 1.0 and w[0] == 1.0
    assert w.dtype == np.float32


def test_sgd_f32_single_rounding_per_fused_op():
    # Each update line is one fused multiply-add: round(a * b + c) once.  Extended
    # precision holds a fp32 product exactly (48 bits) and the sum to 64 bits, so rounding
    # that to fp32 reproduces the single rounding for these inputs.
    n = 20000
    w0 = synth.normal(0, "sgdf32w", (n,), 1.0)
    v0 = synth.normal(0, "sgdf32v", (n,), 0.3)
    g0 = synth.normal(0, "sgdf32g", (n,), 1.0)
    lr, mu, wd = np.float32(0.1), np.float32(0.9), np.float32(1e-4)
    w, v = oracle.sgd_f32(w0, v0, g0, float(lr), float(mu), float(wd))
    L = np.longdouble
    assert np.finfo(L).nmant >= 63
    inner = (L(wd) * w0.astype(L) + g0.astype(L)).astype(np.float32)
    v_ref = (L(mu) * v0.astype(L) + inner.astype(L)).astype(np.float32)
    w_ref = (-L(lr) * v_ref.astype(L) + w0.astype(L)).astype(np.float32)
    assert np.array_equal(v.view(np.int32), v_ref.view(np.int32))
    assert np.array_equal(w.view(np.int32), w_ref.view(np.int32))
    # and it is the fp64 step up to fp32 rounding
    w64, v64 = oracle.sgd(w0, v0, g0, float(lr), float(mu), float(wd))
    assert np.max(np.abs(w - w64)) <= 4 * np.finfo(np.float32).eps * np.max(np.abs(w64))


def test_results_do_not_depend_on_thread_count():
    # the CPU baseline times the oracle single-threaded and on all cores; every output element
    # is one thread's fixed-order sum, so the results are bit-identical either way
    g = (3, 9, 8, 16, 24, 3, 3, 1, 1)
    d = oracle.ConvDesc(*g)
    x = synth.normal(20, "tx", g[:4]).astype(np.float64)
    w = synth.normal(20, "tw", (24, 9 * 16), 0.7)
    q = oracle.quantize(w)
    P, Q = d.out_dims()
    dy = synth.normal(20, "tdy", (3, P, Q, 24)).astype(np.float64)
    n0 = oracle.max_threads()
    outs = []
    for n in (1, max(2, n0)):
        oracle.set_threads(n)
        outs.append((oracle.conv_fwd(d, x, q.codes, q.alpha.astype(np.float64)),
                     oracle.conv_bwd_data(d, dy, q.codes, q.alpha.astype(np.float64)),
                     oracle.conv_bwd_weight(d, x, dy)))
    oracle.set_threads(n0)
    for a, b in zip(*outs):
        assert np.array_equal(a, b)
