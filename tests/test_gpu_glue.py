"""GPU parity of the layers around the two-bit convolutions (max pooling, global average
pooling, batch normalisation in training form, ReLU backward, softmax cross-entropy)
against the fp64 oracle.  Pooling values and argmax positions are bit-exact (the maximum of
bf16 values is a bf16 value); the rest within the normalised 1e-2 bar."""
import numpy as np
import pytest
import torch

import oracle
import synth
from test_gpu_parity import bf16_dev, log, nerr, to_dev

pytestmark = pytest.mark.gpu


def _bits_to_f64(t):
    return oracle.bf16_bits_to_f64(t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16))


@pytest.mark.parametrize("shape,k,s,p", [((2, 112, 112, 64), 3, 2, 1), ((4, 28, 28, 32), 2, 2, 0),
                                          ((3, 9, 7, 5), 3, 2, 1), ((2, 14, 14, 64), 2, 2, 0),
                                          ((2, 15, 17, 16), 3, 2, 1), ((3, 7, 9, 8), 3, 1, 1),
                                          ((2, 11, 13, 24), 2, 2, 0)])
def test_maxpool(tbn, shape, k, s, p):
    log("maxpool %s k%d s%d p%d" % (shape, k, s, p))
    xb = synth.normal_bf16(10, "mp%s" % (shape,), shape)
    # ReLU-like input: many exact zeros, so ties are exercised
    xb = np.where(xb & 0x8000, np.uint16(0), xb).astype(np.uint16)
    x = oracle.bf16_bits_to_f64(xb)
    y_ref, arg_ref = oracle.maxpool_fwd(x, k, s, p)
    y, arg = tbn.maxpool2d_fwd(bf16_dev(xb), k, s, p, want_argmax=True)
    torch.cuda.synchronize()
    assert np.array_equal(_bits_to_f64(y), y_ref)
    N, H, W, C = shape
    pos = arg_ref // C % (H * W)  # oracle's flat NHWC index -> spatial position h*W + w
    assert np.array_equal(arg.cpu().numpy(), np.where(arg_ref < 0, -1, pos))
    dyb = synth.normal_bf16(10, "mpdy%s" % (shape,), y_ref.shape)
    dx_ref = oracle.maxpool_bwd(oracle.bf16_bits_to_f64(dyb), arg_ref, shape, k, s, p)
    dx = tbn.maxpool2d_bwd(bf16_dev(dyb), arg, shape, k, s, p, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert nerr(dx.cpu().numpy(), dx_ref) <= 1e-6


@pytest.mark.parametrize("shape", [(64, 7, 7, 512), (3, 1, 1, 16), (2, 3, 5, 24), (5, 4, 4, 13), (1, 9, 11, 3)])
def test_avgpool(tbn, shape):
    # 16-byte channel groups (C % 8 == 0, fewer or more positions than the 8 lanes that
    # share a group) and the per-channel path (C % 8 != 0)
    xb = synth.normal_bf16(10, "ap%s" % (shape,), shape)
    ref = oracle.avgpool_global(oracle.bf16_bits_to_f64(xb))
    y = tbn.avgpool_global(bf16_dev(xb), out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert nerr(y.cpu().numpy(), ref) <= 1e-5
    yb = tbn.avgpool_global(bf16_dev(xb))
    torch.cuda.synchronize()
    assert nerr(oracle.bf16_bits_to_f64(yb.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)), ref) <= 1e-2


@pytest.mark.parametrize("shape,relu", [((8, 16, 16, 128), True), ((4, 8, 8, 24), False), ((2, 5, 5, 13), True),
                                        ((64, 32, 32, 32), True),    # 65536 rows: many row chunks
                                        ((4, 80, 80, 128), True),    # 200 row chunks: batched and tail sums
                                        ((2, 3, 3, 2056), False),    # more than 256 groups of 8 channels
                                        ((3, 7, 7, 300), True)])     # 300 scalar channels: two slices
def test_batchnorm_train(tbn, shape, relu):
    log("batchnorm %s relu=%s" % (shape, relu))
    C = shape[-1]
    xb = synth.normal_bf16(11, "bnx%s" % (shape,), shape, 2.0)
    g = synth.uniform(11, "bng%s" % (shape,), (C,), 0.5, 1.5)
    b = synth.normal(11, "bnb%s" % (shape,), (C,), 0.1)
    dyb = synth.normal_bf16(11, "bndy%s" % (shape,), shape)
    x = oracle.bf16_bits_to_f64(xb)
    y_ref, m_ref, v_ref = oracle.bn_train_fwd(x, g, b)
    if relu:
        y_ref = np.maximum(y_ref, 0)
    y, mean, inv_std = tbn.batchnorm_train_fwd(bf16_dev(xb), to_dev(g), to_dev(b), relu=relu)
    torch.cuda.synchronize()
    assert nerr(mean.cpu().numpy(), m_ref) <= 1e-5
    assert nerr(inv_std.cpu().numpy(), 1 / np.sqrt(v_ref + 1e-5)) <= 1e-5
    assert nerr(y.float().cpu().numpy(), y_ref) <= 1e-2
    # backward through the GPU's own bf16 output (teacher-forced ReLU mask)
    dy = oracle.bf16_bits_to_f64(dyb)
    if relu:
        dy = dy * (_bits_to_f64(y) > 0)
    dx_ref, dg_ref, db_ref = oracle.bn_train_bwd(x, dy, g)
    dx, dg, db = tbn.batchnorm_train_bwd(bf16_dev(xb), y, bf16_dev(dyb), mean, inv_std, to_dev(g), relu=relu)
    torch.cuda.synchronize()
    assert nerr(dg.cpu().numpy(), dg_ref) <= 1e-3
    assert nerr(db.cpu().numpy(), db_ref) <= 1e-3
    assert nerr(dx.float().cpu().numpy(), dx_ref) <= 1e-2


@pytest.mark.parametrize("count", [1000, 1003, 5, 4096 * 8 + 7])
def test_relu_bwd(tbn, count):
    # 8 elements per thread, a ragged tail element by element; ReLU'(0) = 0 (zeros and
    # negative zeros in y)
    yb = synth.normal_bf16(12, "ry%d" % count, (count,))
    yb = np.where(yb & 0x8000, np.uint16(0), yb).astype(np.uint16)
    yb[::7] = 0x8000  # -0.0
    dyb = synth.normal_bf16(12, "rdy%d" % count, (count,))
    dx = tbn.relu_bwd(bf16_dev(yb), bf16_dev(dyb))
    torch.cuda.synchronize()
    want = np.where(oracle.bf16_bits_to_f64(yb) > 0, oracle.bf16_bits_to_f64(dyb), 0.0)
    assert np.array_equal(_bits_to_f64(dx), want)


@pytest.mark.parametrize("N,K", [(256, 10), (128, 10), (3, 1000), (5000, 10)])
def test_softmax_xent(tbn, N, K):
    z = synth.normal(12, "z%d" % N, (N, K), 3.0)
    lab = synth.labels(12, "l%d" % N, N, K)
    loss_ref, dz_ref = oracle.softmax_xent(z.astype(np.float64), lab)
    loss, dz = tbn.softmax_xent(to_dev(z), to_dev(lab.astype(np.int32)))
    torch.cuda.synchronize()
    assert float(loss.item()) == pytest.approx(loss_ref, rel=1e-5)
    assert nerr(dz.float().cpu().numpy(), dz_ref) <= 1e-2


def test_softmax_xent_out_of_range_labels(tbn):
    # a label outside [0, classes) is not bounds-checked before the launch; the kernel gives
    # that sample a NaN loss and the gradient softmax(z)/n (no one-hot term) and reads
    # nothing outside its row; the other samples are unaffected
    N, K = 6, 10
    z = synth.normal(12, "zbad", (N, K), 3.0)
    lab = synth.labels(12, "lbad", N, K).astype(np.int32)
    bad = lab.copy()
    bad[1], bad[4] = -1, K
    loss, dz = tbn.softmax_xent(to_dev(z), to_dev(bad))
    torch.cuda.synchronize()
    assert np.isnan(float(loss.item()))
    zz = z.astype(np.float64)
    p = np.exp(zz - zz.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    want = p.copy()
    ok = np.array([i not in (1, 4) for i in range(N)])
    want[np.arange(N)[ok], bad[ok]] -= 1.0
    want /= N
    assert nerr(dz.float().cpu().numpy(), want) <= 1e-2
