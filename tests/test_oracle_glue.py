"""Pins for the oracle's layers around the two-bit convolutions (pooling, batch
normalisation, softmax cross-entropy), each against torch's fp64 CPU routine of the same
textbook definition and a hand-worked tie case."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth


def nchw(a):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, np.float64).transpose(0, 3, 1, 2)))


def nhwc(t):
    return t.detach().numpy().transpose(0, 2, 3, 1)


@pytest.mark.parametrize("shape,k,s,p", [((2, 9, 9, 5), 3, 2, 1), ((3, 8, 8, 4), 2, 2, 0),
                                          ((1, 112, 112, 3), 3, 2, 1), ((2, 7, 6, 2), 2, 2, 0)])
def test_maxpool_matches_torch(shape, k, s, p):
    x = synth.normal(0, "mp%s" % (shape,), shape).astype(np.float64)
    y, arg = oracle.maxpool_fwd(x, k, s, p)
    xt = nchw(x).requires_grad_(True)
    yt = F.max_pool2d(xt, k, s, p)
    assert np.array_equal(y, nhwc(yt))
    dy = synth.normal(0, "mpdy%s" % (shape,), y.shape).astype(np.float64)
    yt.backward(nchw(dy))
    dx = oracle.maxpool_bwd(dy, arg, shape, k, s, p)
    assert np.allclose(dx, nhwc(xt.grad), rtol=1e-15, atol=1e-15)


def test_maxpool_ties_go_to_first():
    # 2x2 window of zeros (a ReLU output): the gradient goes to the top-left element only
    x = np.zeros((1, 2, 2, 1))
    y, arg = oracle.maxpool_fwd(x, 2, 2, 0)
    assert y[0, 0, 0, 0] == 0.0 and arg[0, 0, 0, 0] == 0
    dx = oracle.maxpool_bwd(np.ones((1, 1, 1, 1)), arg, x.shape, 2, 2, 0)
    assert dx.ravel().tolist() == [1.0, 0.0, 0.0, 0.0]


def test_avgpool_global():
    x = synth.normal(0, "ap", (3, 7, 7, 16)).astype(np.float64)
    assert np.allclose(oracle.avgpool_global(x), x.mean(axis=(1, 2)), rtol=1e-14, atol=1e-15)


def test_bn_infer_matches_torch():
    C = 12
    x = synth.normal(0, "bnx", (2, 5, 5, C)).astype(np.float64)
    g, b = synth.uniform(0, "g", (C,), 0.5, 1.5), synth.normal(0, "b", (C,), 0.1)
    m, v = synth.normal(0, "m", (C,), 0.1), synth.uniform(0, "v", (C,), 0.5, 1.5)
    y = oracle.bn_infer(x, g, b, m, v)
    ref = F.batch_norm(nchw(x), torch.from_numpy(m.astype(np.float64)), torch.from_numpy(v.astype(np.float64)),
                       torch.from_numpy(g.astype(np.float64)), torch.from_numpy(b.astype(np.float64)),
                       training=False, eps=1e-5)
    assert np.allclose(y, nhwc(ref), rtol=1e-13, atol=1e-13)


def test_bn_train_matches_torch_autograd():
    C = 6
    x = synth.normal(0, "btx", (4, 5, 3, C), 2.0).astype(np.float64)
    g = synth.uniform(0, "btg", (C,), 0.5, 1.5).astype(np.float64)
    b = synth.normal(0, "btb", (C,), 0.1).astype(np.float64)
    dy = synth.normal(0, "btdy", x.shape).astype(np.float64)
    y, mean, var = oracle.bn_train_fwd(x, g, b)
    xt = nchw(x).requires_grad_(True)
    gt = torch.from_numpy(g).requires_grad_(True)
    bt = torch.from_numpy(b).requires_grad_(True)
    yt = F.batch_norm(xt, None, None, gt, bt, training=True, eps=1e-5)
    assert np.allclose(y, nhwc(yt), rtol=1e-12, atol=1e-12)
    assert np.allclose(mean, x.reshape(-1, C).mean(0), rtol=1e-13)
    assert np.allclose(var, x.reshape(-1, C).var(0), rtol=1e-12)
    yt.backward(nchw(dy))
    dx, dg, db = oracle.bn_train_bwd(x, dy, g)
    assert np.allclose(dx, nhwc(xt.grad), rtol=1e-10, atol=1e-12)
    assert np.allclose(dg, gt.grad.numpy(), rtol=1e-11, atol=1e-12)
    assert np.allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_softmax_xent_matches_torch():
    N, K = 16, 10
    z = synth.normal(0, "z", (N, K), 3.0).astype(np.float64)
    y = synth.labels(0, "y", N, K)
    loss, dz = oracle.softmax_xent(z, y)
    zt = torch.from_numpy(z).requires_grad_(True)
    lt = F.cross_entropy(zt, torch.from_numpy(y))
    lt.backward()
    assert loss == pytest.approx(lt.item(), rel=1e-13)
    assert np.allclose(dz, zt.grad.numpy(), rtol=1e-12, atol=1e-15)


def test_learning_rate_schedule():
    # Sec. 4: 0.1, divided by 10 at epochs 30, 40 and 50
    from paper_1701_00485_amd.networks import lr_at
    assert [lr_at(e) for e in (0, 29, 30, 39, 40, 49, 50, 57)] == pytest.approx(
        [0.1, 0.1, 0.01, 0.01, 1e-3, 1e-3, 1e-4, 1e-4])
