"""Pins of the oracle's whole training iterations (oracle/nets.py) against torch fp64 autograd.

The oracle composes its own operations into one iteration of Algorithm 1 (quantise, forward,
softmax cross-entropy, backward through the approximate filters, straight-through filter
gradients, SGD with momentum and weight decay).  Here the same network is written in torch
with the approximate filters alpha * W~ (from the oracle's quantisation, itself pinned in
test_oracle_quantize.py) as leaf tensors; autograd's loss, gradients with respect to those
filters (the straight-through gradients of Sec. 3) and torch's SGD step must agree with the
oracle to fp64 rounding.  A wrong layer order, a dropped ReLU or BN term, a transposed filter
or a mis-routed pooling gradient fails here.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth
from oracle import nets

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")


def _nchw_filter(wflat, cout, k, cin):
    # [K][R*S*C] (KRSC) -> [K][C][R][S]
    return torch.from_numpy(np.ascontiguousarray(wflat.reshape(cout, k, k, cin).transpose(0, 3, 1, 2)))


def _krsc(g, cout, k, cin):
    return g.detach().numpy().transpose(0, 2, 3, 1).reshape(cout, k * k * cin)


def _sgd_torch(w, g, lr, wd):
    p = torch.nn.Parameter(torch.from_numpy(np.asarray(w, np.float64).copy()))
    opt = torch.optim.SGD([p], lr=lr, momentum=nets.MOMENTUM, weight_decay=wd)
    p.grad = torch.from_numpy(np.asarray(g, np.float64).reshape(p.shape).copy())
    opt.step()
    return p.detach().numpy()


def test_lenet_iteration_matches_torch_autograd():
    N = 2
    x = synth.uniform(2, "pin_x", (N, 28, 28, 1)).astype(np.float64)
    lab = synth.labels(2, "pin_lab", N, 10)
    weights, vel = {}, {}
    for name, cin, cout, k, *_ in nets.LENET:
        # N(0, 0.7^2) real filters: both code magnitudes occur
        weights[name] = synth.normal(2, "pin_" + name, (cout, k * k * cin), 0.7)
        vel[name] = np.zeros_like(weights[name], dtype=np.float64)
    loss, new_w, _, grads = nets.lenet_iteration(x, lab, weights, vel, 0.1)

    leaves = {}
    for name, cin, cout, k, *_ in nets.LENET:
        q = oracle.quantize(weights[name])
        what = q.codes.astype(np.float64) * q.alpha.astype(np.float64)[:, None]
        leaves[name] = _nchw_filter(what, cout, k, cin).requires_grad_(True)
    h = torch.from_numpy(x.transpose(0, 3, 1, 2).copy())
    for name, cin, cout, k, st, pd, relu, pool in nets.LENET:
        h = F.conv2d(h, leaves[name], stride=st, padding=pd)
        if relu:
            h = F.relu(h)
        if pool:
            h = F.max_pool2d(h, 2, 2)
    tl = F.cross_entropy(h.reshape(N, 10), torch.from_numpy(lab.astype(np.int64)))
    tl.backward()
    assert loss == pytest.approx(float(tl), rel=1e-12)
    for name, cin, cout, k, *_ in nets.LENET:
        g_ref = _krsc(leaves[name].grad, cout, k, cin)
        assert np.max(np.abs(grads[name] - g_ref)) <= 1e-12 * max(1.0, np.max(np.abs(g_ref))), name
        w_ref = _sgd_torch(weights[name], g_ref, 0.1, nets.WEIGHT_DECAY)
        assert np.max(np.abs(new_w[name] - w_ref)) <= 1e-12, name


def test_vgg_iteration_matches_torch_autograd():
    N = 2
    x = synth.normal(3, "pin_x", (N, 32, 32, 3)).astype(np.float64)
    lab = synth.labels(3, "pin_lab", N, 10)
    weights, vel, bn, bnv = {}, {}, {}, {}
    for name, cin, cout, _ in nets.VGG:
        weights[name] = synth.normal(3, "pin_" + name, (cout, 9 * cin), 0.7)
        vel[name] = np.zeros((cout, 9 * cin))
        bn[name] = (synth.uniform(3, "pin_g" + name, (cout,), 0.5, 1.5).astype(np.float64),
                    synth.normal(3, "pin_b" + name, (cout,), 0.1).astype(np.float64))
        bnv[name] = (np.zeros(cout), np.zeros(cout))
    weights["fc"] = synth.normal(3, "pin_fc", (10, 16 * 512), 0.7)
    vel["fc"] = np.zeros((10, 16 * 512))
    loss, new_w, _, new_bn, _, grads = nets.vgg_iteration(x, lab, weights, vel, bn, bnv, 0.1)

    leaves, gam, bet = {}, {}, {}
    for i, (name, cin, cout, _) in enumerate(nets.VGG):
        if i == 0:
            what = oracle.round_bf16(weights[name])
        else:
            q = oracle.quantize(weights[name])
            what = q.codes.astype(np.float64) * q.alpha.astype(np.float64)[:, None]
        leaves[name] = _nchw_filter(what, cout, 3, cin).requires_grad_(True)
        gam[name] = torch.from_numpy(bn[name][0].copy()).requires_grad_(True)
        bet[name] = torch.from_numpy(bn[name][1].copy()).requires_grad_(True)
    qf = oracle.quantize(weights["fc"])
    leaves["fc"] = _nchw_filter(qf.codes.astype(np.float64) * qf.alpha.astype(np.float64)[:, None], 10, 4,
                                512).requires_grad_(True)
    h = torch.from_numpy(x.transpose(0, 3, 1, 2).copy())
    for name, cin, cout, pool in nets.VGG:
        h = F.conv2d(h, leaves[name], padding=1)
        h = F.relu(F.batch_norm(h, None, None, gam[name], bet[name], training=True, eps=1e-5))
        if pool:
            h = F.max_pool2d(h, 2, 2)
    logits = F.conv2d(h, leaves["fc"]).reshape(N, 10)
    tl = F.cross_entropy(logits, torch.from_numpy(lab.astype(np.int64)))
    tl.backward()
    assert loss == pytest.approx(float(tl), rel=1e-10)
    for name, cin, cout, _ in nets.VGG + [("fc", 512, 10, None)]:
        k = 4 if name == "fc" else 3
        g_ref = _krsc(leaves[name].grad, cout, k, cin)
        assert np.max(np.abs(grads[name] - g_ref)) <= 1e-9 * max(1.0, np.max(np.abs(g_ref))), name
        w_ref = _sgd_torch(weights[name], g_ref, 0.1, nets.WEIGHT_DECAY)
        assert np.max(np.abs(new_w[name] - w_ref)) <= 1e-9, name
    for name, *_ in nets.VGG:
        g_ref = _sgd_torch(bn[name][0], gam[name].grad.numpy(), 0.1, 0.0)
        b_ref = _sgd_torch(bn[name][1], bet[name].grad.numpy(), 0.1, 0.0)
        assert np.max(np.abs(new_bn[name][0] - g_ref)) <= 1e-9, name
        assert np.max(np.abs(new_bn[name][1] - b_ref)) <= 1e-9, name
