"""fp64 oracle of whole training iterations of the two small workload networks.

TEST INFRASTRUCTURE ONLY (like the rest of ``oracle/``): used by the tests and by the CPU
baseline of the benchmark, never by the product library.

One iteration of Algorithm 1 (Sec. 3) composed from the oracle's own operations, in exact
fp64 with no intermediate rounding: quantise every two-bit layer (Eq. 3-5), forward pass
with the approximate filters (Eq. 1), softmax cross-entropy averaged over the batch,
backward pass through the approximate filters (both passes use them, Sec. 3), the gradient
with respect to each approximate filter applied unchanged to its real filter
(straight-through), then SGD with momentum 0.9 and weight decay 1e-4 (Sec. 4; no weight
decay on batch-normalisation parameters).

Networks (the layer lists of the MNIST- and CIFAR-shaped workloads):
  LeNet:  conv 5x5 1->32 pad 2, ReLU, max pool 2; conv 5x5 32->64 pad 2, ReLU, max pool 2;
          FC 3136->512 (7x7 valid convolution), ReLU; FC 512->10.  Every layer two-bit.
  VGG:    conv 3x3 3->128 (full precision, filters rounded to bf16), then two-bit 3x3 convs
          128-256-256-512-512 (max pool 2 after every second conv), each conv followed by
          training-form batch normalisation and ReLU; FC 8192->10 (4x4 valid convolution).
"""
from __future__ import annotations

import numpy as np

from . import (ConvDesc, bn_train_bwd, bn_train_fwd, conv_bwd_data, conv_bwd_weight, conv_fwd,
               conv_fwd_dense, maxpool_bwd, maxpool_fwd, quantize, round_bf16, sgd, softmax_xent)

MOMENTUM, WEIGHT_DECAY = 0.9, 1e-4

# (name, cin, cout, kernel, stride, pad, relu, max pool after)
LENET = [("conv1", 1, 32, 5, 1, 2, True, True), ("conv2", 32, 64, 5, 1, 2, True, True),
         ("fc1", 64, 512, 7, 1, 0, True, False), ("fc2", 512, 10, 1, 1, 0, False, False)]

# (name, cin, cout, max pool after); 3x3, stride 1, pad 1; the FC layer follows
VGG = [("conv1", 3, 128, False), ("conv2", 128, 128, True), ("conv3", 128, 256, False),
       ("conv4", 256, 256, True), ("conv5", 256, 512, False), ("conv6", 512, 512, True)]


def _desc(x, cin, cout, k, stride, pad):
    n, h, w, _ = x.shape
    return ConvDesc(n, h, w, cin, cout, k, k, stride, pad)


def lenet_iteration(x, labels, weights, velocities, lr):
    """x [N][28][28][1] fp64, labels [N]; weights / velocities: name -> [K][R*S*C] arrays
    (real filters and momenta).  Returns (loss, new weights, new velocities, filter
    gradients), all fp64."""
    codes = {name: quantize(np.asarray(weights[name], np.float32)) for name, *_ in LENET}
    acts = []  # per layer: (input, pre-activation, post-ReLU, pool argmax)
    h = x
    for name, cin, cout, k, st, pd, relu, pool in LENET:
        q = codes[name]
        z = conv_fwd(_desc(h, cin, cout, k, st, pd), h, q.codes, q.alpha.astype(np.float64))
        a = np.maximum(z, 0.0) if relu else z
        arg = None
        out = a
        if pool:
            out, arg = maxpool_fwd(a, 2, 2, 0)
        acts.append((h, z, a, arg))
        h = out
    n = x.shape[0]
    loss, dz = softmax_xent(h.reshape(n, -1), labels)
    dh = dz.reshape(h.shape)
    grads = {}
    for (name, cin, cout, k, st, pd, relu, pool), (hin, z, a, arg) in zip(reversed(LENET), reversed(acts)):
        da = maxpool_bwd(dh, arg, a.shape, 2, 2, 0) if pool else dh
        dzl = np.where(z > 0, da, 0.0) if relu else da
        d = _desc(hin, cin, cout, k, st, pd)
        q = codes[name]
        grads[name] = conv_bwd_weight(d, hin, dzl).reshape(cout, -1)
        if name != LENET[0][0]:
            dh = conv_bwd_data(d, dzl, q.codes, q.alpha.astype(np.float64))
    new_w, new_v = {}, {}
    for name, *_ in LENET:
        w2, v2 = sgd(weights[name], velocities[name], grads[name], lr, MOMENTUM, WEIGHT_DECAY)
        new_w[name] = w2.reshape(np.shape(weights[name]))
        new_v[name] = v2.reshape(np.shape(weights[name]))
    return loss, new_w, new_v, grads


def vgg_iteration(x, labels, weights, velocities, bn, bn_vel, lr):
    """x [N][32][32][3] fp64, labels [N]; weights / velocities: name -> [K][R*S*C] (conv1
    full precision, the rest two-bit, and "fc"); bn / bn_vel: name -> (gamma, beta).
    Returns (loss, new weights, new velocities, new bn, new bn velocities, gradients)."""
    codes = {name: quantize(np.asarray(weights[name], np.float32)) for name, *_ in VGG[1:]}
    codes["fc"] = quantize(np.asarray(weights["fc"], np.float32))
    saved = []
    h = x
    for i, (name, cin, cout, pool) in enumerate(VGG):
        d = _desc(h, cin, cout, 3, 1, 1)
        if i == 0:
            w_bf = round_bf16(np.asarray(weights[name], np.float32)).reshape(cout, 3, 3, cin)
            z = conv_fwd_dense(d, h, w_bf)
        else:
            q = codes[name]
            z = conv_fwd(d, h, q.codes, q.alpha.astype(np.float64))
        gamma, beta = bn[name]
        y, _, _ = bn_train_fwd(z, gamma, beta)
        a = np.maximum(y, 0.0)
        arg = None
        out = a
        if pool:
            out, arg = maxpool_fwd(a, 2, 2, 0)
        saved.append((h, z, y, a, arg))
        h = out
    n = x.shape[0]
    dfc = ConvDesc(n, 4, 4, 512, 10, 4, 4, 1, 0)
    qf = codes["fc"]
    logits = conv_fwd(dfc, h, qf.codes, qf.alpha.astype(np.float64)).reshape(n, 10)
    loss, dz = softmax_xent(logits, labels)
    dz = dz.reshape(n, 1, 1, 10)
    grads = {"fc": conv_bwd_weight(dfc, h, dz).reshape(10, -1)}
    dh = conv_bwd_data(dfc, dz, qf.codes, qf.alpha.astype(np.float64))
    bn_grads = {}
    for i in reversed(range(len(VGG))):
        name, cin, cout, pool = VGG[i]
        hin, z, y, a, arg = saved[i]
        da = maxpool_bwd(dh, arg, a.shape, 2, 2, 0) if pool else dh
        dy = np.where(y > 0, da, 0.0)
        dzl, dg, db = bn_train_bwd(z, dy, bn[name][0])
        bn_grads[name] = (dg, db)
        d = _desc(hin, cin, cout, 3, 1, 1)
        grads[name] = conv_bwd_weight(d, hin, dzl).reshape(cout, -1)
        if i > 0:
            q = codes[name]
            dh = conv_bwd_data(d, dzl, q.codes, q.alpha.astype(np.float64))
    new_w, new_v = {}, {}
    for name in [v[0] for v in VGG] + ["fc"]:
        w2, v2 = sgd(weights[name], velocities[name], grads[name], lr, MOMENTUM, WEIGHT_DECAY)
        new_w[name] = w2.reshape(np.shape(weights[name]))
        new_v[name] = v2.reshape(np.shape(weights[name]))
    new_bn, new_bv = {}, {}
    for name, *_ in VGG:
        g2, vg2 = sgd(bn[name][0], bn_vel[name][0], bn_grads[name][0], lr, MOMENTUM, 0.0)
        b2, vb2 = sgd(bn[name][1], bn_vel[name][1], bn_grads[name][1], lr, MOMENTUM, 0.0)
        new_bn[name], new_bv[name] = (g2, b2), (vg2, vb2)
    return loss, new_w, new_v, new_bn, new_bv, grads
