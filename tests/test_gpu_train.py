"""Training iterations of the MNIST-shaped LeNet and the CIFAR-shaped VGG (Algorithm 1 with
the Sec. 4 optimiser) on the C ABI, checked operation by operation against the oracle.

Every recorded operation is recomputed by the oracle from the GPU's own inputs to it
(teacher forcing), so each check is the per-operation bar of the parity suite: codes
bit-exact and alpha within 1 ulp; convolutions, gradients and batch normalisation within a
normalised max error of 1e-2; pooling, its argmax and the ReLU gradient exact; SGD to fp32
rounding.  Operations that are independent per image are checked on sampled images, filter
gradients on sampled elements (each an exact reduction over the whole batch), so the full
workload batches stay within seconds of oracle time.  The loss after the step is reported.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from test_gpu_parity import log, nerr, ulp_diff

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def _f64(t):
    if t.dtype == torch.bfloat16:
        return oracle.bf16_bits_to_f64(_bits(t))
    return t.detach().cpu().numpy().astype(np.float64)


def _odesc(layer, x, n=None):
    N, H, W, _ = x.shape
    return oracle.ConvDesc(N if n is None else n, H, W, layer.cin, layer.cout, layer.k, layer.k, layer.stride,
                           layer.pad)


class Checker:
    def __init__(self, imgs, dw_samples):
        self.imgs = imgs
        self.dw_samples = dw_samples
        self.q = {}       # layer name -> oracle quantisation used by this step
        self.worst = {}

    def note(self, kind, e):
        self.worst[kind] = max(self.worst.get(kind, 0.0), e)

    def run(self, trace):
        for kind, info, t in trace:
            getattr(self, kind)(info, t)

    def quantize(self, layer, t):
        q = oracle.quantize(t["w"].cpu().numpy())
        assert np.array_equal(t["codes"].cpu().numpy().view(np.uint32), oracle.pack(q.codes)), layer.name
        assert ulp_diff(t["alpha"].cpu().numpy(), q.alpha).max() <= 1, layer.name
        self.q[layer.name] = q

    def conv_fwd(self, info, t):
        layer, relu = info
        x, y = t["x"], t["y"]
        im = self.imgs
        xs = _f64(x)[im]
        d = _odesc(layer, x, len(im))
        if layer.name in self.q:
            q = self.q[layer.name]
            ref = oracle.conv_fwd(d, xs, q.codes, q.alpha.astype(np.float64))
        else:  # the full-precision layer: filters rounded to bf16
            ref = oracle.conv_fwd_dense(d, xs, oracle.round_bf16(t["w"].cpu().numpy()))
        if relu:
            ref = np.maximum(ref, 0.0)
        e = nerr(_f64(y)[im].reshape(ref.shape), ref)
        self.note("conv_fwd", e)
        assert e <= 1e-2, "fwd %s: %.3e" % (layer.name, e)

    def maxpool(self, info, t):
        k, s, p = info
        im = self.imgs
        x = _f64(t["x"])[im]
        ref, arg = oracle.maxpool_fwd(x, k, s, p)
        assert np.array_equal(_f64(t["y"])[im], ref)
        N, H, W, C = x.shape
        assert np.array_equal(t["arg"].cpu().numpy()[im], arg // C % (H * W))

    def maxpool_bwd(self, info, t):
        k, s, p = info
        im = self.imgs
        dy = _f64(t["dy"])[im]
        dx_shape = (len(im),) + tuple(t["dx"].shape[1:])
        C, H, W = dx_shape[3], dx_shape[1], dx_shape[2]
        pos = t["arg"].cpu().numpy()[im].astype(np.int64)
        # GPU argmax (h*W + w per channel) -> the oracle's flat NHWC index
        n_idx = np.arange(len(im))[:, None, None, None]
        c_idx = np.arange(C)[None, None, None, :]
        flat = (n_idx * H * W + pos) * C + c_idx
        ref = oracle.maxpool_bwd(dy, flat, dx_shape, k, s, p)
        e = nerr(_f64(t["dx"])[im], ref)
        self.note("maxpool_bwd", e)
        assert e <= 1e-2

    def relu_bwd(self, info, t):
        want = np.where(_f64(t["y"]) > 0, _f64(t["dy"]), 0.0)
        assert np.array_equal(_f64(t["dx"]), want)

    def xent(self, info, t):
        loss, dz = oracle.softmax_xent(_f64(t["z"]), t["labels"].cpu().numpy())
        assert float(t["loss"].item()) == pytest.approx(loss, rel=1e-5)
        e = nerr(_f64(t["dz"]), dz)
        self.note("xent", e)
        assert e <= 1e-2

    def conv_bwd(self, layer, t):
        x, dy = t["x"], t["dy"]
        im = self.imgs
        if t["dx"] is not None:
            q = self.q[layer.name]
            ref = oracle.conv_bwd_data(_odesc(layer, x, len(im)), _f64(dy)[im], q.codes, q.alpha.astype(np.float64))
            e = nerr(_f64(t["dx"])[im], ref)
            self.note("conv_bwd_data", e)
            assert e <= 1e-2, "bwd_data %s: %.3e" % (layer.name, e)
        d = _odesc(layer, x)
        dw = t["dw"].cpu().numpy().ravel()
        idx = synth.sample_indices(20, "dw" + layer.name, dw.size, self.dw_samples)
        ref = oracle.conv_bwd_weight_sampled(d, _bits(x), _bits(dy), idx)
        e = nerr(dw[idx], ref)
        self.note("conv_bwd_weight", e)
        assert e <= 1e-2, "bwd_weight %s: %.3e" % (layer.name, e)

    def bn_fwd(self, bn, t):
        x = _f64(t["x"])
        y, mean, var = oracle.bn_train_fwd(x, t["gamma"].cpu().numpy(), t["beta"].cpu().numpy())
        # fp32 sums over up to 2^17 rows per channel
        assert nerr(t["mean"].cpu().numpy(), mean) <= 1e-4
        assert nerr(t["inv_std"].cpu().numpy(), 1 / np.sqrt(var + 1e-5)) <= 1e-4
        e = nerr(_f64(t["y"]), np.maximum(y, 0.0))
        self.note("bn_fwd", e)
        assert e <= 1e-2, "bn %s: %.3e" % (bn.name, e)

    def bn_bwd(self, bn, t):
        dy = _f64(t["dy"]) * (_f64(t["y"]) > 0)  # ReLU mask from the GPU's own output
        dx, dg, db = oracle.bn_train_bwd(_f64(t["x"]), dy, t["gamma"].cpu().numpy())
        e = max(nerr(_f64(t["dx"]), dx), nerr(t["dgamma"].cpu().numpy(), dg), nerr(t["dbeta"].cpu().numpy(), db))
        self.note("bn_bwd", e)
        assert e <= 1e-2, "bn bwd %s: %.3e" % (bn.name, e)

    def sgd(self, info, t):
        name, wd = info
        import paper_1701_00485_amd.networks as nets
        w = t["w"].cpu().numpy().astype(np.float64)
        v = t["v"].cpu().numpy().astype(np.float64)
        g = t["g"].cpu().numpy().astype(np.float64)
        w_ref, v_ref = oracle.sgd(w, v, g, nets.LR, nets.MOMENTUM, wd)
        assert nerr(t["w_new"].cpu().numpy().ravel(), np.ravel(w_ref)) <= 1e-6, name
        assert nerr(t["v_new"].cpu().numpy().ravel(), np.ravel(v_ref)) <= 1e-6, name


def _run(net, x, labels, imgs, dw_samples):
    trace = []
    loss = net.step(x, labels, trace)
    torch.cuda.synchronize()
    chk = Checker(imgs, dw_samples)
    chk.run(trace)
    return float(loss.item()), chk.worst, len(trace)


def _lenet_batch(n, name):
    x = synth.bf16_bits(synth.uniform(2, "x" + name, (n, 28, 28, 1)))
    lab = synth.labels(2, "lab" + name, n, 10).astype(np.int32)
    return (torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16), torch.from_numpy(lab).cuda())


def _vgg_batch(n, name):
    x = synth.normal_bf16(3, "x" + name, (n, 32, 32, 3))
    lab = synth.labels(3, "lab" + name, n, 10).astype(np.int32)
    return (torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16), torch.from_numpy(lab).cuda())


def test_lenet_step_batch256(tbn):
    from paper_1701_00485_amd.networks import LeNet
    net = LeNet()
    x, lab = _lenet_batch(256, "256")
    imgs = [int(i) for i in synth.sample_indices(2, "imgs", 256, 4)[:4]]
    loss, worst, n = _run(net, x, lab, imgs, 2048)
    log("lenet batch 256: %d ops checked, loss %.4f, worst %s" % (n, loss, worst))
    # a second step runs on the updated weights and is checked the same way
    loss2, worst2, _ = _run(net, x, lab, imgs, 2048)
    log("lenet batch 256 second step: loss %.4f, worst %s" % (loss2, worst2))


def test_vgg_small_step_batch4_full(tbn):
    from paper_1701_00485_amd.networks import VGGSmall
    net = VGGSmall()
    x, lab = _vgg_batch(4, "4")
    loss, worst, n = _run(net, x, lab, list(range(4)), 4096)
    log("vgg-small batch 4: %d ops checked, loss %.4f, worst %s" % (n, loss, worst))


def test_vgg_small_step_batch128_sampled(tbn):
    from paper_1701_00485_amd.networks import VGGSmall
    net = VGGSmall()
    x, lab = _vgg_batch(128, "128")
    imgs = [int(i) for i in synth.sample_indices(3, "imgs", 128, 2)[:2]]
    loss, worst, n = _run(net, x, lab, imgs, 1024)
    log("vgg-small batch 128 images %s: %d ops checked, loss %.4f, worst %s" % (imgs, n, loss, worst))
