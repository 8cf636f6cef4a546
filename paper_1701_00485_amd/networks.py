"""Workload networks built on the C ABI: ResNet-18 inference with every convolution and the
fully-connected layer two-bit (Sec. 4 trains ResNet-18 with batch normalisation; at inference
only the two-bit filters and their scales are used, Sec. 3).

Every operation runs in libtbn: two-bit convolutions with the batch normalisation folded
into the epilogue (inference form: scale = gamma / sqrt(var + eps), bias = beta - mean *
scale, computed once when the network is built, like the quantisation of its filters),
ReLU and the residual add fused into the same epilogue, max pooling, global average
pooling, and the classifier as a 1x1 two-bit convolution with an fp32 bias.  Weights and
batch-normalisation statistics are seeded synthetic values (no trained weights exist).
"""
from __future__ import annotations

import numpy as np
import torch

import paper_1701_00485_amd as tbn

# Workload seed stream of the ResNet-18 inference configuration
RESNET_STREAM = 4


class Conv:
    """One two-bit convolution with its folded batch normalisation."""

    def __init__(self, name, cin, cout, k, stride, pad, device, stream, bn=True, bias=False):
        import zlib
        self.name, self.cin, self.cout, self.k, self.stride, self.pad = name, cin, cout, k, stride, pad
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([1701_00485 + stream, zlib.crc32(name.encode())])))
        n = k * k * cin
        self.w = (g.standard_normal((cout, n), dtype=np.float32) * np.float32(np.sqrt(2.0 / n))).astype(np.float32)
        wt = torch.from_numpy(self.w).to(device)
        self.codes, self.alpha, _ = tbn.quantize(wt, want_counts=False)
        self.scale = self.bias = None
        self.scale_np = self.bias_np = None
        if bn:
            gamma = g.uniform(0.5, 1.5, cout)
            beta = g.normal(0.0, 0.1, cout)
            mean = g.normal(0.0, 0.1, cout)
            var = g.uniform(0.5, 1.5, cout)
            self.bn = (gamma, beta, mean, var)
            scale = gamma / np.sqrt(var + 1e-5)
            self.scale_np = scale.astype(np.float32)
            self.bias_np = (beta - mean * scale).astype(np.float32)
        elif bias:
            self.bias_np = g.normal(0.0, 0.01, cout).astype(np.float32)
        if self.scale_np is not None:
            self.scale = torch.from_numpy(self.scale_np).to(device)
        if self.bias_np is not None:
            self.bias = torch.from_numpy(self.bias_np).to(device)

    def desc(self, x):
        n, h, w, _ = x.shape
        return tbn.ConvDesc(n, h, w, self.cin, self.cout, self.k, self.k, self.stride, self.pad)

    def __call__(self, x, relu, residual=None, out_dtype=torch.bfloat16):
        return tbn.conv2d_fwd(self.desc(x), x, self.codes, self.alpha, out_dtype=out_dtype, scale=self.scale,
                              bias=self.bias, residual=residual, relu=relu)


class ResNet18:
    """ResNet-18 (standard basic-block layout: 7x7/2 stem, 3x3/2 max pool, four stages of
    two basic blocks with 64/128/256/512 channels, 1x1/2 projection where the shape changes,
    global average pool, 1000-way classifier), all convolutions two-bit."""

    STAGES = [(64, 1), (128, 2), (256, 2), (512, 2)]

    def __init__(self, device="cuda", classes=1000, stream=RESNET_STREAM):
        self.device = device
        self.stem = Conv("stem", 3, 64, 7, 2, 3, device, stream)
        self.blocks = []
        cin = 64
        for si, (cout, stride) in enumerate(self.STAGES):
            for bi in range(2):
                s = stride if bi == 0 else 1
                name = "layer%d.%d" % (si + 1, bi)
                c1 = Conv(name + ".conv1", cin, cout, 3, s, 1, device, stream)
                c2 = Conv(name + ".conv2", cout, cout, 3, 1, 1, device, stream)
                ds = Conv(name + ".downsample", cin, cout, 1, s, 0, device, stream) if (s != 1 or cin != cout) else None
                self.blocks.append((c1, c2, ds))
                cin = cout
        self.fc = Conv("fc", 512, classes, 1, 1, 0, device, stream, bn=False, bias=True)
        self.classes = classes

    def convs(self):
        out = [self.stem]
        for c1, c2, ds in self.blocks:
            out += [c1, c2] + ([ds] if ds is not None else [])
        return out + [self.fc]

    def forward(self, x, trace=None):
        """x: [N][224][224][3] bf16 NHWC -> logits fp32 [N][classes].  `trace` (a list)
        receives (kind, layer, input, output, residual) for every step."""
        def rec(kind, layer, inp, out, res=None):
            if trace is not None:
                trace.append((kind, layer, inp, out, res))
        y = self.stem(x, relu=True)
        rec("conv", self.stem, x, y)
        p, _ = tbn.maxpool2d_fwd(y, 3, 2, 1)
        rec("maxpool", (3, 2, 1), y, p)
        h = p
        for c1, c2, ds in self.blocks:
            a = c1(h, relu=True)
            rec("conv", c1, h, a)
            if ds is not None:
                sc = ds(h, relu=False)
                rec("conv", ds, h, sc)
            else:
                sc = h
            o = c2(a, relu=True, residual=sc)
            rec("conv", c2, a, o, sc)
            h = o
        f = tbn.avgpool_global(h)
        rec("avgpool", None, h, f)
        n = f.shape[0]
        logits = self.fc(f.view(n, 1, 1, 512), relu=False, out_dtype=torch.float32).view(n, self.classes)
        rec("conv", self.fc, f.view(n, 1, 1, 512), logits.view(n, 1, 1, self.classes))
        return logits

    @staticmethod
    def flops(batch):
        """Dense FLOP of one forward pass (2 per multiply-add of every convolution)."""
        total = 0
        h = 224
        def conv(hin, cin, cout, k, s, p):
            ho = (hin + 2 * p - k) // s + 1
            return 2 * batch * ho * ho * cout * k * k * cin, ho
        f, h = conv(h, 3, 64, 7, 2, 3)
        total += f
        h = (h + 2 - 3) // 2 + 1
        cin = 64
        for cout, stride in ResNet18.STAGES:
            for bi in range(2):
                s = stride if bi == 0 else 1
                f1, h2 = conv(h, cin, cout, 3, s, 1)
                f2, _ = conv(h2, cout, cout, 3, 1, 1)
                total += f1 + f2
                if s != 1 or cin != cout:
                    total += conv(h, cin, cout, 1, s, 0)[0]
                h, cin = h2, cout
        total += 2 * batch * 512 * 1000
        return total


# --------------------------------------------------------------------------------------
# Training (Algorithm 1): quantise every layer, forward, softmax cross-entropy, backward
# through the approximate filters, straight-through gradient to the real filters, SGD.
# --------------------------------------------------------------------------------------
LR, MOMENTUM, WEIGHT_DECAY = 0.1, 0.9, 1e-4
# Sec. 4 schedule: the learning rate starts at 0.1 and is divided by 10 at epochs 30, 40
# and 50 (Algorithm 1 ends each iteration with a learning-rate update).
LR_MILESTONES = (30, 40, 50)


def lr_at(epoch, base=LR, milestones=LR_MILESTONES, factor=0.1):
    """Learning rate of an epoch under the step schedule of Sec. 4."""
    return base * factor ** sum(1 for m in milestones if epoch >= m)


def _seeded(stream, name):
    import zlib
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([1701_00485 + stream, zlib.crc32(name.encode())])))


class TwoBitLayer:
    """A trainable two-bit convolution (or fully-connected layer as an R x S "valid"
    convolution over the whole map): fp32 real filters [K][R*S*C], momentum buffer, and the
    codes / scales of the current quantisation."""

    def __init__(self, name, cin, cout, k, stride, pad, device, stream, std=0.05):
        self.name, self.cin, self.cout, self.k, self.stride, self.pad = name, cin, cout, k, stride, pad
        g = _seeded(stream, name)
        n = k * k * cin
        self.w = torch.from_numpy((g.standard_normal((cout, n), dtype=np.float32) * np.float32(std))).to(device)
        self.v = torch.zeros_like(self.w)
        self.codes = self.alpha = None

    def desc(self, x):
        n, h, w, _ = x.shape
        return tbn.ConvDesc(n, h, w, self.cin, self.cout, self.k, self.k, self.stride, self.pad)

    def quantize(self):
        self.codes, self.alpha, _ = tbn.quantize(self.w, codes=self.codes, alpha=self.alpha, want_counts=False)

    def forward(self, x, relu=False, out_dtype=torch.bfloat16):
        return tbn.conv2d_fwd(self.desc(x), x, self.codes, self.alpha, out_dtype=out_dtype, relu=relu)

    def backward(self, x, dy, need_dx=True):
        d = self.desc(x)
        dx = tbn.conv2d_bwd_data(d, dy, self.codes, self.alpha) if need_dx else None
        dw = tbn.conv2d_bwd_weight(d, x, dy)
        return dx, dw


class DenseLayer:
    """A trainable full-precision convolution (filters rounded to bf16 at use)."""

    def __init__(self, name, cin, cout, k, stride, pad, device, stream, std=0.05):
        self.name, self.cin, self.cout, self.k, self.stride, self.pad = name, cin, cout, k, stride, pad
        g = _seeded(stream, name)
        self.w = torch.from_numpy((g.standard_normal((cout, k * k * cin), dtype=np.float32) * np.float32(std))).to(device)
        self.v = torch.zeros_like(self.w)

    def desc(self, x):
        n, h, w, _ = x.shape
        return tbn.ConvDesc(n, h, w, self.cin, self.cout, self.k, self.k, self.stride, self.pad)

    def forward(self, x, relu=False, out_dtype=torch.bfloat16):
        return tbn.conv2d_fwd_dense(self.desc(x), x, self.w, out_dtype=out_dtype, relu=relu)

    def backward(self, x, dy, need_dx=False):
        if need_dx:
            raise NotImplementedError("the full-precision layer is the first layer: no input gradient")
        return None, tbn.conv2d_bwd_weight(self.desc(x), x, dy)


class BatchNorm:
    """Batch normalisation in training form (batch statistics), gamma ~ U(0.5, 1.5),
    beta ~ N(0, 0.1); trained without weight decay."""

    def __init__(self, name, c, device, stream):
        g = _seeded(stream, name + ".bn")
        self.name = name + ".bn"
        self.gamma = torch.from_numpy(g.uniform(0.5, 1.5, c).astype(np.float32)).to(device)
        self.beta = torch.from_numpy(g.normal(0.0, 0.1, c).astype(np.float32)).to(device)
        self.vg = torch.zeros_like(self.gamma)
        self.vb = torch.zeros_like(self.beta)


class _Trainer:
    """Shared step logic: `rec` (when given a list) receives (kind, info, tensors) for every
    operation, with copies of whatever the step later overwrites."""

    def _rec(self, trace, kind, info, **t):
        if trace is not None:
            trace.append((kind, info, t))

    def named_state(self):
        """The training state by name: real weights and momenta of every layer, batch-norm
        parameters and their momenta.  The codes and scales are not part of it: they are a
        function of the real weights (Eq. 3-5) and are recomputed after a restore."""
        out, seen = {}, []
        for l in list(getattr(self, "convs", [])) + self.two_bit_layers():
            if any(l is o for o in seen):
                continue
            seen.append(l)
            out[l.name + ".w"], out[l.name + ".v"] = l.w, l.v
        for bn in getattr(self, "bns", []):
            for f in ("gamma", "beta", "vg", "vb"):
                out["%s.%s" % (bn.name, f)] = getattr(bn, f)
        return out

    def save(self, path):
        """Checkpoint the training state and the learning rate to an .npz file."""
        arrays = {k: t.detach().cpu().numpy() for k, t in self.named_state().items()}
        np.savez(path, lr=np.float64(self.lr), **arrays)

    def load(self, path):
        """Restore a checkpoint written by save(); the next step re-quantises the restored
        weights, so training continues bit-identically to an uninterrupted run."""
        with np.load(path) as data:  # plain arrays only (no pickled objects)
            for k, t in self.named_state().items():
                src = torch.from_numpy(data[k])
                if tuple(src.shape) != tuple(t.shape):
                    raise ValueError("checkpoint tensor %s has shape %s, expected %s" % (k, tuple(src.shape),
                                                                                       tuple(t.shape)))
                t.copy_(src.to(t.device))
            self.lr = float(data["lr"])
        self._codes_current = False

    def _sgd(self, trace, name, w, v, g, wd):
        if trace is not None:
            w0, v0 = w.clone(), v.clone()
        tbn.sgd_step(w, v, g, self.lr, MOMENTUM, wd)
        if trace is not None:
            self._rec(trace, "sgd", (name, wd), w=w0, v=v0, g=g, w_new=w, v_new=v)

    def _quantize(self, trace):
        if getattr(self, "_codes_current", False):
            return  # the previous step's fused update already quantised the new weights
        for l in self.two_bit_layers():
            l.quantize()
            if trace is not None:
                self._rec(trace, "quantize", l, w=l.w.clone(), codes=l.codes.clone(), alpha=l.alpha.clone())

    def _update_two_bit(self, trace, layer, g, fused):
        """SGD on a two-bit layer's real filters; with `fused`, the same pass also
        quantises the updated filters for the next iteration."""
        if not fused:
            self._sgd(trace, layer.name, layer.w, layer.v, g, WEIGHT_DECAY)
            return
        if trace is not None:
            w0, v0 = layer.w.clone(), layer.v.clone()
        layer.codes, layer.alpha, _ = tbn.sgd_step_quantize(layer.w, layer.v, g, self.lr, MOMENTUM, WEIGHT_DECAY,
                                                            codes=layer.codes, alpha=layer.alpha,
                                                            want_counts=False)
        if trace is not None:
            self._rec(trace, "sgd_quantize", (layer.name, WEIGHT_DECAY), w=w0, v=v0, g=g, w_new=layer.w,
                      v_new=layer.v, codes=layer.codes.clone(), alpha=layer.alpha.clone())

    def train(self, x, labels, iterations, iters_per_epoch=None, fused=True):
        """Algorithm 1 run for `iterations` iterations on one batch, the learning rate set
        by the Sec. 4 schedule (epochs of `iters_per_epoch` iterations, default: one
        epoch per iteration).  Returns the loss of every iteration (fp32 tensor)."""
        losses = []
        for it in range(iterations):
            self.lr = lr_at(it // (iters_per_epoch or 1))
            losses.append(self.step(x, labels, fused=fused))
        return torch.cat([l.view(1) for l in losses])


class LeNet(_Trainer):
    """MNIST-shaped LeNet, every layer two-bit: conv 5x5 1->32 pad 2, ReLU, max pool 2,
    conv 5x5 32->64 pad 2, ReLU, max pool 2, FC 3136->512 (7x7 "valid" convolution), ReLU,
    FC 512->10; softmax cross-entropy, mean over the batch."""

    def __init__(self, device="cuda", stream=2, lr=LR):
        self.lr = lr
        self.conv1 = TwoBitLayer("conv1", 1, 32, 5, 1, 2, device, stream)
        self.conv2 = TwoBitLayer("conv2", 32, 64, 5, 1, 2, device, stream)
        self.fc1 = TwoBitLayer("fc1", 64, 512, 7, 1, 0, device, stream)
        self.fc2 = TwoBitLayer("fc2", 512, 10, 1, 1, 0, device, stream)

    def two_bit_layers(self):
        return [self.conv1, self.conv2, self.fc1, self.fc2]

    @staticmethod
    def flops(batch):
        """Dense FLOP of one forward pass."""
        f = 0
        for (h, c, k, r, hout) in [(28, 1, 32, 5, 28), (14, 32, 64, 5, 14), (7, 64, 512, 7, 1), (1, 512, 10, 1, 1)]:
            f += 2 * batch * hout * hout * k * r * r * c
        return f

    @staticmethod
    def train_flops(batch):
        """Forward, backward-data (not for the first layer) and backward-weight."""
        return 3 * LeNet.flops(batch) - 2 * batch * 28 * 28 * 32 * 25

    def step(self, x, labels, trace=None, fused=False):
        """x [N][28][28][1] bf16, labels [N] int32 -> loss (fp32 [1]); updates the weights.
        `fused`: update and re-quantise each two-bit layer in one pass (the next step then
        skips its quantisation)."""
        rec = self._rec
        N = x.shape[0]
        self._quantize(trace)
        a1 = self.conv1.forward(x, relu=True)
        rec(trace, "conv_fwd", (self.conv1, True), x=x, y=a1)
        p1, arg1 = tbn.maxpool2d_fwd(a1, 2, 2, 0, want_argmax=True)
        rec(trace, "maxpool", (2, 2, 0), x=a1, y=p1, arg=arg1)
        a2 = self.conv2.forward(p1, relu=True)
        rec(trace, "conv_fwd", (self.conv2, True), x=p1, y=a2)
        p2, arg2 = tbn.maxpool2d_fwd(a2, 2, 2, 0, want_argmax=True)
        rec(trace, "maxpool", (2, 2, 0), x=a2, y=p2, arg=arg2)
        h3 = self.fc1.forward(p2, relu=True)
        rec(trace, "conv_fwd", (self.fc1, True), x=p2, y=h3)
        z = self.fc2.forward(h3, out_dtype=torch.float32)
        rec(trace, "conv_fwd", (self.fc2, False), x=h3, y=z)
        loss, dz = tbn.softmax_xent(z.view(N, 10), labels)
        rec(trace, "xent", None, z=z.view(N, 10), labels=labels, loss=loss, dz=dz)
        dz = dz.view(N, 1, 1, 10)
        dh3, dw4 = self.fc2.backward(h3, dz)
        rec(trace, "conv_bwd", self.fc2, x=h3, dy=dz, dx=dh3, dw=dw4)
        dz3 = tbn.relu_bwd(h3, dh3)
        rec(trace, "relu_bwd", None, y=h3, dy=dh3, dx=dz3)
        dp2, dw3 = self.fc1.backward(p2, dz3)
        rec(trace, "conv_bwd", self.fc1, x=p2, dy=dz3, dx=dp2, dw=dw3)
        da2 = tbn.maxpool2d_bwd(dp2, arg2, a2.shape, 2, 2, 0)
        rec(trace, "maxpool_bwd", (2, 2, 0), dy=dp2, arg=arg2, dx=da2)
        dz2 = tbn.relu_bwd(a2, da2)
        rec(trace, "relu_bwd", None, y=a2, dy=da2, dx=dz2)
        dp1, dw2 = self.conv2.backward(p1, dz2)
        rec(trace, "conv_bwd", self.conv2, x=p1, dy=dz2, dx=dp1, dw=dw2)
        da1 = tbn.maxpool2d_bwd(dp1, arg1, a1.shape, 2, 2, 0)
        rec(trace, "maxpool_bwd", (2, 2, 0), dy=dp1, arg=arg1, dx=da1)
        dz1 = tbn.relu_bwd(a1, da1)
        rec(trace, "relu_bwd", None, y=a1, dy=da1, dx=dz1)
        _, dw1 = self.conv1.backward(x, dz1, need_dx=False)
        rec(trace, "conv_bwd", self.conv1, x=x, dy=dz1, dx=None, dw=dw1)
        for l, g in zip(self.two_bit_layers(), (dw1, dw2, dw3, dw4)):
            self._update_two_bit(trace, l, g.view(l.w.shape), fused)
        self._codes_current = fused
        return loss


class VGGSmall(_Trainer):
    """CIFAR-shaped VGG: conv 3x3 3->128 in full precision (bf16 filters), then two-bit
    conv 3x3 128->128, pool, 128->256, 256->256, pool, 256->512, 512->512, pool, FC 8192->10
    (4x4 "valid" convolution); training-form batch normalisation and ReLU after every
    convolution; softmax cross-entropy, mean over the batch."""

    PLAN = [(3, 128, False), (128, 128, True), (128, 256, False), (256, 256, True), (256, 512, False),
            (512, 512, True)]  # (cin, cout, max pool after)

    def __init__(self, device="cuda", stream=3, lr=LR):
        self.lr = lr
        self.convs, self.bns = [], []
        for i, (cin, cout, _) in enumerate(self.PLAN):
            name = "conv%d" % (i + 1)
            layer = DenseLayer if i == 0 else TwoBitLayer
            self.convs.append(layer(name, cin, cout, 3, 1, 1, device, stream))
            self.bns.append(BatchNorm(name, cout, device, stream))
        self.fc = TwoBitLayer("fc", 512, 10, 4, 1, 0, device, stream)
        # every batch-norm parameter, its momentum and its gradient live in three flat
        # buffers (gamma then beta of each layer), so that one SGD call updates them all
        # (they share the hyperparameters: no weight decay); the layers hold views
        total = sum(2 * bn.gamma.numel() for bn in self.bns)
        self.bn_flat = torch.empty(total, dtype=torch.float32, device=device)
        self.bn_vflat = torch.zeros(total, dtype=torch.float32, device=device)
        self.bn_gflat = torch.zeros(total, dtype=torch.float32, device=device)
        self.bn_grad_views = []
        off = 0
        for bn in self.bns:
            c = bn.gamma.numel()
            views = []
            for f, vf in (("gamma", "vg"), ("beta", "vb")):
                self.bn_flat[off:off + c].copy_(getattr(bn, f))
                setattr(bn, f, self.bn_flat[off:off + c])
                setattr(bn, vf, self.bn_vflat[off:off + c])
                views.append(self.bn_gflat[off:off + c])
                off += c
            self.bn_grad_views.append(tuple(views))

    def two_bit_layers(self):
        return self.convs[1:] + [self.fc]

    @staticmethod
    def flops(batch):
        f, h = 0, 32
        for cin, cout, pool in VGGSmall.PLAN:
            f += 2 * batch * h * h * cout * 9 * cin
            if pool:
                h //= 2
        return f + 2 * batch * 10 * 8192

    @staticmethod
    def train_flops(batch):
        """Forward, backward-data (not for the first layer) and backward-weight."""
        return 3 * VGGSmall.flops(batch) - 2 * batch * 32 * 32 * 128 * 27

    def step(self, x, labels, trace=None, fused=False):
        """x [N][32][32][3] bf16, labels [N] int32 -> loss (fp32 [1]); updates the weights.
        `fused`: update and re-quantise each two-bit layer in one pass."""
        rec = self._rec
        N = x.shape[0]
        self._quantize(trace)
        saved = []  # per conv: (input, pre-BN output, post-BN-ReLU output, mean, inv_std, pool argmax)
        h = x
        for conv, bn, (_, _, pool) in zip(self.convs, self.bns, self.PLAN):
            z = conv.forward(h)
            extra = {"w": conv.w.clone()} if trace is not None and isinstance(conv, DenseLayer) else {}
            rec(trace, "conv_fwd", (conv, False), x=h, y=z, **extra)
            a, mean, inv_std = tbn.batchnorm_train_fwd(z, bn.gamma, bn.beta, relu=True)
            if trace is not None:  # gamma and beta are updated in place at the end of the step
                rec(trace, "bn_fwd", bn, x=z, y=a, mean=mean, inv_std=inv_std, gamma=bn.gamma.clone(),
                    beta=bn.beta.clone())
            arg = None
            out = a
            if pool:
                out, arg = tbn.maxpool2d_fwd(a, 2, 2, 0, want_argmax=True)
                rec(trace, "maxpool", (2, 2, 0), x=a, y=out, arg=arg)
            saved.append((h, z, a, mean, inv_std, arg))
            h = out
        logits = self.fc.forward(h, out_dtype=torch.float32)
        rec(trace, "conv_fwd", (self.fc, False), x=h, y=logits)
        loss, dz = tbn.softmax_xent(logits.view(N, 10), labels)
        rec(trace, "xent", None, z=logits.view(N, 10), labels=labels, loss=loss, dz=dz)
        dh, dwfc = self.fc.backward(h, dz.view(N, 1, 1, 10))
        rec(trace, "conv_bwd", self.fc, x=h, dy=dz.view(N, 1, 1, 10), dx=dh, dw=dwfc)
        grads = [None] * len(self.convs)
        bn_grads = [None] * len(self.convs)
        for i in reversed(range(len(self.convs))):
            conv, bn = self.convs[i], self.bns[i]
            hin, z, a, mean, inv_std, arg = saved[i]
            if arg is not None:
                da = tbn.maxpool2d_bwd(dh, arg, a.shape, 2, 2, 0)
                rec(trace, "maxpool_bwd", (2, 2, 0), dy=dh, arg=arg, dx=da)
            else:
                da = dh
            dzi, dg, db = tbn.batchnorm_train_bwd(z, a, da, mean, inv_std, bn.gamma, relu=True,
                                                  dgamma=self.bn_grad_views[i][0], dbeta=self.bn_grad_views[i][1])
            if trace is not None:
                rec(trace, "bn_bwd", bn, x=z, y=a, dy=da, gamma=bn.gamma.clone(), dx=dzi, dgamma=dg, dbeta=db)
            dh, dw = conv.backward(hin, dzi, need_dx=i > 0)
            rec(trace, "conv_bwd", conv, x=hin, dy=dzi, dx=dh, dw=dw)
            grads[i], bn_grads[i] = dw, (dg, db)
        for conv, g in zip(self.convs, grads):
            if isinstance(conv, TwoBitLayer):
                self._update_two_bit(trace, conv, g.view(conv.w.shape), fused)
            else:
                self._sgd(trace, conv.name, conv.w, conv.v, g.view(conv.w.shape), WEIGHT_DECAY)
        self._update_two_bit(trace, self.fc, dwfc.view(self.fc.w.shape), fused)
        self._codes_current = fused
        # every gamma and beta in one call over the flat buffers (the trace still gets one
        # record per parameter: the update is element-wise)
        if trace is not None:
            w0, v0 = self.bn_flat.clone(), self.bn_vflat.clone()
        tbn.sgd_step(self.bn_flat, self.bn_vflat, self.bn_gflat, self.lr, MOMENTUM, 0.0)
        if trace is not None:
            off = 0
            for bn, (dg, db) in zip(self.bns, bn_grads):
                for f, vf, g in (("gamma", "vg", dg), ("beta", "vb", db)):
                    c = g.numel()
                    self._rec(trace, "sgd", (bn.name + "." + f, 0.0), w=w0[off:off + c], v=v0[off:off + c], g=g,
                              w_new=getattr(bn, f), v_new=getattr(bn, vf))
                    off += c
        return loss
