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
