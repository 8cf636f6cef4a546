"""Model-size accounting of Two-Bit Networks against double-precision networks (the
comparison of Sec. 4, Fig. 2, for AlexNet, ResNet-18 and VGG-19; the figure's values are
not in the text, so they are recomputed here from the architectures).

Every convolution and fully-connected filter is stored as two-bit codes plus one fp32
scale per filter (Sec. 2: W ~ alpha W~, one alpha per filter); biases and batch-norm
parameters are not filters and stay fp32.  Three sizes are reported per architecture:
  * fp64: every parameter in double precision (the paper's baseline);
  * tbn: 2 bits per filter weight + 4 bytes per filter + fp32 for the other parameters;
  * tbn_packed: the same with the codes in this library's packed layout (rows padded to
    64 codes, 64-filter blocks), the bytes the GPU actually holds.
Shapes are (kind, cin, cout, kernel, groups, bias); grouped convolutions have filters of
cin/groups x k x k elements.
"""
from __future__ import annotations


def _conv(cin, cout, k, groups=1, bias=True):
    return ("conv", cin, cout, k, groups, bias)


def _fc(cin, cout, bias=True):
    return ("fc", cin, cout, 1, 1, bias)


def alexnet():
    """The two-tower network of Krizhevsky et al. 2012 (227 x 227 input), grouped layers
    as on its two GPUs."""
    return [_conv(3, 96, 11), _conv(96, 256, 5, 2), _conv(256, 384, 3), _conv(384, 384, 3, 2),
            _conv(384, 256, 3, 2), _fc(256 * 6 * 6, 4096), _fc(4096, 4096), _fc(4096, 1000)]


def vgg19():
    """VGG-19 (configuration E of Simonyan & Zisserman), 224 x 224 input."""
    chans = [64, 64, 128, 128, 256, 256, 256, 256, 512, 512, 512, 512, 512, 512, 512, 512]
    layers, cin = [], 3
    for c in chans:
        layers.append(_conv(cin, c, 3))
        cin = c
    return layers + [_fc(512 * 7 * 7, 4096), _fc(4096, 4096), _fc(4096, 1000)]


def resnet18():
    """ResNet-18 with batch normalisation after every convolution (convolutions without
    bias), 1x1 projections where the shape changes, 1000-way classifier."""
    layers = [_conv(3, 64, 7, bias=False), ("bn", 64)]
    cin = 64
    for cout, stride in ((64, 1), (128, 2), (256, 2), (512, 2)):
        for b in range(2):
            s = stride if b == 0 else 1
            layers += [_conv(cin, cout, 3, bias=False), ("bn", cout), _conv(cout, cout, 3, bias=False), ("bn", cout)]
            if s != 1 or cin != cout:
                layers += [_conv(cin, cout, 1, bias=False), ("bn", cout)]
            cin = cout
    return layers + [_fc(512, 1000)]


ARCHS = {"AlexNet": alexnet, "ResNet-18": resnet18, "VGG-19": vgg19}


def _packed_words(k, n):
    # rows of n codes padded to 64, blocks of 64 filters, 16 codes per 32-bit word
    return ((k + 63) // 64) * ((n + 63) // 64) * 256


def count(layers):
    """(filter weights, filters, other fp32 parameters, packed code words)."""
    weights = filters = other = words = 0
    for l in layers:
        if l[0] == "bn":
            other += 2 * l[1]  # gamma and beta
            continue
        _, cin, cout, k, groups, bias = l
        n = cin // groups * k * k
        weights += cout * n
        filters += cout
        words += _packed_words(cout, n)
        other += cout if bias else 0
    return weights, filters, other, words


def memory_table():
    """Per architecture: parameter counts and the three sizes in bytes."""
    out = {}
    for name, fn in ARCHS.items():
        w, f, o, words = count(fn())
        fp64 = 8 * (w + o)
        tbn = (2 * w + 7) // 8 + 4 * f + 4 * o
        packed = 4 * words + 4 * f + 4 * o
        out[name] = {"filter_weights": w, "filters": f, "other_params": o, "params": w + o,
                     "fp64_bytes": fp64, "tbn_bytes": tbn, "tbn_packed_bytes": packed,
                     "fp64_over_tbn": round(fp64 / tbn, 2), "fp64_over_tbn_packed": round(fp64 / packed, 2)}
    return out
