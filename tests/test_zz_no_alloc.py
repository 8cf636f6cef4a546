"""The forward pass without caller workspace (tbn_conv2d_fwd_noalloc, the entry point for
callers that cannot allocate): on the same inputs it gives exactly what tbn_conv2d_fwd gives
with a caller workspace (the same kernels run), on two calls in a row whose second has a
smaller input, for layers whose plan needs workspace (split reductions of batch-1 layers,
the bordered copy of a thin input); each result is also within the oracle's bar.  A layer
needing more workspace than the static scratch is refused before anything is queued."""
import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


CASES = [
    # (geometry, epilogue) -- each needs workspace under the default plan (batch-1 layers
    # whose reduction is too long for the in-block wave groups split it over the grid)
    ((1, 7, 7, 512, 512, 3, 3, 1, 1), True),      # ResNet-18 layer-4 shape at batch 1
    ((1, 5, 5, 384, 512, 3, 3, 1, 1), True),      # a smaller input, 54 stages
    ((8, 224, 224, 3, 64, 7, 7, 2, 3), False),    # the stem at batch 8 (bordered input copy)
    ((1, 7, 7, 512, 256, 3, 3, 1, 1), False),     # layer-4 input, 256 filters: smaller than the stem
]


def _run(tbn, g, ep, seed):
    n, h, w, c, k, r, s, st, pd = g
    d = oracle.ConvDesc(*g)
    P, Q = d.out_dims()
    xb = synth.normal_bf16(13, "x%d" % seed, (n, h, w, c))
    wr = synth.normal(13, "w%d" % seed, (k, r * s * c), 1.0)
    scale = synth.uniform(13, "sc%d" % seed, (k,), 0.5, 1.5)
    bias = synth.normal(13, "bi%d" % seed, (k,), 0.1)
    resb = synth.normal_bf16(13, "res%d" % seed, (n, P, Q, k))
    dev = torch.device("cuda")
    x = torch.from_numpy(xb.view(np.int16)).to(dev).view(torch.bfloat16)
    codes, alpha, _ = tbn.quantize(torch.from_numpy(wr).to(dev))
    desc = tbn.ConvDesc(*g)
    kw = {}
    if ep:
        kw = dict(scale=torch.from_numpy(scale).to(dev), bias=torch.from_numpy(bias).to(dev),
                  residual=torch.from_numpy(resb.view(np.int16)).to(dev).view(torch.bfloat16), relu=True)
    assert tbn.workspace_size(tbn.OP_FWD, desc) > 0, "case must exercise the workspace"
    y_na = torch.full((n, P, Q, k), 7.0, dtype=torch.bfloat16, device=dev)
    tbn.conv2d_fwd_noalloc(desc, x, codes, alpha, y_na, **kw)
    y_ws = tbn.conv2d_fwd(desc, x, codes, alpha, out_dtype=torch.bfloat16, **kw)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(y_na), _bits(y_ws)), "no-allocation result differs from the workspace call"
    q = oracle.quantize(wr)
    ref = oracle.conv_fwd(d, oracle.bf16_bits_to_f64(xb), q.codes, q.alpha.astype(np.float64))
    if ep:
        ref = np.maximum(ref * scale.astype(np.float64) + bias + oracle.bf16_bits_to_f64(resb), 0.0)
    got = oracle.bf16_bits_to_f64(_bits(y_na)).reshape(ref.shape)
    e = float(np.max(np.abs(got - ref)) / np.max(np.abs(ref)))
    assert e <= 1e-2, "normalised error %.3e" % e


def test_noalloc_matches_workspace_call_twice_smaller_second(tbn):
    for i in range(0, len(CASES), 2):
        (g1, e1), (g2, e2) = CASES[i], CASES[i + 1]
        assert g2[0] * g2[1] * g2[2] * g2[3] < g1[0] * g1[1] * g1[2] * g1[3]
        _run(tbn, g1, e1, i)
        _run(tbn, g2, e2, i + 1)   # second call in a row, smaller input, same scratch


def test_noalloc_refuses_layers_beyond_the_scratch(tbn):
    g = (64, 224, 224, 3, 64, 7, 7, 2, 3)  # the stem at batch 64: its bordered copy exceeds the scratch
    desc = tbn.ConvDesc(*g)
    assert tbn.workspace_size(tbn.OP_FWD, desc) > tbn.NOALLOC_SCRATCH_BYTES
    dev = torch.device("cuda")
    x = torch.zeros((64, 224, 224, 3), dtype=torch.bfloat16, device=dev)
    codes, alpha, _ = tbn.quantize(torch.ones((64, 147), device=dev))
    y = torch.zeros((64, 112, 112, 64), dtype=torch.bfloat16, device=dev)
    with pytest.raises(tbn.TbnError) as e:
        tbn.conv2d_fwd_noalloc(desc, x, codes, alpha, y)
    assert e.value.status == 5  # TBN_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert int(torch.count_nonzero(y)) == 0  # nothing was queued
