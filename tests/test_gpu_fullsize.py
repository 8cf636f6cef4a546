"""The training-layer workload at its full size, in the launch configuration the benchmark
times (conv 3x3, 256 -> 256 channels, 56 x 56, pad 1, batch 128): one step of Algorithm 1
(quantise -> forward -> backward-data -> backward-weight -> SGD) with the benchmark's
buffers, workspaces and inputs, checked against the oracle:
  * codes bit-exact and alpha within 1 ulp over all 256 filters;
  * 4096 sampled outputs of each contraction, each recomputed exactly by the oracle
    (a filter-gradient sample is a full reduction over the 401,408 output pixels);
  * the SGD update over every weight.
The benchmark draws the real weights from N(0, 0.05^2), where Eq. 3 gives only the codes +-1;
a second run with N(0, 1) weights (about a third of the codes +-2) covers the magnitude-2
decode in the same launch configuration.
"""
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import synth
from test_gpu_parity import log, nerr, ulp_diff

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("w_std", [0.05, 1.0])
def test_training_layer_full_size(tbn, w_std):
    sys.path.insert(0, ROOT)
    import bench

    L = bench.LAYER
    g = (L["n"], L["h"], L["w"], L["c"], L["k"], L["r"], L["s"], L["stride"], L["pad"])
    d = oracle.ConvDesc(*g)
    P, Q = d.out_dims()
    n = L["r"] * L["s"] * L["c"]
    xb = synth.normal_bf16(5, "x", (L["n"], L["h"], L["w"], L["c"]))
    dyb = synth.normal_bf16(5, "dy", (L["n"], P, Q, L["k"]))
    w0 = synth.normal(5, "w" if w_std == 0.05 else "w_std1", (L["k"], n), w_std)

    dev = torch.device("cuda")
    desc = tbn.ConvDesc(*g)
    x = torch.from_numpy(xb.view(np.int16)).to(dev).view(torch.bfloat16)
    dy = torch.from_numpy(dyb.view(np.int16)).to(dev).view(torch.bfloat16)
    w = torch.from_numpy(w0).to(dev)
    v = torch.zeros_like(w)
    codes = torch.empty(tbn.packed_words(L["k"], n), dtype=torch.int32, device=dev)
    alpha = torch.empty(L["k"], dtype=torch.float32, device=dev)
    y = torch.empty((L["n"], P, Q, L["k"]), dtype=torch.bfloat16, device=dev)
    dx = torch.empty_like(x)
    dw = torch.empty((L["k"], L["r"], L["s"], L["c"]), dtype=torch.float32, device=dev)
    ws_bd = tbn.workspace(tbn.OP_BWD_DATA, desc, dev)
    ws_bw = tbn.workspace(tbn.OP_BWD_WEIGHT, desc, dev)

    # the benchmark's step, call for call
    tbn.quantize(w, codes, alpha, want_counts=False)
    tbn.conv2d_fwd(desc, x, codes, alpha, y=y)
    tbn.conv2d_bwd_data(desc, dy, codes, alpha, dx=dx, ws=ws_bd)
    tbn.conv2d_bwd_weight(desc, x, dy, dw=dw, ws=ws_bw)
    w_before = w.clone()
    tbn.sgd_step(w, v, dw, bench.LR, bench.MOMENTUM, bench.WD)
    torch.cuda.synchronize()

    q = oracle.quantize(w0)
    assert np.array_equal(codes.cpu().numpy().view(np.uint32), oracle.pack(q.codes))
    frac2 = float(np.mean(np.abs(q.codes) == 2))
    log("full-size layer, real weights N(0, %g^2): %.1f%% of the codes are +-2" % (w_std, 100 * frac2))
    if w_std >= 1.0:
        assert frac2 > 0.25
    assert ulp_diff(alpha.cpu().numpy(), q.alpha).max() <= 1
    a64 = q.alpha.astype(np.float64)

    def bits(t):
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1)

    idx = synth.sample_indices(5, "fwd_idx", y.numel(), 4096)
    ref = oracle.conv_fwd_sampled(d, xb.reshape(-1), q.codes, a64, idx)
    e = nerr(oracle.bf16_bits_to_f64(bits(y)[idx]), ref)
    log("full-size fwd (w std %g), 4096 samples: %.3e" % (w_std, e))
    assert e <= 1e-2

    idx = synth.sample_indices(5, "bd_idx", dx.numel(), 4096)
    ref = oracle.conv_bwd_data_sampled(d, dyb.reshape(-1), q.codes, a64, idx)
    e = nerr(oracle.bf16_bits_to_f64(bits(dx)[idx]), ref)
    log("full-size bwd_data (w std %g), 4096 samples: %.3e" % (w_std, e))
    assert e <= 1e-2

    idx = synth.sample_indices(5, "bw_idx", dw.numel(), 4096)
    ref = oracle.conv_bwd_weight_sampled(d, xb.reshape(-1), dyb.reshape(-1), idx)
    e = nerr(dw.cpu().numpy().reshape(-1)[idx], ref)
    log("full-size bwd_weight (w std %g), 4096 samples over 401408-term reductions: %.3e" % (w_std, e))
    assert e <= 1e-4

    w_ref, _ = oracle.sgd(w_before.cpu().numpy().astype(np.float64), np.zeros(w0.shape),
                          dw.cpu().numpy().reshape(w0.shape).astype(np.float64), bench.LR, bench.MOMENTUM, bench.WD)
    assert nerr(w.cpu().numpy().ravel(), np.ravel(w_ref)) <= 1e-6
