"""The C ABI on the CPU: the library loads, exports every function include/tbn.h declares,
and its host-side shape arithmetic and argument checks behave as documented.  No call
here reaches a kernel (every checked call fails validation before any launch)."""
import ctypes
import os
import re

import pytest

import oracle
import paper_1701_00485_amd as tbn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    inc = os.path.join(ROOT, "include")
    for f in sorted(os.listdir(inc)):
        if f.endswith(".h"):
            text = open(os.path.join(inc, f)).read()
            names |= set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\*?\s+\*?(tbn_[a-z_0-9]+)\(", text, re.M))
    return sorted(names)


def test_library_exports_every_declared_function():
    lib = tbn.load()
    names = _declared()
    assert "tbn_quantize" in names and "tbn_conv2d_bwd_weight" in names
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(tbn.exported_symbols()) == names


def test_tuning_knobs_default_unset_and_round_trip():
    # every knob starts unset (kernel choice from the geometry alone); the context manager
    # restores the previous value; an unknown knob is rejected
    lib = tbn.load()
    for name in tbn.KNOBS:
        assert tbn.tuning_get(name) == -1
    with tbn.tuning(conv_tile=18, conv_splits=3):
        assert tbn.tuning_get("conv_tile") == 18 and tbn.tuning_get("conv_splits") == 3
        with tbn.tuning(conv_tile=12):
            assert tbn.tuning_get("conv_tile") == 12
        assert tbn.tuning_get("conv_tile") == 18
    assert tbn.tuning_get("conv_tile") == -1 and tbn.tuning_get("conv_splits") == -1
    assert lib.tbn_tuning_set(99, 1) == 2 and lib.tbn_tuning_get(99) == -1
    # no environment variable reaches the kernel choice
    src = os.path.join(ROOT, "paper_1701_00485_amd", "csrc")
    for f in os.listdir(src):
        assert "getenv" not in open(os.path.join(src, f)).read(), f


def test_status_strings():
    lib = tbn.load()
    for s, name in enumerate(["TBN_OK", "TBN_ERR_NULL", "TBN_ERR_SHAPE", "TBN_ERR_UNSUPPORTED",
                              "TBN_ERR_ALIGN", "TBN_ERR_WORKSPACE", "TBN_ERR_HIP"]):
        assert lib.tbn_status_str(s).decode() == name
    assert lib.tbn_status_str(99).decode() == "TBN_ERR_UNKNOWN"


@pytest.mark.parametrize("g", [
    (2, 7, 6, 1, 3, 5, 5, 1, 2), (1, 9, 9, 3, 5, 3, 3, 2, 1), (1, 224, 224, 3, 64, 7, 7, 2, 3),
    (64, 56, 56, 64, 128, 1, 1, 2, 0), (128, 56, 56, 256, 256, 3, 3, 1, 1), (1, 4, 4, 6, 2, 4, 4, 1, 0)])
def test_out_dims_match_oracle(g):
    assert tbn.ConvDesc(*g).out_dims() == oracle.ConvDesc(*g).out_dims()


@pytest.mark.parametrize("g", [(0, 4, 4, 1, 1, 1, 1, 1, 0), (1, 2, 2, 1, 1, 5, 5, 1, 0),
                               (1, 4, 4, 1, 1, 1, 1, 0, 0), (1, 4, 4, 1, 1, 1, 1, 1, -1)])
def test_bad_geometry(g):
    with pytest.raises(tbn.TbnError) as e:
        tbn.ConvDesc(*g).out_dims()
    assert e.value.status == 2


@pytest.mark.parametrize("K,n", [(1, 1), (32, 25), (64, 64), (65, 129), (512, 3136), (1000, 512)])
def test_packed_words_match_oracle(K, n):
    assert tbn.packed_words(K, n) == oracle.packed_words(K, n)
    assert tbn.packed_words(0, n) == -1
    # one filter row: whole 64-code groups of 4 words; K filters: 1 KiB per 64 x 64 block
    assert tbn.packed_row_words(n) == 4 * -(-n // 64)
    assert tbn.packed_bytes(K, n) == 4 * oracle.packed_words(K, n) == 1024 * -(-K // 64) * -(-n // 64)
    assert tbn.packed_row_words(0) == -1 and tbn.packed_bytes(K, 0) == -1


def test_argument_errors_before_launch():
    lib = tbn.load()
    vp = ctypes.c_void_p
    # NULL pointers
    assert lib.tbn_quantize(None, 4, 4, None, None, None, None) == 1
    d = tbn.ConvDesc(1, 8, 8, 8, 8, 3, 3, 1, 1)
    assert lib.tbn_conv2d_fwd(ctypes.byref(d), None, 0, None, None, None, None, 0, None, 0, None) == 1
    # misaligned pointers (never dereferenced: validation fails first)
    bad = vp(0x1002)
    good = vp(0x100000)
    assert lib.tbn_quantize(good, 4, 4, bad, good, None, None) == 4
    assert lib.tbn_conv2d_fwd(ctypes.byref(d), bad, 0, good, good, None, good, 0, None, 0, None) == 4
    # shape errors
    assert lib.tbn_quantize(good, 0, 4, good, good, None, None) == 2
    assert lib.tbn_sgd_step(good, good, good, 0, 0.1, 0.9, 0.0, None) == 2
    assert lib.tbn_sgd_step_quantize(good, good, good, 0, 4, 0.1, 0.9, 0.0, good, good, None, None) == 2
    assert lib.tbn_quantize_variant(good, 4, 4, 0.0, None, good, good, None, None) == 2
    assert lib.tbn_quantize_variant(good, 4, 4, float("inf"), None, good, good, None, None) == 2
    assert lib.tbn_quantize_variant(good, 4, 4, 0.5, good, good, good, None, None) == 3
    assert lib.tbn_quantize_variant(good, 4, 4, 1.0, vp(0x1001), good, good, None, None) == 4
    assert lib.tbn_sgd_step_quantize(good, good, good, 4, 4, 0.1, 0.9, 0.0, bad, good, None, None) == 4
    assert lib.tbn_sgd_step_quantize(good, None, good, 4, 4, 0.1, 0.9, 0.0, good, good, None, None) == 1
    # integer-activation variant
    assert lib.tbn_quantize_act_i8(None, 0, 16, 1.0, good, None) == 1
    assert lib.tbn_quantize_act_i8(good, 0, 0, 1.0, good, None) == 2
    assert lib.tbn_quantize_act_i8(good, 0, 16, 0.0, good, None) == 2
    assert lib.tbn_quantize_act_i8(good, 0, 16, float("nan"), good, None) == 2
    assert lib.tbn_quantize_act_i8(good, 0, 16, float("inf"), good, None) == 2
    assert lib.tbn_quantize_act_i8(good, 2, 16, 1.0, good, None) == 3
    assert lib.tbn_quantize_act_i8(good, 0, 16, 1.0, bad, None) == 4
    d16 = tbn.ConvDesc(1, 8, 8, 16, 8, 3, 3, 1, 1)
    assert lib.tbn_conv2d_fwd_i8(ctypes.byref(d16), None, good, good, 1.0, 0, good, 0, None) == 1
    assert lib.tbn_conv2d_fwd_i8(ctypes.byref(d16), good, good, good, float("nan"), 0, good, 0, None) == 2
    assert lib.tbn_conv2d_fwd_i8(ctypes.byref(d16), bad, good, good, 1.0, 0, good, 0, None) == 4
    assert lib.tbn_conv2d_fwd_i8(ctypes.byref(d16), good, good, good, 1.0, 0, good, 5, None) == 3
    assert lib.tbn_conv2d_fwd_i8(ctypes.byref(d), good, good, good, 1.0, 0, good, 0, None) == 3  # C = 8
    d_big = tbn.ConvDesc(1, 8, 8, 16, 8, 8, 8, 1, 1)  # R*S = 64 taps
    assert lib.tbn_conv2d_fwd_i8(ctypes.byref(d_big), good, good, good, 1.0, 0, good, 0, None) == 3
    # fp8-activation variant
    assert lib.tbn_quantize_act_fp8(None, 0, 16, 1.0, good, None) == 1
    assert lib.tbn_quantize_act_fp8(good, 0, 0, 1.0, good, None) == 2
    assert lib.tbn_quantize_act_fp8(good, 0, 16, -1.0, good, None) == 2
    assert lib.tbn_quantize_act_fp8(good, 0, 16, float("nan"), good, None) == 2
    assert lib.tbn_quantize_act_fp8(good, 2, 16, 1.0, good, None) == 3
    assert lib.tbn_quantize_act_fp8(good, 0, 16, 1.0, bad, None) == 4
    assert lib.tbn_repack_codes_fp4(None, 16, good, None) == 1
    assert lib.tbn_repack_codes_fp4(good, 0, vp(0x200000), None) == 2
    assert lib.tbn_repack_codes_fp4(good, 16, vp(0x100002), None) == 4
    assert lib.tbn_repack_codes_fp4(good, 16, vp(0x100020), None) == 2  # overlapping
    assert lib.tbn_conv2d_fwd_fp8(ctypes.byref(d16), None, good, good, 1.0, 0, good, 0, None) == 1
    assert lib.tbn_conv2d_fwd_fp8(ctypes.byref(d16), good, good, good, float("inf"), 0, good, 0, None) == 2
    assert lib.tbn_conv2d_fwd_fp8(ctypes.byref(d16), bad, good, good, 1.0, 0, good, 0, None) == 4
    assert lib.tbn_conv2d_fwd_fp8(ctypes.byref(d16), good, good, good, 1.0, 0, good, 5, None) == 3
    assert lib.tbn_conv2d_fwd_fp8(ctypes.byref(d), good, good, good, 1.0, 0, good, 0, None) == 3  # C = 8
    assert lib.tbn_conv2d_fwd_fp8(ctypes.byref(d_big), good, good, good, 1.0, 0, good, 0, None) == 3
    # stride-2 backward-data is not implemented
    d2 = tbn.ConvDesc(1, 8, 8, 8, 8, 3, 3, 2, 1)
    assert lib.tbn_conv2d_bwd_data(ctypes.byref(d2), good, good, good, good, 0, good, 1 << 20, None) == 3
    # workspace too small
    ws = ctypes.c_size_t()
    assert lib.tbn_workspace_size(tbn.OP_BWD_DATA, ctypes.byref(d), ctypes.byref(ws)) == 0
    assert ws.value > 0
    assert lib.tbn_conv2d_bwd_data(ctypes.byref(d), good, good, good, good, 0, good, ws.value - 1, None) == 5
    assert lib.tbn_last_error().decode() == "workspace too small"


def test_workspace_sizes():
    d = tbn.ConvDesc(128, 56, 56, 256, 256, 3, 3, 1, 1)
    assert tbn.workspace_size(tbn.OP_FWD, d) == 0
    # transposed codes (4 column blocks x 36 element blocks x 1 KiB) + bf16 scale pairs
    assert tbn.workspace_size(tbn.OP_BWD_DATA, d) == 4 * 36 * 1024 + 36 * 32 * 4
    wb = tbn.workspace_size(tbn.OP_BWD_WEIGHT, d)
    assert wb % (256 * 2304 * 4) == 0 and wb >= 256 * 2304 * 4
    # a layer with few output tiles splits its reduction: fp32 partials [splits][M][K]
    d = tbn.ConvDesc(16, 7, 7, 512, 512, 3, 3, 1, 1)
    wf = tbn.workspace_size(tbn.OP_FWD, d)
    assert wf > 0 and wf % (16 * 7 * 7 * 512 * 4) == 0
    codes_pairs = 8 * 72 * 1024 + 72 * 32 * 4
    assert tbn.workspace_size(tbn.OP_BWD_DATA, d) == codes_pairs + wf
    # 196 tiles of 64 x 128 (the 7 x 7 x 512 layers at batch 64): groups of waves inside
    # each block reduce the stage ranges, no partial sums in memory
    d = tbn.ConvDesc(64, 7, 7, 512, 512, 3, 3, 1, 1)
    assert tbn.workspace_size(tbn.OP_FWD, d) == 0
    assert tbn.workspace_size(tbn.OP_BWD_DATA, d) == codes_pairs


def test_stem_workspace_is_the_bordered_copy():
    # 7x7/2 stem over 64 x 224 x 224 x 3: 14 x 4 tiles of 8 x 32 outputs; the bordered copy
    # spans (14-1)*8*2 + 21 = 229 rows and (4-1)*32*2 + 70 = 262 columns of 4 channels
    d = tbn.ConvDesc(64, 224, 224, 3, 64, 7, 7, 2, 3)
    assert tbn.workspace_size(tbn.OP_FWD, d) == (64 * 229 * 262 * 4 * 2 + 255) // 256 * 256
    # small inputs load their patches directly: no workspace
    assert tbn.workspace_size(tbn.OP_FWD, tbn.ConvDesc(16, 28, 28, 1, 32, 5, 5, 1, 2)) == 0


def test_forward_workspace_checked():
    lib = tbn.load()
    good = ctypes.c_void_p(0x100000)
    d = tbn.ConvDesc(16, 7, 7, 512, 512, 3, 3, 1, 1)
    need = tbn.workspace_size(tbn.OP_FWD, d)
    assert need > 0
    args = (ctypes.byref(d), good, 0, good, good, None, good, 0)
    assert lib.tbn_conv2d_fwd(*args, None, 0, None) == 5
    assert lib.tbn_conv2d_fwd(*args, good, need - 1, None) == 5
    assert lib.tbn_last_error().decode() == "workspace too small"
    assert lib.tbn_conv2d_fwd(*args, ctypes.c_void_p(0x100004), need, None) == 4


def test_batchnorm_workspace_checked():
    lib = tbn.load()
    good = ctypes.c_void_p(0x100000)
    need = tbn.batchnorm_workspace_size(131072, 128)
    assert need > 0 and need % (128 * 4) == 0
    args = (good, 131072, 128, good, good, ctypes.c_float(1e-5), 1, good, good, good)
    assert lib.tbn_batchnorm_train_fwd(*args, None, 0, None) == 5
    assert lib.tbn_batchnorm_train_fwd(*args, good, need - 4, None) == 5
    assert lib.tbn_last_error().decode() == "workspace too small"


@pytest.mark.parametrize("g,why", [
    ((1 << 16, 200, 200, 8, 8, 1, 1, 1, 0), "more than 2^31 - 1 pixels"),
    ((1, 8, 8, 1 << 26, 8, 5, 5, 1, 2), "filter has more than 2^30 elements"),
    # N * P * Q = 2^22 * 2^21 * 2^21 = 2^64: wraps to 0 in 64-bit arithmetic
    ((1 << 22, 2, 2, 8, 8, 1, 1, 1, (1 << 20) - 1), "more than 2^31 - 1 pixels"),
])
def test_index_range_limits(g, why):
    # sizes whose pixel or filter indices would overflow the kernels' 32-bit arithmetic are
    # rejected before any launch (pointers are never dereferenced)
    lib = tbn.load()
    good = ctypes.c_void_p(0x100000)
    d = tbn.ConvDesc(*g)
    assert lib.tbn_conv2d_fwd(ctypes.byref(d), good, 0, good, good, None, good, 0, good, 1 << 40, None) == 2
    assert lib.tbn_last_error().decode() == why
    assert lib.tbn_conv2d_bwd_weight(ctypes.byref(d), good, good, good, 0, good, 1 << 40, None) == 2


@pytest.mark.parametrize("pd,why", [
    ((1, 1 << 16, 1 << 16, 8, 2, 2, 0), "more than 2^31 - 1 positions per image"),
    ((1, 8, 8, 8, 2, 1, (1 << 30)), "more than 2^31 - 1 positions per image"),
    ((1 << 30, 1 << 10, 1 << 10, 1 << 30, 2, 2, 0), "tensor too large"),  # 2^80 elements
])
def test_pool_index_range_limits(pd, why):
    # pooling sizes beyond the kernels' 32-bit positions, or whose element count overflows
    # 64-bit arithmetic, are rejected before any launch
    lib = tbn.load()
    good = ctypes.c_void_p(0x100000)
    d = tbn.PoolDesc(*pd)
    assert lib.tbn_maxpool2d_fwd(ctypes.byref(d), good, good, None, None) == 2
    assert lib.tbn_last_error().decode() == why
    assert lib.tbn_avgpool_global(1, 1 << 16, 1 << 16, 8, good, good, 0, None) == 2
    assert lib.tbn_last_error().decode() == "more than 2^31 - 1 positions per image"


def test_unknown_dtype_and_pool_geometry():
    lib = tbn.load()
    good = ctypes.c_void_p(0x100000)
    d = tbn.ConvDesc(1, 8, 8, 8, 8, 3, 3, 1, 1)
    assert lib.tbn_conv2d_fwd(ctypes.byref(d), good, 7, good, good, None, good, 0, None, 0, None) == 3
    pd = tbn.PoolDesc(1, 2, 2, 8, 3, 1, 0)  # window larger than the input
    p, q = ctypes.c_int32(), ctypes.c_int32()
    assert lib.tbn_pool_out_dims(ctypes.byref(pd), ctypes.byref(p), ctypes.byref(q)) == 2
