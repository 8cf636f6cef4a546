"""fp64 CPU oracle for the Two-Bit Networks hot path (arXiv 1701.00485).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the CPU-baseline leg of
the benchmark may import this package; the product library never does.  The oracle
shares no code with the GPU library.  The numerics live in ``tbn_oracle.c`` (plain fp64
loops, one function per step of the method, each citing the passage it follows); this
module only marshals numpy arrays through ctypes.

Sections cited: Sec. 2 Eq. (1) approximate convolution, Eq. (3) discretisation,
Eq. (4)-(5) optimal scale; Sec. 3 Algorithm 1 (quantise, forward, backward, update);
Sec. 4 optimiser settings.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tbn_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (fp64, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
             "-fno-fast-math", "-ffp-contract=off", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    p = ctypes.c_void_p
    i64 = ctypes.c_int64
    lib.orc_round_bf16.argtypes = [p, i64, p]
    lib.orc_round_bf16.restype = None
    lib.orc_codes_of_bits.argtypes = [ctypes.c_uint64, i64, p]
    lib.orc_codes_of_bits.restype = None
    lib.orc_quantize.argtypes = [p, i64, i64, p, p, p, p, p, p, p]
    lib.orc_quantize.restype = ctypes.c_int
    lib.orc_packed_words.argtypes = [i64, i64]
    lib.orc_packed_words.restype = i64
    lib.orc_pack.argtypes = [p, i64, i64, p]
    lib.orc_pack.restype = ctypes.c_int
    lib.orc_unpack.argtypes = [p, i64, i64, p]
    lib.orc_unpack.restype = ctypes.c_int
    lib.orc_out_dims.argtypes = [p, p, p]
    lib.orc_out_dims.restype = ctypes.c_int
    lib.orc_conv_fwd.argtypes = [p, p, p, p, ctypes.c_int, p]
    lib.orc_conv_fwd.restype = ctypes.c_int
    lib.orc_conv_fwd_dense.argtypes = [p, p, p, p]
    lib.orc_conv_fwd_dense.restype = ctypes.c_int
    lib.orc_quantize_act_i8.argtypes = [p, i64, ctypes.c_float, p]
    lib.orc_quantize_act_i8.restype = None
    lib.orc_conv_fwd_i8.argtypes = [p, p, p, p, ctypes.c_float, ctypes.c_int, p, p]
    lib.orc_conv_fwd_i8.restype = ctypes.c_int
    lib.orc_conv_fwd_i8_sampled.argtypes = [p, p, p, p, ctypes.c_float, ctypes.c_int, p, i64, p]
    lib.orc_conv_fwd_i8_sampled.restype = ctypes.c_int
    lib.orc_fp8_value.argtypes = [ctypes.c_uint8]
    lib.orc_fp8_value.restype = ctypes.c_double
    lib.orc_fp8_encode.argtypes = [ctypes.c_float]
    lib.orc_fp8_encode.restype = ctypes.c_uint8
    lib.orc_quantize_act_fp8.argtypes = [p, i64, ctypes.c_float, p]
    lib.orc_quantize_act_fp8.restype = None
    lib.orc_conv_fwd_fp8.argtypes = [p, p, p, p, ctypes.c_float, ctypes.c_int, p]
    lib.orc_conv_fwd_fp8.restype = ctypes.c_int
    lib.orc_conv_fwd_fp8_sampled.argtypes = [p, p, p, p, ctypes.c_float, ctypes.c_int, p, i64, p]
    lib.orc_conv_fwd_fp8_sampled.restype = ctypes.c_int
    lib.orc_conv_bwd_data.argtypes = [p, p, p, p, p]
    lib.orc_conv_bwd_data.restype = ctypes.c_int
    lib.orc_conv_bwd_weight.argtypes = [p, p, p, p]
    lib.orc_conv_bwd_weight.restype = ctypes.c_int
    for name in ("orc_conv_fwd_sampled_bf16", "orc_conv_bwd_data_sampled_bf16"):
        getattr(lib, name).argtypes = [p, p, p, p, p, i64, p]
        getattr(lib, name).restype = ctypes.c_int
    lib.orc_conv_bwd_weight_sampled_bf16.argtypes = [p, p, p, p, i64, p]
    lib.orc_conv_bwd_weight_sampled_bf16.restype = ctypes.c_int
    lib.orc_sgd.argtypes = [p, p, p, i64, ctypes.c_double, ctypes.c_double, ctypes.c_double]
    lib.orc_sgd.restype = None
    lib.orc_quantize_variant.argtypes = [p, i64, i64, ctypes.c_float, p, p, p, p, p, p]
    lib.orc_quantize_variant.restype = ctypes.c_int
    lib.orc_sgd_f32.argtypes = [p, p, p, i64, ctypes.c_float, ctypes.c_float, ctypes.c_float]
    lib.orc_sgd_f32.restype = None
    lib.orc_set_threads.argtypes = [ctypes.c_int]
    lib.orc_set_threads.restype = None
    lib.orc_max_threads.argtypes = []
    lib.orc_max_threads.restype = ctypes.c_int
    lib.orc_maxpool_fwd.argtypes = [p, p, p, p]
    lib.orc_maxpool_fwd.restype = ctypes.c_int
    lib.orc_maxpool_bwd.argtypes = [p, p, p, p]
    lib.orc_maxpool_bwd.restype = ctypes.c_int
    lib.orc_avgpool_global.argtypes = [p, p, p]
    lib.orc_avgpool_global.restype = None
    d = ctypes.c_double
    lib.orc_bn_infer.argtypes = [p, i64, i64, p, p, p, p, d, p]
    lib.orc_bn_infer.restype = None
    lib.orc_bn_train_fwd.argtypes = [p, i64, i64, p, p, d, p, p, p]
    lib.orc_bn_train_fwd.restype = None
    lib.orc_bn_train_bwd.argtypes = [p, p, i64, i64, p, d, p, p, p]
    lib.orc_bn_train_bwd.restype = None
    lib.orc_softmax_xent.argtypes = [p, p, i64, i64, p]
    lib.orc_softmax_xent.restype = ctypes.c_double
    _lib = lib
    return lib


class OracleError(RuntimeError):
    pass


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


class ConvDesc:
    """Geometry of one convolution (NHWC activations, [K][R][S][C] filters)."""

    __slots__ = ("n", "h", "w", "c", "k", "r", "s", "stride_h", "stride_w", "pad_h", "pad_w")

    def __init__(self, n, h, w, c, k, r, s, stride=1, pad=0, stride_w=None, pad_w=None):
        self.n, self.h, self.w, self.c, self.k, self.r, self.s = n, h, w, c, k, r, s
        self.stride_h = stride
        self.stride_w = stride if stride_w is None else stride_w
        self.pad_h = pad
        self.pad_w = pad if pad_w is None else pad_w

    def as_array(self) -> np.ndarray:
        return np.array([self.n, self.h, self.w, self.c, self.k, self.r, self.s,
                         self.stride_h, self.stride_w, self.pad_h, self.pad_w], dtype=np.int32)

    def out_dims(self):
        d = self.as_array()
        p = np.zeros(1, np.int32)
        q = np.zeros(1, np.int32)
        if _load().orc_out_dims(_ptr(d), _ptr(p), _ptr(q)) != 0:
            raise OracleError("invalid convolution geometry")
        return int(p[0]), int(q[0])


# --------------------------------------------------------------------------------------
# bf16 rounding of fp32 inputs (IEEE round-to-nearest-even on the dropped 16 bits)
# --------------------------------------------------------------------------------------
def set_threads(n: int) -> None:
    """Threads of the oracle's parallel loops (timing only; results do not depend on it)."""
    _load().orc_set_threads(int(n))


def max_threads() -> int:
    return int(_load().orc_max_threads())


def round_bf16(x: np.ndarray) -> np.ndarray:
    x = _c(x, np.float32)
    out = np.empty(x.shape, np.float64)
    _load().orc_round_bf16(_ptr(x), x.size, _ptr(out))
    return out


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of raw bf16 bit patterns (uint16) to float64."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------------------
# Sec. 2, Eq. (3)-(5): quantisation
# --------------------------------------------------------------------------------------
class Quantized:
    __slots__ = ("codes", "alpha64", "alpha", "b1_size", "b2_size", "b1_sum", "b2_sum")


def quantize(w: np.ndarray) -> Quantized:
    """w: [K][n] fp32 real weights (one filter per row)."""
    w = _c(w, np.float32)
    if w.ndim != 2:
        raise OracleError("quantize expects [K][n]")
    K, n = w.shape
    out = Quantized()
    out.codes = np.zeros((K, n), np.int8)
    out.alpha64 = np.zeros(K, np.float64)
    out.alpha = np.zeros(K, np.float32)
    out.b1_size = np.zeros(K, np.int64)
    out.b2_size = np.zeros(K, np.int64)
    out.b1_sum = np.zeros(K, np.float64)
    out.b2_sum = np.zeros(K, np.float64)
    st = _load().orc_quantize(_ptr(w), K, n, _ptr(out.codes), _ptr(out.alpha64),
                              _ptr(out.alpha), _ptr(out.b1_size), _ptr(out.b2_size),
                              _ptr(out.b1_sum), _ptr(out.b2_sum))
    if st == 1:
        raise OracleError("non-finite weight: outside the method's domain")
    if st != 0:
        raise OracleError("quantize: bad shape")
    return out


def codes_of_bits(start: int, count: int) -> np.ndarray:
    """Eq. (3) codes of the fp32 values with bit patterns start .. start + count - 1
    (int8; NaN patterns, outside the method, get 0)."""
    out = np.empty(count, np.int8)
    _load().orc_codes_of_bits(int(start), int(count), _ptr(out))
    return out


def quantize_variant(w: np.ndarray, threshold: float = 1.0, uniform=None) -> Quantized:
    """Discretisation variants: magnitude threshold `threshold`, or stochastic rounding
    driven by `uniform` ([K][n] fp32 in [0, 1)); alpha = sum W c / sum c^2."""
    w = _c(w, np.float32)
    if w.ndim != 2:
        raise OracleError("quantize_variant expects [K][n]")
    K, n = w.shape
    u = None if uniform is None else _c(uniform, np.float32).reshape(K, n)
    out = Quantized()
    out.codes = np.zeros((K, n), np.int8)
    out.alpha64 = np.zeros(K, np.float64)
    out.alpha = np.zeros(K, np.float32)
    out.b1_size = np.zeros(K, np.int64)
    out.b2_size = np.zeros(K, np.int64)
    st = _load().orc_quantize_variant(_ptr(w), K, n, float(threshold), None if u is None else _ptr(u),
                                      _ptr(out.codes), _ptr(out.alpha64), _ptr(out.alpha), _ptr(out.b1_size),
                                      _ptr(out.b2_size))
    if st == 1:
        raise OracleError("non-finite weight: outside the method's domain")
    if st != 0:
        raise OracleError("quantize_variant: bad shape or threshold")
    return out


def packed_words(K: int, n: int) -> int:
    return int(_load().orc_packed_words(K, n))


def pack(codes: np.ndarray) -> np.ndarray:
    codes = _c(codes, np.int8)
    K, n = codes.shape
    words = np.zeros(packed_words(K, n), np.uint32)
    if _load().orc_pack(_ptr(codes), K, n, _ptr(words)) != 0:
        raise OracleError("pack: codes outside {-2,-1,1,2} or bad shape")
    return words


def unpack(words: np.ndarray, K: int, n: int) -> np.ndarray:
    words = _c(words, np.uint32)
    if words.size != packed_words(K, n):
        raise OracleError("unpack: wrong word count")
    codes = np.zeros((K, n), np.int8)
    if _load().orc_unpack(_ptr(words), K, n, _ptr(codes)) != 0:
        raise OracleError("unpack: bad shape")
    return codes


# --------------------------------------------------------------------------------------
# Sec. 2 Eq. (1) and Sec. 3 Algorithm 1: convolutions with the two-bit filters
# --------------------------------------------------------------------------------------
def conv_fwd(desc: ConvDesc, x: np.ndarray, codes: np.ndarray, alpha: np.ndarray,
             form: int = 0) -> np.ndarray:
    """x NHWC fp64 (exact values the GPU consumed); codes [K][R][S][C] (or [K][n])."""
    P, Q = desc.out_dims()
    x = _c(x, np.float64)
    codes = _c(codes, np.int8)
    alpha = _c(alpha, np.float64)
    if x.size != desc.n * desc.h * desc.w * desc.c or codes.size != desc.k * desc.r * desc.s * desc.c:
        raise OracleError("conv_fwd: operand sizes do not match the geometry")
    y = np.zeros((desc.n, P, Q, desc.k), np.float64)
    d = desc.as_array()
    if _load().orc_conv_fwd(_ptr(d), _ptr(x), _ptr(codes), _ptr(alpha), form, _ptr(y)) != 0:
        raise OracleError("conv_fwd failed")
    return y


def conv_fwd_dense(desc: ConvDesc, x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """Eq. (1) with real-valued filters w [K][R][S][C] (a full-precision layer)."""
    P, Q = desc.out_dims()
    x = _c(x, np.float64)
    w = _c(w, np.float64)
    if x.size != desc.n * desc.h * desc.w * desc.c or w.size != desc.k * desc.r * desc.s * desc.c:
        raise OracleError("conv_fwd_dense: operand sizes do not match the geometry")
    y = np.zeros((desc.n, P, Q, desc.k), np.float64)
    if _load().orc_conv_fwd_dense(_ptr(desc.as_array()), _ptr(x), _ptr(w), _ptr(y)) != 0:
        raise OracleError("conv_fwd_dense failed")
    return y


# --------------------------------------------------------------------------------------
# Integer-activation variant of Eq. (1): the input replaced by s * q, q int8 (an extension)
# --------------------------------------------------------------------------------------
def quantize_act_i8(x: np.ndarray, inv_scale) -> np.ndarray:
    """q = clamp(round-half-even(fp32(x * inv_scale)), -127, 127), NaN -> 0; x fp32 values."""
    x = _c(x, np.float32)
    q = np.zeros(x.shape, np.int8)
    _load().orc_quantize_act_i8(_ptr(x), x.size, float(np.float32(inv_scale)), _ptr(q))
    return q


def conv_fwd_i8(desc: ConvDesc, xq: np.ndarray, codes: np.ndarray, alpha: np.ndarray, x_scale,
                relu: bool = False):
    """Forward pass on int8 activation codes: returns (y fp32 NHWC, exact int64 sums).
    y = fp32(acc) * fp32(alpha_k * x_scale), then max(., 0) when relu."""
    P, Q = desc.out_dims()
    xq = _c(xq, np.int8)
    codes = _c(codes, np.int8)
    alpha = _c(alpha, np.float32)
    if xq.size != desc.n * desc.h * desc.w * desc.c or codes.size != desc.k * desc.r * desc.s * desc.c:
        raise OracleError("conv_fwd_i8: operand sizes do not match the geometry")
    y = np.zeros((desc.n, P, Q, desc.k), np.float32)
    acc = np.zeros((desc.n, P, Q, desc.k), np.int64)
    if _load().orc_conv_fwd_i8(_ptr(desc.as_array()), _ptr(xq), _ptr(codes), _ptr(alpha),
                               float(np.float32(x_scale)), 1 if relu else 0, _ptr(acc), _ptr(y)) != 0:
        raise OracleError("conv_fwd_i8 failed")
    return y, acc


def conv_fwd_i8_sampled(desc: ConvDesc, xq: np.ndarray, codes: np.ndarray, alpha: np.ndarray, x_scale,
                        idx: np.ndarray, relu: bool = False) -> np.ndarray:
    """conv_fwd_i8's y at flat output indices idx (into [N][P][Q][K]), fp32."""
    xq = _c(xq, np.int8)
    codes = _c(codes, np.int8)
    alpha = _c(alpha, np.float32)
    idx = _c(idx, np.int64)
    if xq.size != desc.n * desc.h * desc.w * desc.c or codes.size != desc.k * desc.r * desc.s * desc.c:
        raise OracleError("conv_fwd_i8_sampled: operand sizes do not match the geometry")
    y = np.zeros(idx.size, np.float32)
    if _load().orc_conv_fwd_i8_sampled(_ptr(desc.as_array()), _ptr(xq), _ptr(codes), _ptr(alpha),
                                       float(np.float32(x_scale)), 1 if relu else 0, _ptr(idx), idx.size,
                                       _ptr(y)) != 0:
        raise OracleError("conv_fwd_i8_sampled: index out of range")
    return y


# --------------------------------------------------------------------------------------
# fp8-activation variant of Eq. (1): the input replaced by s * f, f an E4M3 value (an
# extension)
# --------------------------------------------------------------------------------------
def fp8_value(codes: np.ndarray) -> np.ndarray:
    """float64 value of every E4M3 code (uint8 array); NaN for 0x7F and 0xFF."""
    codes = np.asarray(codes, np.uint8)
    lib = _load()
    table = np.array([lib.orc_fp8_value(c) for c in range(256)], np.float64)
    return table[codes]


def fp8_encode_one(v) -> int:
    """The E4M3 code of one fp32 value (nearest, ties to the even code, saturating at 448)."""
    return int(_load().orc_fp8_encode(float(np.float32(v))))


def quantize_act_fp8(x: np.ndarray, inv_scale) -> np.ndarray:
    """codes = E4M3(fp32(x * inv_scale)), nearest with ties to even, saturating, NaN -> 0."""
    x = _c(x, np.float32)
    q = np.zeros(x.shape, np.uint8)
    _load().orc_quantize_act_fp8(_ptr(x), x.size, float(np.float32(inv_scale)), _ptr(q))
    return q


def conv_fwd_fp8(desc: ConvDesc, xq: np.ndarray, codes: np.ndarray, alpha: np.ndarray, x_scale,
                 relu: bool = False) -> np.ndarray:
    """Forward pass on E4M3 activation codes: y = alpha_k * x_scale * sum f * W~ in fp64
    (NHWC), then max(., 0) when relu."""
    P, Q = desc.out_dims()
    xq = _c(xq, np.uint8)
    codes = _c(codes, np.int8)
    alpha = _c(alpha, np.float32)
    if xq.size != desc.n * desc.h * desc.w * desc.c or codes.size != desc.k * desc.r * desc.s * desc.c:
        raise OracleError("conv_fwd_fp8: operand sizes do not match the geometry")
    y = np.zeros((desc.n, P, Q, desc.k), np.float64)
    if _load().orc_conv_fwd_fp8(_ptr(desc.as_array()), _ptr(xq), _ptr(codes), _ptr(alpha),
                                float(np.float32(x_scale)), 1 if relu else 0, _ptr(y)) != 0:
        raise OracleError("conv_fwd_fp8 failed")
    return y


def conv_fwd_fp8_sampled(desc: ConvDesc, xq: np.ndarray, codes: np.ndarray, alpha: np.ndarray, x_scale,
                         idx: np.ndarray, relu: bool = False) -> np.ndarray:
    """conv_fwd_fp8's y at flat output indices idx (into [N][P][Q][K]), fp64."""
    xq = _c(xq, np.uint8)
    codes = _c(codes, np.int8)
    alpha = _c(alpha, np.float32)
    idx = _c(idx, np.int64)
    if xq.size != desc.n * desc.h * desc.w * desc.c or codes.size != desc.k * desc.r * desc.s * desc.c:
        raise OracleError("conv_fwd_fp8_sampled: operand sizes do not match the geometry")
    y = np.zeros(idx.size, np.float64)
    if _load().orc_conv_fwd_fp8_sampled(_ptr(desc.as_array()), _ptr(xq), _ptr(codes), _ptr(alpha),
                                        float(np.float32(x_scale)), 1 if relu else 0, _ptr(idx), idx.size,
                                        _ptr(y)) != 0:
        raise OracleError("conv_fwd_fp8_sampled failed")
    return y


def conv_bwd_data(desc: ConvDesc, dy: np.ndarray, codes: np.ndarray, alpha: np.ndarray) -> np.ndarray:
    P, Q = desc.out_dims()
    dy = _c(dy, np.float64)
    codes = _c(codes, np.int8)
    alpha = _c(alpha, np.float64)
    if dy.size != desc.n * P * Q * desc.k:
        raise OracleError("conv_bwd_data: dy size does not match the geometry")
    dx = np.zeros((desc.n, desc.h, desc.w, desc.c), np.float64)
    d = desc.as_array()
    if _load().orc_conv_bwd_data(_ptr(d), _ptr(dy), _ptr(codes), _ptr(alpha), _ptr(dx)) != 0:
        raise OracleError("conv_bwd_data failed")
    return dx


def conv_bwd_weight(desc: ConvDesc, x: np.ndarray, dy: np.ndarray) -> np.ndarray:
    P, Q = desc.out_dims()
    x = _c(x, np.float64)
    dy = _c(dy, np.float64)
    if dy.size != desc.n * P * Q * desc.k or x.size != desc.n * desc.h * desc.w * desc.c:
        raise OracleError("conv_bwd_weight: operand sizes do not match the geometry")
    dw = np.zeros((desc.k, desc.r, desc.s, desc.c), np.float64)
    d = desc.as_array()
    if _load().orc_conv_bwd_weight(_ptr(d), _ptr(x), _ptr(dy), _ptr(dw)) != 0:
        raise OracleError("conv_bwd_weight failed")
    return dw


def conv_fwd_sampled(desc, x_bits, codes, alpha, idx):
    x_bits = _c(x_bits, np.uint16)
    codes = _c(codes, np.int8)
    alpha = _c(alpha, np.float64)
    idx = _c(idx, np.int64)
    out = np.zeros(idx.size, np.float64)
    d = desc.as_array()
    if _load().orc_conv_fwd_sampled_bf16(_ptr(d), _ptr(x_bits), _ptr(codes), _ptr(alpha),
                                         _ptr(idx), idx.size, _ptr(out)) != 0:
        raise OracleError("conv_fwd_sampled failed")
    return out


def conv_bwd_data_sampled(desc, dy_bits, codes, alpha, idx):
    dy_bits = _c(dy_bits, np.uint16)
    codes = _c(codes, np.int8)
    alpha = _c(alpha, np.float64)
    idx = _c(idx, np.int64)
    out = np.zeros(idx.size, np.float64)
    d = desc.as_array()
    if _load().orc_conv_bwd_data_sampled_bf16(_ptr(d), _ptr(dy_bits), _ptr(codes), _ptr(alpha),
                                              _ptr(idx), idx.size, _ptr(out)) != 0:
        raise OracleError("conv_bwd_data_sampled failed")
    return out


def conv_bwd_weight_sampled(desc, x_bits, dy_bits, idx):
    x_bits = _c(x_bits, np.uint16)
    dy_bits = _c(dy_bits, np.uint16)
    idx = _c(idx, np.int64)
    out = np.zeros(idx.size, np.float64)
    d = desc.as_array()
    if _load().orc_conv_bwd_weight_sampled_bf16(_ptr(d), _ptr(x_bits), _ptr(dy_bits),
                                                _ptr(idx), idx.size, _ptr(out)) != 0:
        raise OracleError("conv_bwd_weight_sampled failed")
    return out


# --------------------------------------------------------------------------------------
# Algorithm 1 update step with the Sec. 4 optimiser
# --------------------------------------------------------------------------------------
def sgd(w, v, g, eta, mu=0.9, lam=1e-4):
    """Returns (w_new, v_new) in fp64; inputs are not modified."""
    w = np.array(w, dtype=np.float64, copy=True).ravel()
    v = np.array(v, dtype=np.float64, copy=True).ravel()
    g = _c(g, np.float64).ravel()
    _load().orc_sgd(_ptr(w), _ptr(v), _ptr(g), w.size, float(eta), float(mu), float(lam))
    return w, v


def sgd_f32(w, v, g, eta, mu=0.9, lam=1e-4):
    """The SGD step in fp32 with fused multiply-adds (the rounding that decides the next
    codes).  Returns (w_new, v_new) fp32; inputs are not modified."""
    w = np.array(w, dtype=np.float32, copy=True).ravel()
    v = np.array(v, dtype=np.float32, copy=True).ravel()
    g = _c(g, np.float32).ravel()
    _load().orc_sgd_f32(_ptr(w), _ptr(v), _ptr(g), w.size, float(eta), float(mu), float(lam))
    return w, v


# --------------------------------------------------------------------------------------
# Layers around the two-bit convolutions (Sec. 4: ResNet-18 with batch normalisation)
# --------------------------------------------------------------------------------------
def maxpool_fwd(x, k, s, p):
    """x NHWC fp64 -> (y, argmax flat input index; ties to the first in window order)."""
    x = _c(x, np.float64)
    N, H, W, C = x.shape
    dims = np.array([N, H, W, C, k, s, p], np.int32)
    P, Q = (H + 2 * p - k) // s + 1, (W + 2 * p - k) // s + 1
    y = np.zeros((N, P, Q, C))
    arg = np.zeros((N, P, Q, C), np.int64)
    if _load().orc_maxpool_fwd(_ptr(dims), _ptr(x), _ptr(y), _ptr(arg)) != 0:
        raise OracleError("maxpool_fwd: bad geometry")
    return y, arg


def maxpool_bwd(dy, arg, x_shape, k, s, p):
    dy = _c(dy, np.float64)
    arg = _c(arg, np.int64)
    N, H, W, C = x_shape
    dims = np.array([N, H, W, C, k, s, p], np.int32)
    dx = np.zeros(x_shape)
    _load().orc_maxpool_bwd(_ptr(dims), _ptr(dy), _ptr(arg), _ptr(dx))
    return dx


def avgpool_global(x):
    x = _c(x, np.float64)
    N, H, W, C = x.shape
    dims = np.array([N, H, W, C], np.int32)
    y = np.zeros((N, C))
    _load().orc_avgpool_global(_ptr(dims), _ptr(x), _ptr(y))
    return y


def bn_infer(x, gamma, beta, mean, var, eps=1e-5):
    x = _c(x, np.float64)
    C = x.shape[-1]
    y = np.zeros_like(x)
    _load().orc_bn_infer(_ptr(x), x.size // C, C, _ptr(_c(gamma, np.float64)), _ptr(_c(beta, np.float64)),
                         _ptr(_c(mean, np.float64)), _ptr(_c(var, np.float64)), float(eps), _ptr(y))
    return y


def bn_train_fwd(x, gamma, beta, eps=1e-5):
    x = _c(x, np.float64)
    C = x.shape[-1]
    y = np.zeros_like(x)
    mean = np.zeros(C)
    var = np.zeros(C)
    _load().orc_bn_train_fwd(_ptr(x), x.size // C, C, _ptr(_c(gamma, np.float64)), _ptr(_c(beta, np.float64)),
                             float(eps), _ptr(y), _ptr(mean), _ptr(var))
    return y, mean, var


def bn_train_bwd(x, dy, gamma, eps=1e-5):
    x = _c(x, np.float64)
    dy = _c(dy, np.float64)
    C = x.shape[-1]
    dx = np.zeros_like(x)
    dg = np.zeros(C)
    db = np.zeros(C)
    _load().orc_bn_train_bwd(_ptr(x), _ptr(dy), x.size // C, C, _ptr(_c(gamma, np.float64)), float(eps),
                             _ptr(dx), _ptr(dg), _ptr(db))
    return dx, dg, db


def softmax_xent(z, labels):
    """Mean softmax cross-entropy and its gradient with respect to the logits."""
    z = _c(z, np.float64)
    labels = _c(labels, np.int64)
    N, K = z.shape
    dz = np.zeros_like(z)
    loss = _load().orc_softmax_xent(_ptr(z), _ptr(labels), N, K, _ptr(dz))
    return loss, dz
