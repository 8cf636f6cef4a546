"""Two-Bit Networks (arXiv 1701.00485) hot path on MI355X: Python binding of libtbn.

A thin ctypes layer over the C ABI in ``include/tbn.h``.  It only marshals arguments:
torch supplies device memory and the current stream, and every step of the computation
runs in the library's HIP kernels.  If ``libtbn.so`` is missing or does not load, every
call raises; there is no fallback.

Calls (same names as the C ABI, without the ``tbn_`` prefix):
  quantize(w)                      Sec. 2 Eq. (3)-(5)   -> packed codes, alpha, counts
  quantize_variant(w, threshold, uniform)  other thresholds / stochastic discretisation
  conv2d_fwd(desc, x, codes, alpha) Sec. 2 Eq. (1)       -> y
  conv2d_bwd_data(desc, dy, codes, alpha)  Sec. 3        -> dx
  conv2d_bwd_weight(desc, x, dy)    Sec. 3 (straight-through) -> dW
  sgd_step(w, v, g, lr, momentum, weight_decay)  Sec. 4 optimiser
  sgd_step_quantize(w, v, g, lr, ...)  the update fused with the next quantisation
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtbn.so")

TBN_BF16, TBN_F32 = 0, 1
OP_FWD, OP_BWD_DATA, OP_BWD_WEIGHT = 0, 1, 2

_lib = None


class TbnError(RuntimeError):
    def __init__(self, status: int, call: str, detail: str):
        self.status = status
        super().__init__("%s failed: %s (%s)" % (call, _status_name(status), detail))


class ConvDesc(ctypes.Structure):
    """Layer geometry: input N x H x W x C (NHWC), K filters of R x S x C."""

    _fields_ = [(f, ctypes.c_int32) for f in
                ("n", "h", "w", "c", "k", "r", "s", "stride_h", "stride_w", "pad_h", "pad_w")]

    def __init__(self, n, h, w, c, k, r, s, stride=1, pad=0, stride_w=None, pad_w=None):
        super().__init__(n, h, w, c, k, r, s, stride, stride if stride_w is None else stride_w,
                         pad, pad if pad_w is None else pad_w)

    def out_dims(self):
        p, q = ctypes.c_int32(), ctypes.c_int32()
        _call("tbn_conv_out_dims", ctypes.byref(self), ctypes.byref(p), ctypes.byref(q))
        return p.value, q.value

    def __repr__(self):
        return "ConvDesc(n=%d,h=%d,w=%d,c=%d,k=%d,r=%d,s=%d,stride=%d/%d,pad=%d/%d)" % (
            self.n, self.h, self.w, self.c, self.k, self.r, self.s, self.stride_h, self.stride_w,
            self.pad_h, self.pad_w)


class Epilogue(ctypes.Structure):
    _fields_ = [("scale", ctypes.c_void_p), ("bias", ctypes.c_void_p), ("residual", ctypes.c_void_p),
                ("relu", ctypes.c_int32)]


def load():
    """Load libtbn.so (built in-tree by build.py); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libtbn.so not built: run `python -c 'import __graft_entry__ as g; g.build()'`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    sigs = {
        "tbn_status_str": ([i32], ctypes.c_char_p),
        "tbn_last_error": ([], ctypes.c_char_p),
        "tbn_conv_out_dims": ([vp, vp, vp], i32),
        "tbn_packed_words": ([i64, i64], i64),
        "tbn_packed_row_words": ([i64], i64),
        "tbn_packed_bytes": ([i64, i64], i64),
        "tbn_workspace_size": ([i32, vp, vp], i32),
        "tbn_quantize": ([vp, i64, i64, vp, vp, vp, vp], i32),
        "tbn_quantize_variant": ([vp, i64, i64, f32, vp, vp, vp, vp, vp], i32),
        "tbn_conv2d_fwd": ([vp, vp, i32, vp, vp, vp, vp, i32, vp, ctypes.c_size_t, vp], i32),
        "tbn_conv2d_fwd_dense": ([vp, vp, i32, vp, vp, vp, i32, vp], i32),
        "tbn_quantize_act_i8": ([vp, i32, i64, f32, vp, vp], i32),
        "tbn_conv2d_fwd_i8": ([vp, vp, vp, vp, f32, i32, vp, i32, vp], i32),
        "tbn_quantize_act_fp8": ([vp, i32, i64, f32, vp, vp], i32),
        "tbn_repack_codes_fp4": ([vp, i64, vp, vp], i32),
        "tbn_conv2d_fwd_fp8": ([vp, vp, vp, vp, f32, i32, vp, i32, vp], i32),
        "tbn_conv2d_bwd_data": ([vp, vp, vp, vp, vp, i32, vp, ctypes.c_size_t, vp], i32),
        "tbn_conv2d_bwd_weight": ([vp, vp, vp, vp, i32, vp, ctypes.c_size_t, vp], i32),
        "tbn_sgd_step": ([vp, vp, vp, i64, f32, f32, f32, vp], i32),
        "tbn_sgd_step_quantize": ([vp, vp, vp, i64, i64, f32, f32, f32, vp, vp, vp, vp], i32),
        "tbn_pool_out_dims": ([vp, vp, vp], i32),
        "tbn_maxpool2d_fwd": ([vp, vp, vp, vp, vp], i32),
        "tbn_maxpool2d_bwd": ([vp, vp, vp, vp, i32, vp], i32),
        "tbn_avgpool_global": ([i32, i32, i32, i32, vp, vp, i32, vp], i32),
        "tbn_batchnorm_workspace_size": ([i64, i32, vp], i32),
        "tbn_batchnorm_train_fwd": ([vp, i64, i32, vp, vp, f32, i32, vp, vp, vp, vp, ctypes.c_size_t, vp], i32),
        "tbn_batchnorm_train_bwd": ([vp, vp, vp, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp],
                                    i32),
        "tbn_relu_bwd": ([vp, vp, i64, vp, vp], i32),
        "tbn_softmax_xent": ([vp, vp, i32, i32, vp, vp, vp, vp], i32),
        "tbn_conv2d_fwd_noalloc": ([vp, vp, i32, vp, vp, vp, vp, i32, vp], i32),
        "tbn_tuning_set": ([i32, i32], i32),
        "tbn_tuning_get": ([i32], i32),
    }
    for name, (args, res) in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def exported_symbols():
    return sorted(["tbn_status_str", "tbn_last_error", "tbn_conv_out_dims", "tbn_packed_words",
                   "tbn_packed_row_words", "tbn_packed_bytes",
                   "tbn_workspace_size", "tbn_quantize", "tbn_quantize_variant", "tbn_conv2d_fwd", "tbn_conv2d_fwd_dense",
                   "tbn_quantize_act_i8", "tbn_conv2d_fwd_i8",
                   "tbn_quantize_act_fp8", "tbn_repack_codes_fp4", "tbn_conv2d_fwd_fp8",
                   "tbn_conv2d_bwd_data",
                   "tbn_conv2d_bwd_weight", "tbn_sgd_step", "tbn_sgd_step_quantize", "tbn_pool_out_dims", "tbn_maxpool2d_fwd",
                   "tbn_maxpool2d_bwd", "tbn_avgpool_global", "tbn_batchnorm_workspace_size",
                   "tbn_batchnorm_train_fwd", "tbn_batchnorm_train_bwd", "tbn_relu_bwd", "tbn_softmax_xent",
                   "tbn_tuning_set", "tbn_tuning_get", "tbn_conv2d_fwd_noalloc"])


# Test and tuning knobs of include/tbn_tuning.h (names -> tbn_knob values).  Production code
# leaves them unset; the parity tests force every kernel variant through them.
KNOBS = {"conv_tile": 0, "conv_splits": 1, "wgrad_cfg": 2, "wgrad_pix": 3, "wgrad_pf": 4, "i8_tile": 5,
         "fc_variant": 6, "fp8_tile": 7}


def tuning_get(name: str) -> int:
    return int(load().tbn_tuning_get(KNOBS[name]))


def tuning_set(name: str, value: int) -> None:
    _call("tbn_tuning_set", KNOBS[name], int(value))


class tuning:
    """Context manager that sets knobs for its body and restores their previous values:
    ``with tbn.tuning(conv_tile=18, conv_splits=3): ...``."""

    def __init__(self, **knobs):
        for k in knobs:
            if k not in KNOBS:
                raise KeyError("unknown tuning knob %r" % k)
        self.knobs = {k: int(v) for k, v in knobs.items()}
        self.saved = {}

    def __enter__(self):
        for k, v in self.knobs.items():
            self.saved[k] = tuning_get(k)
            tuning_set(k, v)
        return self

    def __exit__(self, *exc):
        for k, v in self.saved.items():
            tuning_set(k, v)
        return False


def _status_name(s: int) -> str:
    try:
        return load().tbn_status_str(s).decode()
    except Exception:
        return str(s)


def _call(name, *args):
    lib = load()
    st = getattr(lib, name)(*args)
    if st != 0:
        raise TbnError(st, name, lib.tbn_last_error().decode())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t: torch.Tensor, name: str, dtypes=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("%s must be a CUDA (HIP) tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous (NHWC order for activations)" % name)
    if dtypes is not None and t.dtype not in dtypes:
        raise TypeError("%s has dtype %s, expected one of %s" % (name, t.dtype, dtypes))
    return ctypes.c_void_p(t.data_ptr())


def _dtype_code(dt):
    if dt == torch.bfloat16:
        return TBN_BF16
    if dt == torch.float32:
        return TBN_F32
    raise TypeError("unsupported dtype %s" % dt)


def packed_words(k: int, n: int) -> int:
    return int(load().tbn_packed_words(k, n))


def packed_row_words(n: int) -> int:
    return int(load().tbn_packed_row_words(n))


def packed_bytes(k: int, n: int) -> int:
    return int(load().tbn_packed_bytes(k, n))


def workspace_size(op: int, desc: ConvDesc) -> int:
    b = ctypes.c_size_t()
    _call("tbn_workspace_size", op, ctypes.byref(desc), ctypes.byref(b))
    return b.value


def workspace(op: int, desc: ConvDesc, device="cuda"):
    n = workspace_size(op, desc)
    return torch.empty(max(n, 16), dtype=torch.uint8, device=device)


def _numel(t, expect, name):
    if t.numel() != expect:
        raise ValueError("%s has %d elements, expected %d" % (name, t.numel(), expect))


def quantize(w: torch.Tensor, codes=None, alpha=None, counts=None, want_counts=True):
    """w: [K][n] fp32 (or [K][R][S][C]).  Returns (codes int32 words, alpha fp32, counts)."""
    K = w.shape[0]
    n = w.numel() // K
    pw = _dev(w, "w", (torch.float32,))
    if codes is None:
        codes = torch.empty(packed_words(K, n), dtype=torch.int32, device=w.device)
    if alpha is None:
        alpha = torch.empty(K, dtype=torch.float32, device=w.device)
    if counts is None and want_counts:
        counts = torch.empty((K, 2), dtype=torch.int32, device=w.device)
    _numel(codes, packed_words(K, n), "codes")
    _numel(alpha, K, "alpha")
    pc = _dev(counts, "counts", (torch.int32,)) if counts is not None else None
    _call("tbn_quantize", pw, K, n, _dev(codes, "codes", (torch.int32,)),
          _dev(alpha, "alpha", (torch.float32,)), pc, _stream())
    return codes, alpha, counts


def quantize_variant(w: torch.Tensor, threshold=1.0, uniform=None, codes=None, alpha=None, counts=None,
                     want_counts=True):
    """Discretisation variants: magnitude threshold `threshold` (Eq. 3 has 1), or stochastic
    discretisation driven by `uniform` ([K][n] fp32 in [0, 1)).  Returns (codes, alpha, counts)."""
    K = w.shape[0]
    n = w.numel() // K
    pw = _dev(w, "w", (torch.float32,))
    pu = None
    if uniform is not None:
        _numel(uniform, K * n, "uniform")
        pu = _dev(uniform, "uniform", (torch.float32,))
    if codes is None:
        codes = torch.empty(packed_words(K, n), dtype=torch.int32, device=w.device)
    if alpha is None:
        alpha = torch.empty(K, dtype=torch.float32, device=w.device)
    if counts is None and want_counts:
        counts = torch.empty((K, 2), dtype=torch.int32, device=w.device)
    _numel(codes, packed_words(K, n), "codes")
    _numel(alpha, K, "alpha")
    pc = _dev(counts, "counts", (torch.int32,)) if counts is not None else None
    _call("tbn_quantize_variant", pw, K, n, float(threshold), pu, _dev(codes, "codes", (torch.int32,)),
          _dev(alpha, "alpha", (torch.float32,)), pc, _stream())
    return codes, alpha, counts


NOALLOC_SCRATCH_BYTES = 8 << 20  # TBN_NOALLOC_SCRATCH_BYTES of include/tbn.h


def conv2d_fwd_noalloc(desc: ConvDesc, x, codes, alpha, y, scale=None, bias=None, residual=None, relu=False):
    """tbn_conv2d_fwd_noalloc: the forward pass with the library's static scratch as its
    workspace (for callers that cannot allocate); `y` is caller-provided."""
    P, Q = desc.out_dims()
    _numel(x, desc.n * desc.h * desc.w * desc.c, "x")
    _numel(codes, packed_words(desc.k, desc.r * desc.s * desc.c), "codes")
    _numel(alpha, desc.k, "alpha")
    _numel(y, desc.n * P * Q * desc.k, "y")
    ep = None
    if scale is not None or bias is not None or residual is not None or relu:
        if residual is not None:
            _numel(residual, y.numel(), "residual")
            if residual.dtype != y.dtype:
                raise TypeError("residual must have y's dtype")
        ep = Epilogue(_dev(scale, "scale", (torch.float32,)).value if scale is not None else None,
                      _dev(bias, "bias", (torch.float32,)).value if bias is not None else None,
                      _dev(residual, "residual").value if residual is not None else None,
                      1 if relu else 0)
    _call("tbn_conv2d_fwd_noalloc", ctypes.byref(desc), _dev(x, "x", (torch.bfloat16, torch.float32)),
          _dtype_code(x.dtype), _dev(codes, "codes", (torch.int32,)), _dev(alpha, "alpha", (torch.float32,)),
          ctypes.byref(ep) if ep is not None else None, _dev(y, "y", (torch.bfloat16, torch.float32)),
          _dtype_code(y.dtype), _stream())
    return y


def conv2d_fwd(desc: ConvDesc, x, codes, alpha, y=None, out_dtype=torch.bfloat16, scale=None, bias=None,
               residual=None, relu=False, ws=None):
    """y = act(alpha_k * scale_k * (x conv W~) + bias_k + residual), NHWC.  `ws`: workspace
    of workspace_size(OP_FWD, desc) bytes (allocated here when None and needed)."""
    P, Q = desc.out_dims()
    _numel(x, desc.n * desc.h * desc.w * desc.c, "x")
    _numel(codes, packed_words(desc.k, desc.r * desc.s * desc.c), "codes")
    _numel(alpha, desc.k, "alpha")
    if y is None:
        y = torch.empty((desc.n, P, Q, desc.k), dtype=out_dtype, device=x.device)
    _numel(y, desc.n * P * Q * desc.k, "y")
    ep = None
    if scale is not None or bias is not None or residual is not None or relu:
        if residual is not None:
            _numel(residual, y.numel(), "residual")
            if residual.dtype != y.dtype:
                raise TypeError("residual must have y's dtype")
        ep = Epilogue(_dev(scale, "scale", (torch.float32,)).value if scale is not None else None,
                      _dev(bias, "bias", (torch.float32,)).value if bias is not None else None,
                      _dev(residual, "residual").value if residual is not None else None,
                      1 if relu else 0)
    if ws is None:
        need = workspace_size(OP_FWD, desc)
        ws = torch.empty(need, dtype=torch.uint8, device=x.device) if need else None
    _call("tbn_conv2d_fwd", ctypes.byref(desc), _dev(x, "x", (torch.bfloat16, torch.float32)),
          _dtype_code(x.dtype), _dev(codes, "codes", (torch.int32,)), _dev(alpha, "alpha", (torch.float32,)),
          ctypes.byref(ep) if ep is not None else None, _dev(y, "y", (torch.bfloat16, torch.float32)),
          _dtype_code(y.dtype), _dev(ws, "ws") if ws is not None else None,
          ws.numel() * ws.element_size() if ws is not None else 0, _stream())
    return y


def quantize_act_i8(x: torch.Tensor, inv_scale: float, q=None):
    """int8 activation codes q = clamp(round-half-even(x * inv_scale), -127, 127) (NaN -> 0),
    elementwise over a bf16 or fp32 tensor; returns q (int8, x's shape)."""
    if q is None:
        q = torch.empty(x.shape, dtype=torch.int8, device=x.device)
    _numel(q, x.numel(), "q")
    _call("tbn_quantize_act_i8", _dev(x, "x", (torch.bfloat16, torch.float32)), _dtype_code(x.dtype), x.numel(),
          float(inv_scale), _dev(q, "q", (torch.int8,)), _stream())
    return q


def conv2d_fwd_i8(desc: ConvDesc, xq, codes, alpha, x_scale: float, y=None, out_dtype=torch.bfloat16, relu=False):
    """Forward pass on int8 activation codes (int8 matrix cores):
    y = act(float(xq conv W~) * float(alpha_k * x_scale)), NHWC."""
    P, Q = desc.out_dims()
    _numel(xq, desc.n * desc.h * desc.w * desc.c, "xq")
    _numel(codes, packed_words(desc.k, desc.r * desc.s * desc.c), "codes")
    _numel(alpha, desc.k, "alpha")
    if y is None:
        y = torch.empty((desc.n, P, Q, desc.k), dtype=out_dtype, device=xq.device)
    _numel(y, desc.n * P * Q * desc.k, "y")
    _call("tbn_conv2d_fwd_i8", ctypes.byref(desc), _dev(xq, "xq", (torch.int8,)), _dev(codes, "codes", (torch.int32,)),
          _dev(alpha, "alpha", (torch.float32,)), float(x_scale), 1 if relu else 0,
          _dev(y, "y", (torch.bfloat16, torch.float32)), _dtype_code(y.dtype), _stream())
    return y


def quantize_act_fp8(x: torch.Tensor, inv_scale: float, q=None):
    """E4M3 activation codes f = E4M3(x * inv_scale) (nearest, ties to even, saturating at
    +-448, NaN -> 0), elementwise over a bf16 or fp32 tensor; returns the codes (uint8)."""
    if q is None:
        q = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    _numel(q, x.numel(), "q")
    _call("tbn_quantize_act_fp8", _dev(x, "x", (torch.bfloat16, torch.float32)), _dtype_code(x.dtype), x.numel(),
          float(inv_scale), _dev(q, "q", (torch.uint8,)), _stream())
    return q


def repack_codes_fp4(codes, out=None):
    """The packed codes rewritten in the E2M1 operand layout of conv2d_fwd_fp8 (int32, same size)."""
    if out is None:
        out = torch.empty_like(codes)
    _numel(out, codes.numel(), "out")
    _call("tbn_repack_codes_fp4", _dev(codes, "codes", (torch.int32,)), codes.numel(),
          _dev(out, "out", (torch.int32,)), _stream())
    return out


def conv2d_fwd_fp8(desc: ConvDesc, xq, codes_fp4, alpha, x_scale: float, y=None, out_dtype=torch.bfloat16,
                   relu=False):
    """Forward pass on E4M3 activation codes (scaled fp8 x fp4 matrix cores):
    y = act((f conv W~) * float(alpha_k * x_scale)), NHWC; codes_fp4 from repack_codes_fp4."""
    P, Q = desc.out_dims()
    _numel(xq, desc.n * desc.h * desc.w * desc.c, "xq")
    _numel(codes_fp4, packed_words(desc.k, desc.r * desc.s * desc.c), "codes")
    _numel(alpha, desc.k, "alpha")
    if y is None:
        y = torch.empty((desc.n, P, Q, desc.k), dtype=out_dtype, device=xq.device)
    _numel(y, desc.n * P * Q * desc.k, "y")
    _call("tbn_conv2d_fwd_fp8", ctypes.byref(desc), _dev(xq, "xq", (torch.uint8,)),
          _dev(codes_fp4, "codes", (torch.int32,)), _dev(alpha, "alpha", (torch.float32,)), float(x_scale),
          1 if relu else 0, _dev(y, "y", (torch.bfloat16, torch.float32)), _dtype_code(y.dtype), _stream())
    return y


def conv2d_fwd_dense(desc: ConvDesc, x, w, y=None, out_dtype=torch.bfloat16, scale=None, bias=None,
                     residual=None, relu=False):
    """Full-precision layer: y = act(scale_k * (x conv bf16(w)) + bias_k + residual), NHWC;
    w fp32 [K][R][S][C]."""
    P, Q = desc.out_dims()
    _numel(x, desc.n * desc.h * desc.w * desc.c, "x")
    _numel(w, desc.k * desc.r * desc.s * desc.c, "w")
    if y is None:
        y = torch.empty((desc.n, P, Q, desc.k), dtype=out_dtype, device=x.device)
    _numel(y, desc.n * P * Q * desc.k, "y")
    ep = None
    if scale is not None or bias is not None or residual is not None or relu:
        if residual is not None:
            _numel(residual, y.numel(), "residual")
            if residual.dtype != y.dtype:
                raise TypeError("residual must have y's dtype")
        ep = Epilogue(_dev(scale, "scale", (torch.float32,)).value if scale is not None else None,
                      _dev(bias, "bias", (torch.float32,)).value if bias is not None else None,
                      _dev(residual, "residual").value if residual is not None else None,
                      1 if relu else 0)
    _call("tbn_conv2d_fwd_dense", ctypes.byref(desc), _dev(x, "x", (torch.bfloat16, torch.float32)),
          _dtype_code(x.dtype), _dev(w, "w", (torch.float32,)), ctypes.byref(ep) if ep is not None else None,
          _dev(y, "y", (torch.bfloat16, torch.float32)), _dtype_code(y.dtype), _stream())
    return y


def conv2d_bwd_data(desc: ConvDesc, dy, codes, alpha, dx=None, out_dtype=torch.bfloat16, ws=None):
    P, Q = desc.out_dims()
    _numel(dy, desc.n * P * Q * desc.k, "dy")
    _numel(codes, packed_words(desc.k, desc.r * desc.s * desc.c), "codes")
    _numel(alpha, desc.k, "alpha")
    if dx is None:
        dx = torch.empty((desc.n, desc.h, desc.w, desc.c), dtype=out_dtype, device=dy.device)
    _numel(dx, desc.n * desc.h * desc.w * desc.c, "dx")
    if ws is None:
        ws = workspace(OP_BWD_DATA, desc, dy.device)
    _call("tbn_conv2d_bwd_data", ctypes.byref(desc), _dev(dy, "dy", (torch.bfloat16,)),
          _dev(codes, "codes", (torch.int32,)), _dev(alpha, "alpha", (torch.float32,)),
          _dev(dx, "dx", (torch.bfloat16, torch.float32)), _dtype_code(dx.dtype), _dev(ws, "ws"),
          ws.numel() * ws.element_size(), _stream())
    return dx


def conv2d_bwd_weight(desc: ConvDesc, x, dy, dw=None, accumulate=False, ws=None):
    P, Q = desc.out_dims()
    _numel(x, desc.n * desc.h * desc.w * desc.c, "x")
    _numel(dy, desc.n * P * Q * desc.k, "dy")
    if dw is None:
        dw = torch.empty((desc.k, desc.r, desc.s, desc.c), dtype=torch.float32, device=x.device)
    _numel(dw, desc.k * desc.r * desc.s * desc.c, "dw")
    if ws is None:
        ws = workspace(OP_BWD_WEIGHT, desc, x.device)
    _call("tbn_conv2d_bwd_weight", ctypes.byref(desc), _dev(x, "x", (torch.bfloat16,)),
          _dev(dy, "dy", (torch.bfloat16,)), _dev(dw, "dw", (torch.float32,)), 1 if accumulate else 0,
          _dev(ws, "ws"), ws.numel() * ws.element_size(), _stream())
    return dw


def sgd_step(w, v, g, lr, momentum=0.9, weight_decay=1e-4):
    n = w.numel()
    _numel(v, n, "v")
    _numel(g, n, "g")
    _call("tbn_sgd_step", _dev(w, "w", (torch.float32,)), _dev(v, "v", (torch.float32,)),
          _dev(g, "g", (torch.float32,)), n, float(lr), float(momentum), float(weight_decay), _stream())
    return w, v


def sgd_step_quantize(w, v, g, lr, momentum=0.9, weight_decay=1e-4, codes=None, alpha=None, counts=None,
                      want_counts=True):
    """SGD update of w [K][n] (in place, with momentum v) fused with the quantisation of
    the updated filters.  Returns (codes, alpha, counts) as quantize() does."""
    K = w.shape[0]
    n = w.numel() // K
    _numel(v, K * n, "v")
    _numel(g, K * n, "g")
    if codes is None:
        codes = torch.empty(packed_words(K, n), dtype=torch.int32, device=w.device)
    if alpha is None:
        alpha = torch.empty(K, dtype=torch.float32, device=w.device)
    if counts is None and want_counts:
        counts = torch.empty((K, 2), dtype=torch.int32, device=w.device)
    _numel(codes, packed_words(K, n), "codes")
    _numel(alpha, K, "alpha")
    pc = _dev(counts, "counts", (torch.int32,)) if counts is not None else None
    _call("tbn_sgd_step_quantize", _dev(w, "w", (torch.float32,)), _dev(v, "v", (torch.float32,)),
          _dev(g, "g", (torch.float32,)), K, n, float(lr), float(momentum), float(weight_decay),
          _dev(codes, "codes", (torch.int32,)), _dev(alpha, "alpha", (torch.float32,)), pc, _stream())
    return codes, alpha, counts


# --------------------------------------------------------------------------------------
# Layers around the two-bit convolutions
# --------------------------------------------------------------------------------------
class PoolDesc(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int32) for f in ("n", "h", "w", "c", "k", "stride", "pad")]

    def out_dims(self):
        p, q = ctypes.c_int32(), ctypes.c_int32()
        _call("tbn_pool_out_dims", ctypes.byref(self), ctypes.byref(p), ctypes.byref(q))
        return p.value, q.value


def maxpool2d_fwd(x, k, stride, pad, want_argmax=False):
    """x NHWC bf16 -> (y, argmax int32 or None)."""
    n, h, w, c = x.shape
    d = PoolDesc(n, h, w, c, k, stride, pad)
    P, Q = d.out_dims()
    y = torch.empty((n, P, Q, c), dtype=torch.bfloat16, device=x.device)
    arg = torch.empty((n, P, Q, c), dtype=torch.int32, device=x.device) if want_argmax else None
    _call("tbn_maxpool2d_fwd", ctypes.byref(d), _dev(x, "x", (torch.bfloat16,)), _dev(y, "y"),
          _dev(arg, "argmax", (torch.int32,)) if arg is not None else None, _stream())
    return y, arg


def maxpool2d_bwd(dy, argmax, x_shape, k, stride, pad, out_dtype=torch.bfloat16):
    n, h, w, c = x_shape
    d = PoolDesc(n, h, w, c, k, stride, pad)
    dx = torch.empty(tuple(x_shape), dtype=out_dtype, device=dy.device)
    _call("tbn_maxpool2d_bwd", ctypes.byref(d), _dev(dy, "dy", (torch.bfloat16,)),
          _dev(argmax, "argmax", (torch.int32,)), _dev(dx, "dx"), _dtype_code(out_dtype), _stream())
    return dx


def avgpool_global(x, out_dtype=torch.bfloat16):
    n, h, w, c = x.shape
    y = torch.empty((n, c), dtype=out_dtype, device=x.device)
    _call("tbn_avgpool_global", n, h, w, c, _dev(x, "x", (torch.bfloat16,)), _dev(y, "y"),
          _dtype_code(out_dtype), _stream())
    return y


def batchnorm_workspace_size(rows: int, c: int) -> int:
    b = ctypes.c_size_t()
    _call("tbn_batchnorm_workspace_size", int(rows), int(c), ctypes.byref(b))
    return b.value


def _bn_ws(rows, c, ws, device):
    need = batchnorm_workspace_size(rows, c)
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=device)
    return ws


def batchnorm_train_fwd(x, gamma, beta, eps=1e-5, relu=False, ws=None):
    c = x.shape[-1]
    rows = x.numel() // c
    y = torch.empty_like(x)
    mean = torch.empty(c, dtype=torch.float32, device=x.device)
    inv_std = torch.empty(c, dtype=torch.float32, device=x.device)
    ws = _bn_ws(rows, c, ws, x.device)
    _call("tbn_batchnorm_train_fwd", _dev(x, "x", (torch.bfloat16,)), rows, c,
          _dev(gamma, "gamma", (torch.float32,)), _dev(beta, "beta", (torch.float32,)), float(eps),
          1 if relu else 0, _dev(y, "y"), _dev(mean, "mean"), _dev(inv_std, "inv_std"), _dev(ws, "ws"),
          ws.numel() * ws.element_size(), _stream())
    return y, mean, inv_std


def batchnorm_train_bwd(x, y, dy, mean, inv_std, gamma, relu=False, ws=None, dgamma=None, dbeta=None):
    """Returns (dx, dgamma, dbeta); `dgamma` / `dbeta` may be caller-provided fp32 [C] outputs
    (for example views into one flat gradient buffer)."""
    c = x.shape[-1]
    rows = x.numel() // c
    dx = torch.empty_like(x)
    if dgamma is None:
        dgamma = torch.empty(c, dtype=torch.float32, device=x.device)
    if dbeta is None:
        dbeta = torch.empty(c, dtype=torch.float32, device=x.device)
    _numel(dgamma, c, "dgamma")
    _numel(dbeta, c, "dbeta")
    ws = _bn_ws(rows, c, ws, x.device)
    _call("tbn_batchnorm_train_bwd", _dev(x, "x", (torch.bfloat16,)), _dev(y, "y", (torch.bfloat16,)),
          _dev(dy, "dy", (torch.bfloat16,)), rows, c, 1 if relu else 0, _dev(mean, "mean"),
          _dev(inv_std, "inv_std"), _dev(gamma, "gamma"), _dev(dgamma, "dgamma"), _dev(dbeta, "dbeta"),
          _dev(dx, "dx"), _dev(ws, "ws"), ws.numel() * ws.element_size(), _stream())
    return dx, dgamma, dbeta


def relu_bwd(y, dy):
    dx = torch.empty_like(dy)
    _call("tbn_relu_bwd", _dev(y, "y", (torch.bfloat16,)), _dev(dy, "dy", (torch.bfloat16,)), dy.numel(),
          _dev(dx, "dx"), _stream())
    return dx


def softmax_xent(logits, labels):
    """logits fp32 [n][classes], labels int32 [n] -> (loss fp32 [1], dlogits bf16)."""
    n, k = logits.shape
    loss = torch.empty(1, dtype=torch.float32, device=logits.device)
    per = torch.empty(n, dtype=torch.float32, device=logits.device)
    dz = torch.empty((n, k), dtype=torch.bfloat16, device=logits.device)
    _call("tbn_softmax_xent", _dev(logits, "logits", (torch.float32,)), _dev(labels, "labels", (torch.int32,)),
          n, k, _dev(loss, "loss"), _dev(per, "per"), _dev(dz, "dz"), _stream())
    return loss, dz
