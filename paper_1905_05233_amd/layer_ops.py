"""Python binding of the library's operations around the layer (argument
marshalling only; the work runs in the gfx950 kernels of layer_ops.hip):
ReLU and 2x2 max-pooling, a float64 direct convolution and the error sums of
a result against it."""
import ctypes
import math

import torch

from . import _native as N

_DTYPE_OF = {torch.float32: "f32", torch.float16: "f16", torch.bfloat16: "bf16"}


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _desc(t, name):
    if not t.is_cuda or not t.is_contiguous() or t.dim() != 4:
        raise ValueError(f"{name} must be a contiguous 4-D device tensor")
    return N.WgTensor(ctypes.c_void_p(t.data_ptr()), *[int(v) for v in t.shape])


def _dtype_code(t):
    if t.dtype not in _DTYPE_OF:
        raise TypeError(f"unsupported dtype {t.dtype}")
    return N.DTYPE_CODES[_DTYPE_OF[t.dtype]]


def relu_pool(x, pool, out=None, stream=None):
    """ReLU of an NHWC tensor, then 2x2 stride-2 max-pooling if ``pool``."""
    Nn, H, W, C = x.shape
    shape = (Nn, H // 2, W // 2, C) if pool else (Nn, H, W, C)
    y = torch.empty(shape, dtype=x.dtype, device=x.device) if out is None else out
    xt, yt = _desc(x, "x"), _desc(y, "y")
    N.check(N.lib().winograd_relu_pool(_dtype_code(x), ctypes.byref(xt), ctypes.byref(yt), 1 if pool else 0,
                                       _stream(stream)))
    return y


def direct_conv_f64(x, w, stream=None):
    """float64 direct convolution of x [N][H][W][C] with w [K][3][3][C] (pad 1)
    or, for w [K][1][3][C], of each row along W (pad 1); x and w in their
    storage dtype.  Returns y [N][H][W][K] float64."""
    if x.dtype != w.dtype:
        raise TypeError("x and w must share a dtype")
    Nn, H, W, _ = x.shape
    y = torch.empty((Nn, H, W, w.shape[0]), dtype=torch.float64, device=x.device)
    xt, wt = _desc(x, "x"), _desc(w, "w")
    N.check(N.lib().winograd_direct_conv_f64(_dtype_code(x), ctypes.byref(xt), ctypes.byref(wt),
                                             ctypes.c_void_p(y.data_ptr()), _stream(stream)))
    return y


def error_sums(y, ref, stream=None):
    """(sum (y - ref)^2, sum ref^2) in float64, reduced on the device."""
    if y.numel() != ref.numel() or ref.dtype != torch.float64 or not (y.is_contiguous() and ref.is_contiguous()):
        raise ValueError("y and a contiguous float64 ref of the same size are needed")
    sums = torch.empty(N.SQ_SUMS_DOUBLES, dtype=torch.float64, device=y.device)
    N.check(N.lib().winograd_sq_error_sums(_dtype_code(y), ctypes.c_void_p(y.data_ptr()),
                                           ctypes.c_void_p(ref.data_ptr()), y.numel(),
                                           ctypes.c_void_p(sums.data_ptr()), _stream(stream)))
    e2, r2 = sums[:2].cpu().tolist()
    return e2, r2


def rel_l2(y, ref, stream=None):
    """||y - ref||_2 / ||ref||_2 with both sums from the device."""
    e2, r2 = error_sums(y, ref, stream)
    return math.sqrt(e2 / r2) if r2 > 0 else math.sqrt(e2)
