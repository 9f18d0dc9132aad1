"""ctypes wrapper around ``libcaffe_ref.so`` (the plain C oracle).

TEST INFRASTRUCTURE ONLY.  Every array is converted to contiguous float64
before the call and every result is float64.  The C library states the
definitions it implements (Caffe, Sec. 3.2 layer forward/backward roles; the
textbook strided, padded, grouped cross-correlation for convolution).
"""
import contextlib
import ctypes

import numpy as np

from .build import ensure_built

_lib = None
_lib_path = None  # another build of caffe_ref.c (see library())
_dp = ctypes.POINTER(ctypes.c_double)


@contextlib.contextmanager
def library(path):
    """Inside the block, every wrapper below calls the oracle library built
    at `path` instead of libcaffe_ref.so (the planted-mistake tests build
    altered copies of caffe_ref.c and run the pins against them)."""
    global _lib, _lib_path
    saved = _lib, _lib_path
    _lib, _lib_path = None, path
    try:
        yield
    finally:
        _lib, _lib_path = saved


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(_lib_path or ensure_built())
        i = ctypes.c_int
        d = ctypes.c_double
        lib.caffe_ref_num_threads.restype = i
        lib.caffe_ref_conv_out_shape.argtypes = [i] * 8 + [ctypes.POINTER(i)] * 2
        lib.caffe_ref_conv_forward.argtypes = [i] * 13 + [_dp] * 4
        lib.caffe_ref_conv_backward.argtypes = [i] * 13 + [_dp] * 7
        lib.caffe_ref_maxpool_forward.argtypes = [i] * 7 + [_dp] * 2
        lib.caffe_ref_maxpool_backward.argtypes = [i] * 7 + [_dp] * 3
        lib.caffe_ref_lrn_forward.argtypes = [i] * 5 + [d] * 3 + [_dp] * 2
        lib.caffe_ref_lrn_backward.argtypes = [i] * 5 + [d] * 3 + [_dp] * 3
        for f in ("caffe_ref_conv_out_shape", "caffe_ref_conv_forward", "caffe_ref_conv_backward",
                  "caffe_ref_maxpool_forward", "caffe_ref_maxpool_backward",
                  "caffe_ref_lrn_forward", "caffe_ref_lrn_backward"):
            getattr(lib, f).restype = i
        _lib = lib
    return _lib


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(_dp)


def num_threads() -> int:
    return _load().caffe_ref_num_threads()


def conv_out_shape(H, W, kh, kw, sh, sw, ph, pw):
    Ho, Wo = ctypes.c_int(), ctypes.c_int()
    rc = _load().caffe_ref_conv_out_shape(H, W, kh, kw, sh, sw, ph, pw,
                                          ctypes.byref(Ho), ctypes.byref(Wo))
    if rc:
        raise ValueError("invalid convolution geometry")
    return Ho.value, Wo.value


def _conv_args(x_shape, w_shape, stride, pad, group):
    N, C, H, W = x_shape
    K, Cg, kh, kw = w_shape
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    if Cg * group != C:
        raise ValueError("weight channels x group != input channels")
    return N, C, H, W, K, kh, kw, sh, sw, ph, pw, group


def conv_forward(x, w, b=None, stride=1, pad=0, group=1, relu=False):
    """Y = [relu] (W * X + b): the forward pass, fp64 in and out."""
    x, w, b = _f64(x), _f64(w), _f64(b)
    a = _conv_args(x.shape, w.shape, stride, pad, group)
    N, C, H, W, K, kh, kw, sh, sw, ph, pw, g = a
    Ho, Wo = conv_out_shape(H, W, kh, kw, sh, sw, ph, pw)
    y = np.empty((N, K, Ho, Wo), np.float64)
    rc = _load().caffe_ref_conv_forward(*a, int(bool(relu)), _ptr(x), _ptr(w), _ptr(b), _ptr(y))
    if rc:
        raise ValueError("invalid convolution arguments")
    return y


def conv_backward(x, w, top_diff, top=None, stride=1, pad=0, group=1, relu=False,
                  need=("dx", "dw", "db")):
    """Returns (dx, dw, db) (None where not requested) for D = G [Y > 0] (relu) or G."""
    x, w, g, top = _f64(x), _f64(w), _f64(top_diff), _f64(top)
    a = _conv_args(x.shape, w.shape, stride, pad, group)
    dx = np.empty(x.shape, np.float64) if "dx" in need else None
    dw = np.empty(w.shape, np.float64) if "dw" in need else None
    db = np.empty((w.shape[0],), np.float64) if "db" in need else None
    rc = _load().caffe_ref_conv_backward(*a, int(bool(relu)), _ptr(x), _ptr(w), _ptr(top), _ptr(g),
                                         _ptr(dx), _ptr(dw), _ptr(db))
    if rc:
        raise ValueError("invalid convolution arguments")
    return dx, dw, db


def maxpool_forward(x, k, s, p=0):
    x = _f64(x)
    N, C, H, W = x.shape
    Ho, Wo = conv_out_shape(H, W, k, k, s, s, p, p)
    y = np.empty((N, C, Ho, Wo), np.float64)
    if _load().caffe_ref_maxpool_forward(N, C, H, W, k, s, p, _ptr(x), _ptr(y)):
        raise ValueError("invalid pooling arguments")
    return y


def maxpool_backward(x, top_diff, k, s, p=0):
    x, g = _f64(x), _f64(top_diff)
    N, C, H, W = x.shape
    dx = np.empty(x.shape, np.float64)
    if _load().caffe_ref_maxpool_backward(N, C, H, W, k, s, p, _ptr(x), _ptr(g), _ptr(dx)):
        raise ValueError("invalid pooling arguments")
    return dx


def lrn_forward(x, size=5, alpha=1e-4, beta=0.75, k=1.0):
    x = _f64(x)
    N, C, H, W = x.shape
    y = np.empty(x.shape, np.float64)
    if _load().caffe_ref_lrn_forward(N, C, H, W, size, alpha, beta, k, _ptr(x), _ptr(y)):
        raise ValueError("invalid LRN arguments")
    return y


def lrn_backward(x, top_diff, size=5, alpha=1e-4, beta=0.75, k=1.0):
    x, g = _f64(x), _f64(top_diff)
    N, C, H, W = x.shape
    dx = np.empty(x.shape, np.float64)
    if _load().caffe_ref_lrn_backward(N, C, H, W, size, alpha, beta, k, _ptr(x), _ptr(g), _ptr(dx)):
        raise ValueError("invalid LRN arguments")
    return dx
