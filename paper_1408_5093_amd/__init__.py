"""MI355X (gfx950) convolution layer of Caffe (Jia et al., 2014): Python binding.

The layer (paper Sec. 3.2: forward pass, and a backward pass giving the
parameter and input gradients) runs entirely in the HIP kernels of
``libcaffe_conv.so`` behind the C ABI in ``include/caffe_conv.h`` and
``include/caffe_layers.h``.  This module only marshals arguments: it takes
PyTorch device tensors, checks dtype/device/contiguity, and passes their data
pointers and the current HIP stream.  The functions named ``caffe_*`` take
the same arguments as their C counterparts; the short names allocate outputs
and workspace with PyTorch and call them.
"""
import ctypes

import torch

from . import _lib
from ._lib import (  # noqa: F401
    CAFFE_ERR_UNSUPPORTED, CAFFE_ERR_WORKSPACE, NOALLOC_SCRATCH_BYTES, BACKWARD_BOTTOM_STAGED,
    BACKWARD_MASK_BOTTOM_DIFF, BACKWARD_POOL_MASK_OFFSETS, BACKWARD_TOP_DIFF_MASKED,
    BACKWARD_TOP_STAGED,
    FORWARD_BOTTOM_STAGED, CAFFE_BF16, CAFFE_BF16_F32_BOTTOM, CAFFE_F32, CAFFE_LR_EXP,
    CAFFE_LR_FIXED, CAFFE_LR_INV, CAFFE_LR_STEP, LrSchedule, PASS_BACKWARD,
    PASS_BACKWARD_DATA, PASS_BACKWARD_POOL_LRN, PASS_BACKWARD_WEIGHTS, PASS_FORWARD,
    POOL_LRN_STAGE_ONLY, POOL_MASK_OFFSETS, POOL_RELU_INPUT, CaffeError, ConvDesc,
    LrnDesc, PoolDesc, check, load, LIB_PATH,
)

__all__ = [
    "conv_desc", "conv_out_shape", "conv_workspace_size", "conv_forward", "conv_backward",
    "conv_backward_data", "conv_backward_weights", "maxpool_forward", "maxpool_backward",
    "lrn_forward", "lrn_backward", "cast_f32_to_bf16", "Workspace", "CaffeError",
    "sgd_learning_rate", "softmax_loss", "sgd_update", "pool_lrn_forward", "lrn_pool_backward",
    "pool_lrn_supported", "caffe_conv_backward_pool_lrn", "relu_backward",
    "caffe_conv_backward_into", "conv_stage_below_supported", "pool_lrn_stage_supported",
]


def _pair(v):
    return (int(v), int(v)) if isinstance(v, int) else (int(v[0]), int(v[1]))


def conv_desc(x_shape, w_shape, stride=1, pad=0, group=1, relu=False, dtype=CAFFE_F32):
    """Descriptor for bottom x_shape = (N, C, H, W) and weight w_shape = (K, C/group, kh, kw)."""
    N, C, H, W = (int(d) for d in x_shape)
    K, Cg, kh, kw = (int(d) for d in w_shape)
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    if Cg * group != C:
        raise ValueError(f"weight has {Cg} channels per group but C={C}, group={group}")
    return ConvDesc(N, C, H, W, K, kh, kw, sh, sw, ph, pw, int(group), int(bool(relu)), int(dtype))


def conv_out_shape(desc):
    Ho, Wo = ctypes.c_int32(), ctypes.c_int32()
    check(load().caffe_conv_out_shape(ctypes.byref(desc), ctypes.byref(Ho), ctypes.byref(Wo)))
    return Ho.value, Wo.value


def conv_workspace_size(desc, pass_):
    n = ctypes.c_size_t()
    check(load().caffe_conv_workspace_size(ctypes.byref(desc), int(pass_), ctypes.byref(n)))
    return n.value


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t, name, dtype=None):
    if t is None:
        return
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")


class Workspace:
    """A growable device byte buffer for the library's scratch space."""

    def __init__(self, device=None):
        self.device = device
        self.buf = None

    def get(self, nbytes):
        if nbytes == 0:
            return None
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.empty(nbytes, dtype=torch.uint8, device=self.device or "cuda")
        return self.buf


def _op_dtype(desc):
    """dtype of the weight (and of the bottom, see _bottom_dtype)."""
    return torch.bfloat16 if desc.dtype in (CAFFE_BF16, CAFFE_BF16_F32_BOTTOM) else torch.float32


def _bottom_dtype(desc):
    return torch.bfloat16 if desc.dtype == CAFFE_BF16 else torch.float32


# ----------------------------------------------------- C-ABI-shaped calls
def caffe_conv_forward(desc, bottom, weight, bias, top, workspace=None, stream=None, flags=0):
    """caffe_conv_forward, or with flags caffe_conv_forward_ex."""
    t = _op_dtype(desc)
    _dev(bottom, "bottom", _bottom_dtype(desc)), _dev(weight, "weight", t)
    _dev(bias, "bias", torch.float32)
    _dev(top, "top", torch.float32)
    ws_bytes = 0 if workspace is None else workspace.numel()
    args = (ctypes.byref(desc), _ptr(bottom), _ptr(weight), _ptr(bias), _ptr(top),
            _ptr(workspace), ws_bytes)
    if flags:
        check(load().caffe_conv_forward_ex(*args, int(flags), _stream(stream)))
    else:
        check(load().caffe_conv_forward(*args, _stream(stream)))


def caffe_conv_backward(desc, top_diff, top, bottom, weight, bottom_diff, weight_diff, bias_diff,
                        accumulate=0, flags=0, workspace=None, stream=None, weight_stream=None):
    """caffe_conv_backward, or with weight_stream caffe_conv_backward_ex (the
    weight and bias gradients ordered on that stream, not joined)."""
    t = _op_dtype(desc)
    for x, n in ((top_diff, "top_diff"), (top, "top"), (bottom_diff, "bottom_diff"),
                 (weight_diff, "weight_diff"), (bias_diff, "bias_diff")):
        _dev(x, n, torch.float32)
    _dev(bottom, "bottom", _bottom_dtype(desc)), _dev(weight, "weight", t)
    ws_bytes = 0 if workspace is None else workspace.numel()
    args = (ctypes.byref(desc), _ptr(top_diff), _ptr(top), _ptr(bottom), _ptr(weight),
            _ptr(bottom_diff), _ptr(weight_diff), _ptr(bias_diff), int(accumulate), int(flags),
            _ptr(workspace), ws_bytes, _stream(stream))
    if weight_stream is None:
        check(load().caffe_conv_backward(*args))
    else:
        check(load().caffe_conv_backward_ex(*args, _stream(weight_stream)))


def caffe_conv_backward_into(desc, top_diff, top, bottom, weight, weight_diff, bias_diff,
                             accumulate, flags, workspace, below, below_workspace, stream=None,
                             weight_stream=None):
    """caffe_conv_backward_into: the data gradient staged as the top gradient
    of the layer `below` (a ConvDesc) in its workspace."""
    t = _op_dtype(desc)
    for x, n in ((top_diff, "top_diff"), (top, "top"), (weight_diff, "weight_diff"),
                 (bias_diff, "bias_diff")):
        _dev(x, n, torch.float32)
    _dev(bottom, "bottom", _bottom_dtype(desc)), _dev(weight, "weight", t)
    ws_bytes = 0 if workspace is None else workspace.numel()
    bws_bytes = 0 if below_workspace is None else below_workspace.numel()
    check(load().caffe_conv_backward_into(
        ctypes.byref(desc), _ptr(top_diff), _ptr(top), _ptr(bottom), _ptr(weight),
        _ptr(weight_diff), _ptr(bias_diff), int(accumulate), int(flags), _ptr(workspace),
        ws_bytes, ctypes.byref(below), _ptr(below_workspace), bws_bytes, _stream(stream),
        _stream(weight_stream if weight_stream is not None else stream)))


def conv_stage_below_supported(desc, below):
    """Whether caffe_conv_backward_into can stage desc's data gradient for below."""
    return bool(load().caffe_conv_stage_below_supported(ctypes.byref(desc), ctypes.byref(below)))


def caffe_conv_backward_data(desc, top_diff, top, weight, bottom_diff, workspace=None, stream=None):
    _dev(top_diff, "top_diff", torch.float32), _dev(top, "top", torch.float32)
    _dev(weight, "weight", _op_dtype(desc)), _dev(bottom_diff, "bottom_diff", torch.float32)
    ws_bytes = 0 if workspace is None else workspace.numel()
    check(load().caffe_conv_backward_data(ctypes.byref(desc), _ptr(top_diff), _ptr(top),
                                          _ptr(weight), _ptr(bottom_diff), _ptr(workspace),
                                          ws_bytes, _stream(stream)))


def caffe_conv_backward_weights(desc, top_diff, top, bottom, weight_diff, bias_diff, accumulate=0,
                                workspace=None, stream=None):
    _dev(top_diff, "top_diff", torch.float32), _dev(top, "top", torch.float32)
    _dev(bottom, "bottom", _bottom_dtype(desc)), _dev(weight_diff, "weight_diff", torch.float32)
    _dev(bias_diff, "bias_diff", torch.float32)
    ws_bytes = 0 if workspace is None else workspace.numel()
    check(load().caffe_conv_backward_weights(ctypes.byref(desc), _ptr(top_diff), _ptr(top),
                                             _ptr(bottom), _ptr(weight_diff), _ptr(bias_diff),
                                             int(accumulate), _ptr(workspace), ws_bytes,
                                             _stream(stream)))


# ------------------------------------------------------ allocating helpers
def _dtype_of(x, w):
    """The descriptor dtype for a bottom x and weight w: bf16 weights with a
    float bottom take CAFFE_BF16_F32_BOTTOM (the library rounds the bottom)."""
    if w.dtype == torch.bfloat16:
        return CAFFE_BF16 if x.dtype == torch.bfloat16 else CAFFE_BF16_F32_BOTTOM
    return CAFFE_F32


def conv_forward(x, w, b=None, stride=1, pad=0, group=1, relu=False, out=None, ws=None):
    dtype = _dtype_of(x, w)
    d = conv_desc(x.shape, w.shape, stride, pad, group, relu, dtype)
    Ho, Wo = conv_out_shape(d)
    if out is None:
        out = torch.empty((d.N, d.K, Ho, Wo), dtype=torch.float32, device=x.device)
    need = conv_workspace_size(d, PASS_FORWARD)
    buf = (ws or Workspace(x.device)).get(need)
    caffe_conv_forward(d, x, w, b, out, buf)
    return out


def conv_backward(x, w, top_diff, top=None, stride=1, pad=0, group=1, relu=False,
                  need=("dx", "dw", "db"), accumulate=0, outs=None, ws=None, flags=0):
    """Returns (dx, dw, db), None where not requested."""
    dtype = _dtype_of(x, w)
    d = conv_desc(x.shape, w.shape, stride, pad, group, relu, dtype)
    dev = top_diff.device
    if outs is None:
        dx = torch.empty(x.shape, dtype=torch.float32, device=dev) if "dx" in need else None
        dw = torch.empty(w.shape, dtype=torch.float32, device=dev) if "dw" in need else None
        db = torch.empty((w.shape[0],), dtype=torch.float32, device=dev) if "db" in need else None
    else:
        dx, dw, db = outs
    buf = (ws or Workspace(dev)).get(conv_workspace_size(d, PASS_BACKWARD))
    need_x = dw is not None or (flags & BACKWARD_MASK_BOTTOM_DIFF)
    caffe_conv_backward(d, top_diff, top, x if need_x else None, w if dx is not None else None,
                        dx, dw, db, accumulate, flags, buf)
    return dx, dw, db


def conv_backward_data(x_shape, w, top_diff, top=None, stride=1, pad=0, group=1, relu=False,
                       ws=None):
    dtype = CAFFE_BF16 if w.dtype == torch.bfloat16 else CAFFE_F32
    d = conv_desc(x_shape, w.shape, stride, pad, group, relu, dtype)
    dx = torch.empty(tuple(x_shape), dtype=torch.float32, device=top_diff.device)
    buf = (ws or Workspace(top_diff.device)).get(conv_workspace_size(d, PASS_BACKWARD_DATA))
    caffe_conv_backward_data(d, top_diff, top, w, dx, buf)
    return dx


def conv_backward_weights(x, w_shape, top_diff, top=None, stride=1, pad=0, group=1, relu=False,
                          with_bias=True, accumulate=0, ws=None):
    dtype = CAFFE_BF16 if x.dtype == torch.bfloat16 else CAFFE_F32
    d = conv_desc(x.shape, w_shape, stride, pad, group, relu, dtype)
    dw = torch.empty(tuple(w_shape), dtype=torch.float32, device=x.device)
    db = torch.empty((w_shape[0],), dtype=torch.float32, device=x.device) if with_bias else None
    buf = (ws or Workspace(x.device)).get(conv_workspace_size(d, PASS_BACKWARD_WEIGHTS))
    caffe_conv_backward_weights(d, top_diff, top, x, dw, db, accumulate, buf)
    return dw, db


def pool_desc(x_shape, kernel, stride, pad=0):
    N, C, H, W = (int(v) for v in x_shape)
    kh, kw = _pair(kernel)
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    return PoolDesc(N, C, H, W, kh, kw, sh, sw, ph, pw)


def pool_out_shape(desc):
    Ho, Wo = ctypes.c_int32(), ctypes.c_int32()
    check(load().caffe_pool_out_shape(ctypes.byref(desc), ctypes.byref(Ho), ctypes.byref(Wo)))
    return Ho.value, Wo.value


def maxpool_forward(x, kernel, stride, pad=0, out=None, mask=None, with_mask=True, flags=0,
                    stream=None):
    _dev(x, "bottom", torch.float32)
    d = pool_desc(x.shape, kernel, stride, pad)
    Ho, Wo = pool_out_shape(d)
    if out is None:
        out = torch.empty((d.N, d.C, Ho, Wo), dtype=torch.float32, device=x.device)
    if mask is None and with_mask:
        mask = torch.empty((d.N, d.C, Ho, Wo), dtype=torch.int32, device=x.device)
    _dev(out, "top", torch.float32), _dev(mask, "mask", torch.int32)
    check(load().caffe_maxpool_forward(ctypes.byref(d), _ptr(x), _ptr(out), _ptr(mask), int(flags),
                                       _stream(stream)))
    return out, mask


def maxpool_backward(x_shape, top_diff, mask, kernel, stride, pad=0, out=None, stream=None):
    _dev(top_diff, "top_diff", torch.float32), _dev(mask, "mask", torch.int32)
    d = pool_desc(x_shape, kernel, stride, pad)
    if out is None:
        out = torch.empty(tuple(x_shape), dtype=torch.float32, device=top_diff.device)
    _dev(out, "bottom_diff", torch.float32)
    check(load().caffe_maxpool_backward(ctypes.byref(d), _ptr(top_diff), _ptr(mask), _ptr(out),
                                        _stream(stream)))
    return out


def lrn_desc(x_shape, size=5, alpha=1e-4, beta=0.75, k=1.0):
    N, C, H, W = (int(v) for v in x_shape)
    return LrnDesc(N, C, H, W, int(size), float(alpha), float(beta), float(k))


def lrn_forward(x, size=5, alpha=1e-4, beta=0.75, k=1.0, out=None, stream=None):
    _dev(x, "bottom", torch.float32)
    d = lrn_desc(x.shape, size, alpha, beta, k)
    if out is None:
        out = torch.empty_like(x)
    _dev(out, "top", torch.float32)
    check(load().caffe_lrn_forward(ctypes.byref(d), _ptr(x), _ptr(out), _stream(stream)))
    return out


def lrn_backward(x, y, top_diff, size=5, alpha=1e-4, beta=0.75, k=1.0, out=None, stream=None):
    for t, n in ((x, "bottom"), (y, "top"), (top_diff, "top_diff")):
        _dev(t, n, torch.float32)
    d = lrn_desc(x.shape, size, alpha, beta, k)
    if out is None:
        out = torch.empty_like(x)
    _dev(out, "bottom_diff", torch.float32)
    check(load().caffe_lrn_backward(ctypes.byref(d), _ptr(x), _ptr(y), _ptr(top_diff), _ptr(out),
                                    _stream(stream)))
    return out


def _pool_lrn_descs(x_shape, kernel, stride, pad, size, alpha, beta, k):
    pd = pool_desc(x_shape, kernel, stride, pad)
    Ho, Wo = pool_out_shape(pd)
    ld = lrn_desc((pd.N, pd.C, Ho, Wo), size, alpha, beta, k)
    return pd, ld, (pd.N, pd.C, Ho, Wo)


def pool_lrn_supported(x_shape, kernel, stride, pad=0, size=5, alpha=1e-4, beta=0.75, k=1.0):
    """Whether the fused max-pool + LRN kernels take this geometry (no launch)."""
    shape = (0,) + tuple(x_shape[1:])
    pd, ld, _ = _pool_lrn_descs(shape, kernel, stride, pad, size, alpha, beta, k)
    st = load().caffe_pool_lrn_forward(ctypes.byref(pd), ctypes.byref(ld), None, None, None, None,
                                       0, None)
    if st == CAFFE_ERR_UNSUPPORTED:
        return False
    check(st)
    return True


def pool_lrn_forward(x, kernel, stride, pad=0, size=5, alpha=1e-4, beta=0.75, k=1.0,
                     pooled=None, mask=None, out=None, flags=0, stream=None, stage_for=None):
    """Max-pool then LRN in one pass; returns (pooled, mask, out).  With
    stage_for=(conv desc, its forward workspace), caffe_pool_lrn_forward_into:
    the output is also staged as that convolution's bf16 bottom."""
    _dev(x, "bottom", torch.float32)
    pd, ld, shape = _pool_lrn_descs(x.shape, kernel, stride, pad, size, alpha, beta, k)
    mdt = torch.uint8 if flags & POOL_MASK_OFFSETS else torch.int32
    pooled = torch.empty(shape, dtype=torch.float32, device=x.device) if pooled is None else pooled
    mask = torch.empty(shape, dtype=mdt, device=x.device) if mask is None else mask
    out = torch.empty(shape, dtype=torch.float32, device=x.device) if out is None else out
    for t, n in ((pooled, "pooled"), (out, "top")):
        _dev(t, n, torch.float32)
    _dev(mask, "mask", mdt)
    args = (ctypes.byref(pd), ctypes.byref(ld), _ptr(x), _ptr(pooled), _ptr(mask), _ptr(out),
            int(flags))
    if stage_for is None:
        check(load().caffe_pool_lrn_forward(*args, _stream(stream)))
    else:
        nd, nws = stage_for
        check(load().caffe_pool_lrn_forward_into(*args, ctypes.byref(nd), _ptr(nws),
                                                 0 if nws is None else nws.numel(),
                                                 _stream(stream)))
    return pooled, mask, out


def pool_lrn_stage_supported(x_shape, kernel, stride, pad, size, alpha, beta, k, next_desc):
    """Whether pool_lrn_forward can stage its output for the convolution next_desc."""
    pd, ld, _ = _pool_lrn_descs(x_shape, kernel, stride, pad, size, alpha, beta, k)
    return bool(load().caffe_pool_lrn_stage_supported(ctypes.byref(pd), ctypes.byref(ld),
                                                      ctypes.byref(next_desc)))


def lrn_pool_backward(x_shape, pooled, top, top_diff, mask, kernel, stride, pad=0, size=5,
                      alpha=1e-4, beta=0.75, k=1.0, out=None, stream=None, flags=0):
    """The backward of pool_lrn_forward in one pass; returns bottom_diff.  With
    flags (BACKWARD_POOL_MASK_OFFSETS: a byte mask) caffe_lrn_pool_backward_ex."""
    pd, ld, _ = _pool_lrn_descs(x_shape, kernel, stride, pad, size, alpha, beta, k)
    for t, n in ((pooled, "pooled"), (top, "top"), (top_diff, "top_diff")):
        _dev(t, n, torch.float32)
    _dev(mask, "mask", torch.uint8 if flags & BACKWARD_POOL_MASK_OFFSETS else torch.int32)
    if out is None:
        out = torch.empty(tuple(x_shape), dtype=torch.float32, device=top_diff.device)
    _dev(out, "bottom_diff", torch.float32)
    args = (ctypes.byref(pd), ctypes.byref(ld), _ptr(pooled), _ptr(top), _ptr(top_diff),
            _ptr(mask), _ptr(out))
    if flags:
        check(load().caffe_lrn_pool_backward_ex(*args, int(flags), _stream(stream)))
    else:
        check(load().caffe_lrn_pool_backward(*args, _stream(stream)))
    return out


def caffe_conv_backward_pool_lrn(desc, pool, lrn, pooled, lrn_top, lrn_top_diff, pool_mask, top,
                                 bottom, weight, bottom_diff, weight_diff, bias_diff,
                                 accumulate=0, flags=0, workspace=None, stream=None,
                                 weight_stream=None):
    """caffe_conv_backward_pool_lrn: the layer's backward from the gradient
    of the LRN that follows its max-pool (pool, lrn: PoolDesc, LrnDesc); with
    weight_stream, caffe_conv_backward_pool_lrn_ex."""
    t = _op_dtype(desc)
    for x, n in ((pooled, "pooled"), (lrn_top, "lrn_top"), (lrn_top_diff, "lrn_top_diff"),
                 (top, "top"), (bottom_diff, "bottom_diff"), (weight_diff, "weight_diff"),
                 (bias_diff, "bias_diff")):
        _dev(x, n, torch.float32)
    _dev(pool_mask, "pool_mask",
         torch.uint8 if flags & BACKWARD_POOL_MASK_OFFSETS else torch.int32)
    _dev(bottom, "bottom", _bottom_dtype(desc)), _dev(weight, "weight", t)
    ws_bytes = 0 if workspace is None else workspace.numel()
    args = (ctypes.byref(desc), ctypes.byref(pool), ctypes.byref(lrn), _ptr(pooled),
            _ptr(lrn_top), _ptr(lrn_top_diff), _ptr(pool_mask), _ptr(top), _ptr(bottom),
            _ptr(weight), _ptr(bottom_diff), _ptr(weight_diff), _ptr(bias_diff), int(accumulate),
            int(flags), _ptr(workspace), ws_bytes, _stream(stream))
    if weight_stream is None:
        check(load().caffe_conv_backward_pool_lrn(*args))
    else:
        check(load().caffe_conv_backward_pool_lrn_ex(*args, _stream(weight_stream)))


def relu_backward(top, top_diff, out=None, stream=None):
    """bottom_diff = top_diff [top > 0] (the ReLU layer's backward)."""
    for t, n in ((top, "top"), (top_diff, "top_diff")):
        _dev(t, n, torch.float32)
    if top.shape != top_diff.shape:
        raise ValueError("top and top_diff differ in shape")
    if out is None:
        out = torch.empty_like(top_diff)
    _dev(out, "bottom_diff", torch.float32)
    check(load().caffe_relu_backward(_ptr(top), _ptr(top_diff), _ptr(out), top.numel(),
                                     _stream(stream)))
    return out


def cast_f32_to_bf16(x, out=None, stream=None):
    _dev(x, "in", torch.float32)
    if out is None:
        out = torch.empty(x.shape, dtype=torch.bfloat16, device=x.device)
    _dev(out, "out", torch.bfloat16)
    check(load().caffe_cast_f32_to_bf16(_ptr(x), _ptr(out), x.numel(), _stream(stream)))
    return out


# ------------------------------------------------------------------ solver
_POLICIES = {"fixed": CAFFE_LR_FIXED, "step": CAFFE_LR_STEP, "exp": CAFFE_LR_EXP,
             "inv": CAFFE_LR_INV}


def sgd_learning_rate(policy, base_lr, it, gamma=0.0, power=0.0, stepsize=1):
    """The schedule's learning rate at iteration `it` (host-only C call)."""
    sc = LrSchedule(_POLICIES[policy] if isinstance(policy, str) else int(policy),
                    float(base_lr), float(gamma), float(power), int(stepsize))
    out = ctypes.c_float()
    check(load().caffe_sgd_learning_rate(ctypes.byref(sc), int(it), ctypes.byref(out)))
    return out.value


def caffe_softmax_loss(scores, labels, N, K, loss_weight, loss, sample_loss, prob, scores_diff,
                       stream=None):
    check(load().caffe_softmax_loss(_ptr(scores), _ptr(labels), int(N), int(K),
                                    float(loss_weight), _ptr(loss), _ptr(sample_loss), _ptr(prob),
                                    _ptr(scores_diff), _stream(stream)))


def softmax_loss(scores, labels, loss_weight=1.0, prob=False, diff=True, out=None, stream=None):
    """scores: (N, K, ...) float32 with K classes per row, labels: (N,) int32.
    Returns (loss (1,), sample_loss (N,), prob or None, scores_diff or None);
    `out` may hold preallocated (loss, sample_loss, prob, diff) tensors."""
    _dev(scores, "scores", torch.float32)
    _dev(labels, "labels", torch.int32)
    N = scores.shape[0]
    K = scores.numel() // N if N else int(torch.tensor(scores.shape[1:]).prod())
    dev = scores.device
    if out is None:
        out = (torch.empty(1, dtype=torch.float32, device=dev),
               torch.empty(N, dtype=torch.float32, device=dev),
               torch.empty(scores.shape, dtype=torch.float32, device=dev) if prob else None,
               torch.empty(scores.shape, dtype=torch.float32, device=dev) if diff else None)
    caffe_softmax_loss(scores, labels, N, K, loss_weight, *out, stream=stream)
    return out


def sgd_update(w, g, v, lr, momentum=0.0, weight_decay=0.0, stream=None):
    """In place: v <- momentum v + lr (g + weight_decay w); w <- w - v.  `lr`
    is a number, or a one-element float32 device tensor read when the kernel
    runs (for graph capture)."""
    for t, n in ((w, "w"), (g, "g"), (v, "v")):
        _dev(t, n, torch.float32)
    if not (w.numel() == g.numel() == v.numel()):
        raise ValueError("w, g and v must have the same number of elements")
    if isinstance(lr, torch.Tensor):
        _dev(lr, "lr", torch.float32)
        check(load().caffe_sgd_update_device_lr(_ptr(w), _ptr(g), _ptr(v), w.numel(), _ptr(lr),
                                                float(momentum), float(weight_decay),
                                                _stream(stream)))
        return
    check(load().caffe_sgd_update(_ptr(w), _ptr(g), _ptr(v), w.numel(), float(lr),
                                  float(momentum), float(weight_decay), _stream(stream)))
