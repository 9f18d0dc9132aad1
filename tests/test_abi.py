"""The C ABI on the CPU: the library loads, exports every symbol the public
headers declare, and turns every invalid argument into its status code
before any GPU work (so none of these calls needs a GPU)."""
import ctypes
import glob
import os
import re

import pytest

import paper_1408_5093_amd as cc
from paper_1408_5093_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(caffe_[a-z0-9_]+)\s*\(", src))
    return names


def test_library_exports_every_declared_symbol():
    lib = cc.load()
    declared = _declared()
    assert declared, "no declarations found"
    assert declared == set(_lib.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name
    assert lib.caffe_version() >= 100


def test_status_strings():
    lib = cc.load()
    for code, name in [(0, b"CAFFE_OK"), (-1, b"CAFFE_ERR_INVALID_ARG"), (-2, b"CAFFE_ERR_ALIGN"),
                       (-3, b"CAFFE_ERR_WORKSPACE"), (-4, b"CAFFE_ERR_UNSUPPORTED"),
                       (-5, b"CAFFE_ERR_HIP")]:
        assert lib.caffe_status_string(code) == name
        assert lib.caffe_conv_status_string(code) == name
    assert lib.caffe_conv_status_string(-99) == b"CAFFE_ERR_UNKNOWN"


def test_workspace_bytes_matches_workspace_size():
    """caffe_conv_workspace_bytes returns what caffe_conv_workspace_size
    stores, and SIZE_MAX for an invalid descriptor or pass."""
    lib = cc.load()
    size_max = ctypes.c_size_t(-1).value
    for dt in (cc.CAFFE_F32, cc.CAFFE_BF16):
        d = cc.conv_desc((256, 96, 27, 27), (256, 48, 5, 5), 1, 2, 2, True, dt)
        for pass_ in range(4):
            assert lib.caffe_conv_workspace_bytes(ctypes.byref(d), pass_) == \
                cc.conv_workspace_size(d, pass_)
        assert lib.caffe_conv_workspace_bytes(ctypes.byref(d), 9) == size_max
    bad = _desc(group=3)
    assert lib.caffe_conv_workspace_bytes(ctypes.byref(bad), 0) == size_max
    assert lib.caffe_conv_workspace_bytes(None, 0) == size_max
    assert lib.caffe_last_error() != b""


def test_tuning_overrides_need_the_switch(monkeypatch):
    """A CAFFE_* tuning variable changes nothing unless
    CAFFE_PROFILE_OVERRIDES=1: the quad-order weight gradient's column table
    (part of conv2's weight-gradient workspace) is planned either way, and
    only the switch lets CAFFE_CONV_WGRAD_QUAD=0 drop it."""
    d = cc.conv_desc((256, 96, 27, 27), (256, 48, 5, 5), 1, 2, 2, True)
    default = cc.conv_workspace_size(d, cc.PASS_BACKWARD_WEIGHTS)
    monkeypatch.delenv("CAFFE_PROFILE_OVERRIDES", raising=False)
    monkeypatch.setenv("CAFFE_CONV_WGRAD_QUAD", "0")
    assert cc.conv_workspace_size(d, cc.PASS_BACKWARD_WEIGHTS) == default
    monkeypatch.setenv("CAFFE_PROFILE_OVERRIDES", "1")
    assert cc.conv_workspace_size(d, cc.PASS_BACKWARD_WEIGHTS) < default


@pytest.mark.parametrize("x,w,s,p,g,out", [
    ((256, 3, 227, 227), (96, 3, 11, 11), 4, 0, 1, (55, 55)),
    ((256, 96, 27, 27), (256, 48, 5, 5), 1, 2, 2, (27, 27)),
    ((256, 256, 13, 13), (384, 256, 3, 3), 1, 1, 1, (13, 13)),
    ((256, 384, 13, 13), (384, 192, 3, 3), 1, 1, 2, (13, 13)),
    ((256, 384, 13, 13), (256, 192, 3, 3), 1, 1, 2, (13, 13)),
    ((64, 1, 28, 28), (20, 1, 5, 5), 1, 0, 1, (24, 24)),
    ((64, 20, 12, 12), (50, 20, 5, 5), 1, 0, 1, (8, 8)),
    ((2, 3, 7, 9), (4, 3, 3, 2), (2, 3), (1, 0), 1, (4, 3)),
])
def test_out_shape(x, w, s, p, g, out):
    assert cc.conv_out_shape(cc.conv_desc(x, w, s, p, g)) == out


def _status(fn, *args):
    return fn(*args)


def _desc(**kw):
    d = cc.conv_desc((2, 4, 9, 9), (6, 2, 3, 3), 1, 1, 2, True)
    for k, v in kw.items():
        setattr(d, k, v)
    return d


@pytest.mark.parametrize("field,value,code", [
    ("C", 0, -1), ("H", -1, -1), ("K", 0, -1), ("N", -1, -1), ("kernel_h", 0, -1),
    ("stride_w", 0, -1), ("pad_h", -1, -1), ("group", 0, -1), ("group", 3, -1),
    ("K", 7, -1), ("relu", 2, -1), ("dtype", 7, -4), ("dtype", 3, -4), ("kernel_h", 12, -1),
    ("H", 20000, -4), ("pad_w", 17000, -4),
])
def test_invalid_descriptor(field, value, code):
    lib = cc.load()
    d = _desc(**{field: value})
    Ho, Wo = ctypes.c_int32(), ctypes.c_int32()
    assert lib.caffe_conv_out_shape(ctypes.byref(d), ctypes.byref(Ho), ctypes.byref(Wo)) == code
    n = ctypes.c_size_t()
    assert lib.caffe_conv_workspace_size(ctypes.byref(d), 3, ctypes.byref(n)) == code
    P = ctypes.c_void_p
    assert lib.caffe_conv_forward(ctypes.byref(d), P(0x1000), P(0x2000), None, P(0x3000), None, 0,
                                  None) == code
    assert lib.caffe_last_error() != b""


def test_float_bottom_bf16_dtype_plans_like_bf16():
    """CAFFE_BF16_F32_BOTTOM takes a float bottom but plans the bf16 path:
    the same workspace sizes as CAFFE_BF16 for every pass."""
    for x, w, s, p, g in [((256, 3, 227, 227), (96, 3, 11, 11), 4, 0, 1),
                          ((8, 96, 27, 27), (256, 48, 5, 5), 1, 2, 2)]:
        d1 = cc.conv_desc(x, w, s, p, g, True, cc.CAFFE_BF16)
        d2 = cc.conv_desc(x, w, s, p, g, True, cc.CAFFE_BF16_F32_BOTTOM)
        for pas in range(5):
            assert cc.conv_workspace_size(d1, pas) == cc.conv_workspace_size(d2, pas)


def test_null_desc_and_outputs():
    lib = cc.load()
    Ho = ctypes.c_int32()
    assert lib.caffe_conv_out_shape(None, ctypes.byref(Ho), ctypes.byref(Ho)) == -1
    d = _desc()
    assert lib.caffe_conv_out_shape(ctypes.byref(d), None, None) == -1
    assert lib.caffe_conv_workspace_size(ctypes.byref(d), 9, ctypes.byref(ctypes.c_size_t())) == -1


def test_tensor_size_limit():
    lib = cc.load()
    d = cc.conv_desc((4096, 256, 256, 256), (8, 256, 3, 3))  # 2^36 bytes of input
    n = ctypes.c_size_t()
    assert lib.caffe_conv_workspace_size(ctypes.byref(d), 0, ctypes.byref(n)) == -4


def test_workspace_sizes():
    d = cc.conv_desc((256, 3, 227, 227), (96, 3, 11, 11), 4, 0, 1, True)
    # the forward packs the weights into the kernel's layout
    assert cc.conv_workspace_size(d, cc.PASS_FORWARD) >= 96 * 3 * 11 * 11 * 4
    d2 = cc.conv_desc((256, 96, 27, 27), (256, 48, 5, 5), 1, 2, 2, True)
    assert cc.conv_workspace_size(d2, cc.PASS_FORWARD) >= 256 * 48 * 25 * 4  # packed weights
    for desc, top_hw in ((d, 55 * 55), (d2, 27 * 27)):
        data = cc.conv_workspace_size(desc, cc.PASS_BACKWARD_DATA)
        wts = cc.conv_workspace_size(desc, cc.PASS_BACKWARD_WEIGHTS)
        both = cc.conv_workspace_size(desc, cc.PASS_BACKWARD)
        assert both >= max(data, wts)
        for v in (data, wts, both):
            assert v % 256 == 0
        top_bytes = desc.N * desc.K * top_hw * 4
        assert data >= top_bytes  # room for the masked top gradient (relu)
        desc.relu = 0
        assert cc.conv_workspace_size(desc, cc.PASS_BACKWARD_DATA) < top_bytes
        desc.relu = 1

def test_workspace_sizes_bf16():
    # bf16 operands are staged channel-contiguous on a zero-bordered grid next
    # to the packed weights (rows padded to 64).  A single group of 3 channels
    # with an even horizontal stride is padded to 4 channels, two taps per
    # 16-byte chunk: 5 taps per kernel row round up to 6, the staged width to
    # 64 (the last tap pair reads one column past the image)
    d1 = cc.conv_desc((8, 3, 63, 63), (16, 3, 5, 5), 2, 0, 1, True, cc.CAFFE_BF16)
    assert cc.conv_workspace_size(d1, cc.PASS_FORWARD) >= 8 * 63 * 64 * 4 * 2 + 16 * 128 * 2
    # conv1 (stride 4) is staged space-to-depth: 4 x 4 pixel blocks of its 3
    # channels become 48 channels of a 57 x 57 grid, its 11 x 11 kernel 3 x 3
    # taps of them (432 reduction elements, rows padded to 448)
    d = cc.conv_desc((256, 3, 227, 227), (96, 3, 11, 11), 4, 0, 1, True, cc.CAFFE_BF16)
    xh = 256 * 57 * 57 * 48 * 2
    assert cc.conv_workspace_size(d, cc.PASS_FORWARD) >= xh + 96 * 448 * 2
    assert cc.conv_workspace_size(d, cc.PASS_FORWARD) < 256 * 227 * 228 * 4 * 2
    dh = 256 * 55 * 55 * 96 * 2
    both = cc.conv_workspace_size(d, cc.PASS_BACKWARD)
    assert both >= dh + xh
    assert both >= cc.conv_workspace_size(d, cc.PASS_BACKWARD_DATA)
    for p in range(4):
        assert cc.conv_workspace_size(d, p) % 256 == 0
    d2 = cc.conv_desc((2, 20, 9, 9), (8, 5, 3, 3), 1, 1, 4, False, cc.CAFFE_BF16)
    assert cc.conv_workspace_size(d2, cc.PASS_FORWARD) >= 2 * 81 * 4 * 8 * 2


def test_workspace_sizes_split_data_gradient():
    # one image with a long reduction: the data gradient's split partials
    # make its pass larger than the weight pass; PASS_BACKWARD covers both
    d = cc.conv_desc((1, 64, 6, 6), (64, 64, 5, 5), 1, 2, 1, True)
    data = cc.conv_workspace_size(d, cc.PASS_BACKWARD_DATA)
    wts = cc.conv_workspace_size(d, cc.PASS_BACKWARD_WEIGHTS)
    both = cc.conv_workspace_size(d, cc.PASS_BACKWARD)
    assert both == max(data, wts)
    assert cc.conv_workspace_size(d, cc.PASS_FORWARD) >= 64 * 64 * 25 * 4


def test_workspace_sizes_inner_product():
    # a 1x1 convolution of a 1x1 image (one group, fp32) runs as dense GEMMs:
    # the forward holds split-K partials (and X^T, W^T when C % 4 != 0), the
    # backward D and D^T next to the partials
    N, C, K = 256, 9216, 4096
    d = cc.conv_desc((N, C, 1, 1), (K, C, 1, 1), 1, 0, 1, True)
    assert cc.conv_workspace_size(d, cc.PASS_FORWARD) >= N * K * 4
    d3 = cc.conv_desc((N, C - 1, 1, 1), (K, C - 1, 1, 1), 1, 0, 1, True)
    assert cc.conv_workspace_size(d3, cc.PASS_FORWARD) >= (N * (C - 1) + K * (C - 1) + N * K) * 4
    both = cc.conv_workspace_size(d, cc.PASS_BACKWARD)
    assert both >= (2 * N * K + max(N * C, K * C)) * 4
    for p in range(4):
        assert cc.conv_workspace_size(d, p) % 256 == 0
    # an empty batch plans (no tiles) without failing
    d0 = cc.conv_desc((0, C, 1, 1), (K, C, 1, 1), 1, 0, 1, True)
    for p in range(4):
        assert cc.conv_workspace_size(d0, p) >= 0
    # partials of 2^31 bytes or more are refused
    with pytest.raises(cc.CaffeError):
        cc.conv_workspace_size(cc.conv_desc((1, 1 << 20, 1, 1), (1 << 12, 1 << 20, 1, 1)),
                               cc.PASS_BACKWARD)


def test_pointer_checks_before_any_launch():
    lib = cc.load()
    P = ctypes.c_void_p
    d = _desc()
    ws = cc.conv_workspace_size(d, cc.PASS_BACKWARD)
    fwd = lambda *a: lib.caffe_conv_forward(ctypes.byref(d), *a)
    assert fwd(None, P(0x2000), None, P(0x3000), None, 0, None) == -1          # bottom NULL
    assert fwd(P(0x1000), None, None, P(0x3000), None, 0, None) == -1          # weight NULL
    assert fwd(P(0x1004), P(0x2000), None, P(0x3000), None, 0, None) == -2     # misaligned
    assert fwd(P(0x1000), P(0x2000), P(0x4008), P(0x3000), None, 0, None) == -2  # bias
    bwd = lambda *a: lib.caffe_conv_backward(ctypes.byref(d), *a)
    # relu needs top (unless the top gradient comes masked)
    assert bwd(P(0x1000), None, P(0x2000), P(0x3000), P(0x4000), P(0x5000), P(0x6000), 0, 0,
               P(0x100000), ws, None) == -1
    # workspace too small / NULL / misaligned
    assert bwd(P(0x1000), P(0x1800), P(0x2000), P(0x3000), P(0x4000), P(0x5000), P(0x6000), 0, 0,
               P(0x100000), ws - 1, None) == -3
    assert bwd(P(0x1000), P(0x1800), P(0x2000), P(0x3000), P(0x4000), P(0x5000), P(0x6000), 0, 0,
               None, ws, None) == -1
    assert bwd(P(0x1000), P(0x1800), P(0x2000), P(0x3000), P(0x4000), P(0x5000), P(0x6000), 0, 0,
               P(0x100080), ws, None) == -2
    # accumulate flag, unknown backward flags
    assert bwd(P(0x1000), P(0x1800), P(0x2000), P(0x3000), P(0x4000), P(0x5000), P(0x6000), 2, 0,
               P(0x100000), ws, None) == -1
    assert bwd(P(0x1000), P(0x1800), P(0x2000), P(0x3000), P(0x4000), P(0x5000), P(0x6000), 0, 32,
               P(0x100000), ws, None) == -1
    # the staged top gradient is a bf16 mode's
    assert bwd(P(0x1000), P(0x1800), P(0x2000), P(0x3000), P(0x4000), P(0x5000), P(0x6000), 0,
               16, P(0x100000), ws, None) == -1
    # weight gradient needs bottom; data gradient needs weight; a masked
    # bottom gradient needs bottom
    assert bwd(P(0x1000), P(0x1800), None, P(0x3000), None, P(0x5000), None, 0, 0,
               P(0x100000), ws, None) == -1
    assert bwd(P(0x1000), P(0x1800), P(0x2000), None, P(0x4000), None, None, 0, 0,
               P(0x100000), ws, None) == -1
    assert bwd(P(0x1000), P(0x1800), None, P(0x3000), P(0x4000), None, None, 0, 2,
               P(0x100000), ws, None) == -1
    # forward flags: unknown ones, and a staged bottom is a bf16 mode's
    fx = lambda fl: lib.caffe_conv_forward_ex(ctypes.byref(d), P(0x1000), P(0x2000), None,
                                              P(0x3000), P(0x100000), ws, fl, None)
    assert fx(2) == -1 and fx(cc.FORWARD_BOTTOM_STAGED) == -1
    bd = lib.caffe_conv_backward_data
    assert bd(ctypes.byref(d), P(0x1000), P(0x1800), P(0x2000), None, P(0x100000), ws, None) == -1
    bw = lib.caffe_conv_backward_weights
    assert bw(ctypes.byref(d), P(0x1000), P(0x1800), P(0x2000), None, None, 0, P(0x100000), ws,
              None) == -1


def test_glue_validation():
    lib = cc.load()
    P = ctypes.c_void_p
    pd = cc.pool_desc((2, 3, 55, 55), 3, 2)
    assert cc.pool_out_shape(pd) == (27, 27)
    assert cc.pool_out_shape(cc.pool_desc((2, 3, 24, 24), 2, 2)) == (12, 12)
    bad = cc.pool_desc((2, 3, 55, 55), 3, 2, 3)  # pad >= kernel
    assert lib.caffe_maxpool_forward(ctypes.byref(bad), P(0x1000), P(0x2000), None, 0, None) == -1
    assert lib.caffe_maxpool_forward(ctypes.byref(pd), P(0x1004), P(0x2000), None, 0, None) == -2
    assert lib.caffe_maxpool_forward(ctypes.byref(pd), P(0x1000), P(0x2000), None, 2, None) == -1
    assert lib.caffe_maxpool_backward(ctypes.byref(pd), P(0x1000), None, P(0x2000), None) == -1
    ld = cc.lrn_desc((2, 3, 5, 5), 0)
    assert lib.caffe_lrn_forward(ctypes.byref(ld), P(0x1000), P(0x2000), None) == -1
    ld = cc.lrn_desc((2, 3, 5, 5), 5, k=0.0)
    assert lib.caffe_lrn_forward(ctypes.byref(ld), P(0x1000), P(0x2000), None) == -1
    # an LRN output staged for the next convolution: the shapes must meet,
    # the convolution must run on bf16 operands with whole 16-channel groups
    pd2 = cc.pool_desc((2, 96, 55, 55), 3, 2)
    ld2 = cc.lrn_desc((2, 96, 27, 27), 5)
    nxt = lambda C, dt: cc.conv_desc((2, C, 27, 27), (256, C // 2, 5, 5), 1, 2, 2, True, dt)
    into = lambda nd: lib.caffe_pool_lrn_forward_into(
        ctypes.byref(pd2), ctypes.byref(ld2), P(0x1000), P(0x2000), None, P(0x3000), 0,
        ctypes.byref(nd), P(0x100000), 1 << 30, None)
    # byte winner offsets need windows of at most 255 taps
    big = cc.pool_desc((2, 96, 40, 40), 16, 2)
    bigl = cc.lrn_desc((2, 96) + cc.pool_out_shape(big), 5)
    assert lib.caffe_pool_lrn_forward(ctypes.byref(big), ctypes.byref(bigl), P(0x1000), P(0x2000),
                                      P(0x4000), P(0x3000), cc.POOL_MASK_OFFSETS, None) in (-4,)
    assert lib.caffe_lrn_pool_backward_ex(ctypes.byref(pd2), ctypes.byref(ld2), P(0x1000),
                                          P(0x2000), P(0x3000), P(0x4000), P(0x5000), 1,
                                          None) == -1       # an unknown flag
    # the stage-only flag belongs to the staging call
    assert lib.caffe_pool_lrn_forward(ctypes.byref(pd2), ctypes.byref(ld2), P(0x1000), P(0x2000),
                                      None, P(0x3000), cc.POOL_LRN_STAGE_ONLY, None) == -1
    assert lib.caffe_pool_lrn_stage_supported(ctypes.byref(pd2), ctypes.byref(ld2),
                                              ctypes.byref(nxt(96, cc.CAFFE_BF16_F32_BOTTOM)))
    for nd, code in [(nxt(96, cc.CAFFE_F32), -4), (nxt(192, cc.CAFFE_BF16_F32_BOTTOM), -1)]:
        assert not lib.caffe_pool_lrn_stage_supported(ctypes.byref(pd2), ctypes.byref(ld2),
                                                      ctypes.byref(nd))
        assert into(nd) == code
    assert lib.caffe_cast_f32_to_bf16(P(0x1000), P(0x2000), -1, None) == -1
    assert lib.caffe_cast_f32_to_bf16(P(0x1002), P(0x2000), 5, None) == -2


def test_fastdiv_formula():
    # the host-side magic numbers for unsigned division used by the weight-
    # gradient kernel: q = (x * mul) >> (31 + ceil(log2 d)) for x < 2^31
    import random
    random.seed(3)
    for d in list(range(1, 2000)) + [3025, 3249, 169, 729, 12544, 1 << 20, (1 << 30) + 3]:
        l = (d - 1).bit_length()
        sh = 31 + l
        mul = ((1 << sh) + d - 1) // d
        assert mul < (1 << 32)
        for x in [0, d - 1, d, 2 ** 31 - 1] + [random.randrange(2 ** 31) for _ in range(50)]:
            assert (x * mul) >> sh == x // d


# ------------------------------------------------------------------ solver ABI
def test_learning_rate_schedules_match_oracle():
    import oracle
    cases = [("fixed", dict()), ("step", dict(gamma=0.1, stepsize=100)),
             ("exp", dict(gamma=0.999)), ("inv", dict(gamma=1e-4, power=0.75))]
    import numpy as np
    f32 = lambda v: float(np.float32(v))  # the schedule's parameters are stored as float32
    for policy, kw in cases:
        kw32 = {k: (f32(v) if k != "stepsize" else v) for k, v in kw.items()}
        for it in (0, 1, 99, 100, 101, 250, 5000, 10000):
            got = cc.sgd_learning_rate(policy, 0.01, it, **kw)
            ref = oracle.learning_rate(policy, f32(0.01), it, **kw32)
            assert abs(got - ref) <= 1e-7 * ref + 1e-30, (policy, it, got, ref)


def test_solver_argument_checks():
    lib = cc.load()
    P = ctypes.c_void_p
    sm = lambda *a: lib.caffe_softmax_loss(*a)
    ok = (P(0x1000), P(0x2000), 4, 10, 1.0, P(0x3000), P(0x4000), None, None, None)
    bad = list(ok)
    bad[3] = 0
    assert sm(*bad) == -1                                          # K = 0
    bad = list(ok)
    bad[2] = -1
    assert sm(*bad) == -1                                          # N < 0
    bad = list(ok)
    bad[5] = None
    assert sm(*bad) == -1                                          # loss NULL
    bad = list(ok)
    bad[0] = P(0x1004)
    assert sm(*bad) == -2                                          # misaligned scores
    bad = list(ok)
    bad[4] = float("nan")
    assert sm(*bad) == -1                                          # loss_weight NaN
    assert sm(P(0x1000), P(0x2000), 1 << 16, 1 << 14, 1.0, P(0x3000), P(0x4000), None, None,
              None) == -4                                          # 2^32 bytes of scores
    up = lambda *a: lib.caffe_sgd_update(*a)
    assert up(P(0x1000), P(0x2000), P(0x3000), -1, 0.1, 0.9, 0.0, None) == -1
    assert up(None, P(0x2000), P(0x3000), 8, 0.1, 0.9, 0.0, None) == -1
    assert up(P(0x1000), P(0x2000), P(0x3008), 8, 0.1, 0.9, 0.0, None) == -2
    assert up(P(0x1000), P(0x2000), P(0x3000), 8, float("inf"), 0.9, 0.0, None) == -1
    assert up(None, None, None, 0, 0.1, 0.9, 0.0, None) == 0       # nothing to do
    upd = lambda *a: lib.caffe_sgd_update_device_lr(*a)
    assert upd(P(0x1000), P(0x2000), P(0x3000), 8, None, 0.9, 0.0, None) == -1   # lr NULL
    assert upd(P(0x1000), P(0x2000), P(0x3000), 8, P(0x4002), 0.9, 0.0, None) == -2
    assert upd(P(0x1000), P(0x2000), P(0x3000), -1, P(0x4000), 0.9, 0.0, None) == -1
    with pytest.raises(cc.CaffeError):
        cc.sgd_learning_rate(7, 0.01, 0)                           # unknown policy
    with pytest.raises(cc.CaffeError):
        cc.sgd_learning_rate("step", 0.01, 5, gamma=0.1, stepsize=0)
    with pytest.raises(cc.CaffeError):
        cc.sgd_learning_rate("fixed", 0.01, -1)
    with pytest.raises(cc.CaffeError):
        cc.sgd_learning_rate("inv", 0.01, 2, gamma=-1.0, power=0.75)  # (1 - 2)^-0.75
