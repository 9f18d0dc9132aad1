"""GPU parity of the glue layers (max pooling, LRN) and the bf16 cast
against the CPU oracle / the round-to-nearest-even definition."""
import numpy as np
import pytest
import torch

import oracle
import paper_1408_5093_amd as cc
from paper_1408_5093_amd import workloads as wl
from helpers import TOL_F32, assert_close

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def _np(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


@pytest.mark.parametrize("shape,k,s,p", [
    ((2, 5, 55, 55), 3, 2, 0), ((3, 4, 24, 24), 2, 2, 0), ((1, 3, 13, 11), 3, 2, 1),
    ((2, 2, 9, 10), 3, 3, 2), ((1, 1, 5, 5), 5, 1, 0), ((2, 7, 27, 27), 3, 2, 0),
])
def test_maxpool(shape, k, s, p):
    print(f"maxpool {shape} k={k} s={s} p={p}", flush=True)
    rng = np.random.default_rng([3, *shape, k, s, p])
    x = rng.standard_normal(shape).astype(np.float32)
    y, mask = cc.maxpool_forward(_t(x), k, s, p)
    y_ref = oracle.maxpool_forward(x, k, s, p)
    np.testing.assert_array_equal(_np(y), y_ref.astype(np.float32))
    g = rng.standard_normal(y_ref.shape).astype(np.float32)
    dx = cc.maxpool_backward(x.shape, _t(g), mask, k, s, p)
    assert_close(_np(dx), oracle.maxpool_backward(x, g, k, s, p), TOL_F32, "maxpool backward")


def test_maxpool_ties_first_max():
    x = np.zeros((1, 1, 6, 6), np.float32)  # every window is a tie
    y, mask = cc.maxpool_forward(_t(x), 3, 2, 0)
    g = np.arange(1, 5, dtype=np.float32).reshape(1, 1, 2, 2)
    dx = cc.maxpool_backward(x.shape, _t(g), mask, 3, 2, 0)
    np.testing.assert_array_equal(_np(dx), oracle.maxpool_backward(x, g, 3, 2, 0))


@pytest.mark.parametrize("shape,size,alpha,beta,k", [
    ((2, 96, 27, 27), 5, 1e-4, 0.75, 1.0), ((2, 256, 13, 13), 5, 1e-4, 0.75, 1.0),
    ((1, 7, 5, 4), 5, 0.5, 0.75, 2.0), ((2, 3, 3, 3), 3, 1.0, 0.5, 1.0), ((1, 9, 2, 2), 4, 0.2, 0.6, 1.5),
])
def test_lrn(shape, size, alpha, beta, k):
    print(f"lrn {shape} size={size}", flush=True)
    rng = np.random.default_rng([4, *shape, size])
    x = (rng.standard_normal(shape) * 20).astype(np.float32)
    y = cc.lrn_forward(_t(x), size, alpha, beta, k)
    y_ref = oracle.lrn_forward(x, size, alpha, beta, k)
    assert_close(_np(y), y_ref, TOL_F32, "LRN forward")
    g = rng.standard_normal(shape).astype(np.float32)
    dx = cc.lrn_backward(_t(x), _t(y_ref), _t(g), size, alpha, beta, k)
    assert_close(_np(dx), oracle.lrn_backward(x, g, size, alpha, beta, k), TOL_F32,
                 "LRN backward")


def test_cast_bf16_round_to_nearest_even():
    rng = np.random.default_rng(8)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 100,
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.4e38, -3.4e38,
                                  1e-40, np.inf, -np.inf], np.float32)])
    b = cc.cast_f32_to_bf16(_t(x))
    torch.cuda.synchronize()
    got = b.view(torch.int16).cpu().numpy().view(np.uint16)
    np.testing.assert_array_equal(got, wl.to_bf16_bits(x))
    # torch's own float -> bfloat16 conversion also rounds to nearest even
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(got, ref)
    # eight values per thread and step, then the tail one by one
    for n in (1, 7, 8, 9, 23, 4096 + 5):
        bn = cc.cast_f32_to_bf16(_t(x[:n]))
        torch.cuda.synchronize()
        np.testing.assert_array_equal(bn.view(torch.int16).cpu().numpy().view(np.uint16),
                                      wl.to_bf16_bits(x[:n]))


def test_maxpool_relu_input_flag():
    """CAFFE_POOL_RELU_INPUT: same forward output; the backward pass also
    applies the backward of the ReLU that produced the input."""
    rng = np.random.default_rng(31)
    x = np.maximum(rng.standard_normal((2, 6, 27, 27)), 0).astype(np.float32)
    x[0, 0, :5, :5] = 0.0  # whole windows of zeros
    y, mask = cc.maxpool_forward(_t(x), 3, 2, 0, flags=cc.POOL_RELU_INPUT)
    np.testing.assert_array_equal(_np(y), oracle.maxpool_forward(x, 3, 2).astype(np.float32))
    m = _np(mask)
    assert np.all(m[_np(y) <= 0] == -1) and np.all(m[_np(y) > 0] >= 0)
    g = rng.standard_normal(m.shape).astype(np.float32)
    dx = cc.maxpool_backward(x.shape, _t(g), mask, 3, 2, 0)
    assert_close(_np(dx), oracle.maxpool_backward(x, g, 3, 2) * (x > 0), TOL_F32,
                 "pool backward with ReLU input")


# ------------------------------------------------ fused max-pool + LRN
FUSED = [
    # shape, pool k, s, p, LRN size, alpha, beta, k
    ((3, 96, 55, 55), 3, 2, 0, 5, 1e-4, 0.75, 1.0),    # CaffeNet pool1 + norm1 (3 strips)
    ((2, 256, 27, 27), 3, 2, 0, 5, 1e-4, 0.75, 1.0),   # pool2 + norm2
    ((2, 20, 17, 19), 3, 2, 0, 5, 0.5, 0.75, 2.0),     # a partial 16-channel chunk
    ((1, 5, 21, 23), 3, 2, 1, 3, 1.0, 0.5, 1.0),       # padded windows, LRN size 3
    ((2, 18, 24, 24), 2, 2, 0, 5, 0.3, 0.6, 1.5),      # 2x2/2
    ((1, 33, 80, 78), 3, 3, 2, 5, 0.4, 0.75, 1.0),     # any-window path, several strips
]


@pytest.mark.parametrize("shape,pk,ps,pp,size,alpha,beta,k", FUSED)
@pytest.mark.parametrize("relu_input", [False, True])
def test_pool_lrn_fused(shape, pk, ps, pp, size, alpha, beta, k, relu_input):
    print(f"fused pool+lrn {shape} pool {pk}/{ps}/{pp} lrn {size} relu_input={relu_input}",
          flush=True)
    rng = np.random.default_rng([5, *shape, pk, ps, pp, size, int(relu_input)])
    x = (rng.standard_normal(shape) * 20).astype(np.float32)
    if relu_input:
        x = np.maximum(x, 0)
    flags = cc.POOL_RELU_INPUT if relu_input else 0
    assert cc.pool_lrn_supported(shape, pk, ps, pp, size, alpha, beta, k)
    pooled, mask, y = cc.pool_lrn_forward(_t(x), pk, ps, pp, size, alpha, beta, k, flags=flags)
    p_ref = oracle.maxpool_forward(x, pk, ps, pp)
    np.testing.assert_array_equal(_np(pooled), p_ref.astype(np.float32))
    assert_close(_np(y), oracle.lrn_forward(_np(pooled), size, alpha, beta, k), TOL_F32,
                 "fused forward (LRN)")
    # the same values and winners as the two separate layers
    y2, mask2 = cc.maxpool_forward(_t(x), pk, ps, pp, flags=flags)
    np.testing.assert_array_equal(_np(mask), _np(mask2))
    z2 = cc.lrn_forward(y2, size, alpha, beta, k)
    assert_close(_np(y), _np(z2), 1e-6, "fused vs separate forward")
    g = rng.standard_normal(p_ref.shape).astype(np.float32)
    dx = cc.lrn_pool_backward(shape, pooled, y, _t(g), mask, pk, ps, pp, size, alpha, beta, k)
    dp_ref = oracle.lrn_backward(_np(pooled), g, size, alpha, beta, k)
    dx_ref = oracle.maxpool_backward(x, dp_ref, pk, ps, pp)
    if relu_input:
        dx_ref = dx_ref * (x > 0)
    assert_close(_np(dx), dx_ref, TOL_F32, "fused backward")
    dp2 = cc.lrn_backward(pooled, y, _t(g), size, alpha, beta, k)
    dx2 = cc.maxpool_backward(shape, dp2, mask, pk, ps, pp)
    assert_close(_np(dx), _np(dx2), 1e-6, "fused vs separate backward")


@pytest.mark.parametrize("shape,pk,ps,pp,size,alpha,beta,k",
                         [c for c in FUSED if c[1:3] == (3, 2)])
def test_pool_lrn_backward_empty_windows(shape, pk, ps, pp, size, alpha, beta, k):
    """The fused backward (3x3 / stride 2: four input positions per thread
    from one read of their covering windows) on a ReLU input where about half
    the windows hold no winner: against the separate LRN and pool backward
    passes and the oracle."""
    print(f"fused backward, empty windows {shape} pool {pk}/{ps}/{pp}", flush=True)
    rng = np.random.default_rng([6, *shape, pp])
    x = np.maximum(rng.standard_normal(shape) - 1.5, 0).astype(np.float32)
    pooled, mask, y = cc.pool_lrn_forward(_t(x), pk, ps, pp, size, alpha, beta, k,
                                          flags=cc.POOL_RELU_INPUT)
    assert (_np(mask) == -1).mean() > 0.2
    g = rng.standard_normal(tuple(y.shape)).astype(np.float32)
    dx = cc.lrn_pool_backward(shape, pooled, y, _t(g), mask, pk, ps, pp, size, alpha, beta, k)
    dp2 = cc.lrn_backward(pooled, y, _t(g), size, alpha, beta, k)
    dx2 = cc.maxpool_backward(shape, dp2, mask, pk, ps, pp)
    assert_close(_np(dx), _np(dx2), 1e-6, "fused vs separate backward")
    dp_ref = oracle.lrn_backward(_np(pooled), g, size, alpha, beta, k)
    dx_ref = oracle.maxpool_backward(x, dp_ref, pk, ps, pp) * (x > 0)
    assert_close(_np(dx), dx_ref, TOL_F32, "fused backward vs the oracle")


def test_pool_lrn_fused_unsupported_and_empty():
    # 3 staged pooled rows of 200 columns exceed 256 positions
    assert not cc.pool_lrn_supported((1, 4, 401, 401), 3, 2, 0, 5)
    with pytest.raises(cc.CaffeError):
        cc.pool_lrn_forward(torch.zeros((1, 4, 401, 401), device=DEV), 3, 2, 0, 5)
    assert not cc.pool_lrn_supported((1, 4, 55, 55), 3, 2, 0, 7)   # LRN size 7
    x = torch.zeros((0, 8, 9, 9), device=DEV)
    pooled, mask, y = cc.pool_lrn_forward(x, 3, 2, 0, 5)
    dx = cc.lrn_pool_backward(x.shape, pooled, y, torch.zeros_like(y), mask, 3, 2, 0, 5)
    torch.cuda.synchronize()
    assert dx.shape == x.shape


def test_relu_backward():
    """bottom_diff = top_diff [top > 0] (exact select; NaN top gives 0), in
    place too, and with a length that is not a multiple of 4."""
    rng = np.random.default_rng(31)
    for n in (1, 7, 4099, 100000):
        top = torch.from_numpy(rng.standard_normal(n).astype(np.float32)).to(DEV)
        top[0] = float("nan")
        g = torch.from_numpy(rng.standard_normal(n).astype(np.float32)).to(DEV)
        ref = torch.where(top > 0, g, torch.zeros_like(g))
        assert torch.equal(cc.relu_backward(top, g), ref)
        g2 = g.clone()
        cc.relu_backward(top, g2, out=g2)
        assert torch.equal(g2, ref)
