"""Pins for the convolution oracle (oracle/caffe_ref.c), all on the CPU.

The paper (Sec. 3.2) fixes only the roles of a layer's forward and backward
passes; it prints no formula and no numeric example.  Each test below pins the
oracle to something other than its own loops: hand-worked examples, closed
forms, special cases that reduce to a library routine (numpy matmul, torch's
float64 CPU convolution), invariants (linearity, adjointness) and finite
differences of the forward pass.
"""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

RNG = np.random.default_rng(20140818)


def _rand(*shape):
    return RNG.standard_normal(shape)


# ---------------------------------------------------------------- hand-worked
def test_worked_examples(golden_dir):
    cases = json.load(open(os.path.join(golden_dir, "conv_worked_examples.json")))["cases"]
    for c in cases:
        x, w, b = np.array(c["x"], float), np.array(c["w"], float), np.array(c["b"], float)
        y = oracle.conv_forward(x, w, b, c["stride"], c["pad"], c["group"], c["relu"])
        np.testing.assert_array_equal(y, np.array(c["y"], float), err_msg=c["name"])
        dx, dw, db = oracle.conv_backward(x, w, np.array(c["top_diff"], float), top=y,
                                          stride=c["stride"], pad=c["pad"], group=c["group"],
                                          relu=c["relu"])
        np.testing.assert_array_equal(dx, np.array(c["dx"], float), err_msg=c["name"])
        np.testing.assert_array_equal(dw, np.array(c["dw"], float), err_msg=c["name"])
        np.testing.assert_array_equal(db, np.array(c["db"], float), err_msg=c["name"])


# ------------------------------------------------------------ closed forms
def test_out_shape_closed_form():
    # floor((H + 2p - k)/s) + 1 on the CaffeNet / LeNet geometries
    assert oracle.conv_out_shape(227, 227, 11, 11, 4, 4, 0, 0) == (55, 55)
    assert oracle.conv_out_shape(27, 27, 5, 5, 1, 1, 2, 2) == (27, 27)
    assert oracle.conv_out_shape(13, 13, 3, 3, 1, 1, 1, 1) == (13, 13)
    assert oracle.conv_out_shape(28, 28, 5, 5, 1, 1, 0, 0) == (24, 24)
    assert oracle.conv_out_shape(12, 12, 5, 5, 1, 1, 0, 0) == (8, 8)
    assert oracle.conv_out_shape(7, 9, 3, 2, 2, 3, 1, 0) == (4, 3)
    with pytest.raises(ValueError):
        oracle.conv_out_shape(2, 2, 5, 5, 1, 1, 0, 0)


def test_identity_1x1_reproduces_input():
    x = _rand(2, 5, 6, 7)
    w = np.eye(5).reshape(5, 5, 1, 1)
    np.testing.assert_array_equal(oracle.conv_forward(x, w), x)
    # depthwise identity: group = C, one 1x1 tap per channel
    wd = np.ones((5, 1, 1, 1))
    np.testing.assert_array_equal(oracle.conv_forward(x, wd, group=5), x)


def test_delta_image_gives_rotated_filter():
    # cross-correlation: a unit impulse at (a,b) produces W rotated by 180 degrees
    kh, kw, H, W = 3, 4, 9, 10
    w = _rand(2, 1, kh, kw)
    x = np.zeros((1, 1, H, W))
    a, b = 4, 5
    x[0, 0, a, b] = 1.0
    y = oracle.conv_forward(x, w)
    for k in range(2):
        patch = y[0, k, a - kh + 1:a + 1, b - kw + 1:b + 1]
        np.testing.assert_array_equal(patch, w[k, 0, ::-1, ::-1])
        assert np.count_nonzero(y[0, k]) == np.count_nonzero(w[k])


def test_delta_top_diff_gives_filter_and_window():
    kh, kw, H, W = 3, 3, 8, 8
    x = _rand(1, 2, H, W)
    w = _rand(3, 2, kh, kw)
    g = np.zeros((1, 3, H - kh + 1, W - kw + 1))
    i, j, k = 2, 3, 1
    g[0, k, i, j] = 1.0
    dx, dw, db = oracle.conv_backward(x, w, g)
    expect_dx = np.zeros_like(x)
    expect_dx[0, :, i:i + kh, j:j + kw] = w[k]
    np.testing.assert_array_equal(dx, expect_dx)
    expect_dw = np.zeros_like(w)
    expect_dw[k] = x[0, :, i:i + kh, j:j + kw]
    np.testing.assert_array_equal(dw, expect_dw)
    np.testing.assert_array_equal(db, np.eye(3)[k])


# ------------------------------------------------------ library special cases
def test_1x1_conv_is_matmul():
    x = _rand(3, 6, 4, 5)
    w = _rand(7, 6, 1, 1)
    b = _rand(7)
    y = oracle.conv_forward(x, w, b)
    ref = np.einsum("kc,nchw->nkhw", w[:, :, 0, 0], x) + b[None, :, None, None]
    np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-13)
    g = _rand(3, 7, 4, 5)
    dx, dw, db = oracle.conv_backward(x, w, g)
    np.testing.assert_allclose(dx, np.einsum("kc,nkhw->nchw", w[:, :, 0, 0], g), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw[:, :, 0, 0], np.einsum("nkhw,nchw->kc", g, x), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, g.sum(axis=(0, 2, 3)), rtol=1e-12, atol=1e-12)


def test_full_size_kernel_is_inner_product():
    x = _rand(4, 3, 5, 6)
    w = _rand(8, 3, 5, 6)
    y = oracle.conv_forward(x, w)
    assert y.shape == (4, 8, 1, 1)
    np.testing.assert_allclose(y[:, :, 0, 0], x.reshape(4, -1) @ w.reshape(8, -1).T,
                               rtol=1e-12, atol=1e-12)


def test_inner_product_with_relu_is_masked_matmuls():
    # an inner-product layer (Sec. 3.2's fully connected layers) is the 1x1
    # convolution of a 1x1 image: y = relu(W x + b); with D = G [y > 0],
    # dx = D W, dW = D^T x, db = sum over the batch of D
    x = _rand(5, 9, 1, 1)
    w = _rand(4, 9, 1, 1)
    b = _rand(4)
    X, Wm = x[:, :, 0, 0], w[:, :, 0, 0]
    y = oracle.conv_forward(x, w, b, relu=True)
    np.testing.assert_allclose(y[:, :, 0, 0], np.maximum(X @ Wm.T + b, 0), rtol=1e-13, atol=1e-13)
    g = _rand(5, 4, 1, 1)
    dx, dw, db = oracle.conv_backward(x, w, g, top=y, relu=True)
    D = g[:, :, 0, 0] * (y[:, :, 0, 0] > 0)
    np.testing.assert_allclose(dx[:, :, 0, 0], D @ Wm, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw[:, :, 0, 0], D.T @ X, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, D.sum(axis=0), rtol=1e-12, atol=1e-12)


CASES = [
    # N, C, H, W, K, kh, kw, s, p, g
    (2, 3, 11, 9, 4, 3, 3, 1, 1, 1),
    (2, 4, 13, 13, 6, 5, 5, 1, 2, 2),
    (1, 3, 23, 23, 5, 11, 11, 4, 0, 1),
    (3, 6, 7, 8, 9, 3, 2, 2, 1, 3),
    (2, 1, 12, 12, 4, 5, 5, 1, 0, 1),
    (1, 4, 6, 5, 4, 2, 3, 3, 2, 4),
]


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("relu", [False, True])
def test_matches_torch_float64(case, relu):
    N, C, H, W, K, kh, kw, s, p, g = case
    x = torch.from_numpy(_rand(N, C, H, W))
    w = torch.from_numpy(_rand(K, C // g, kh, kw))
    b = torch.from_numpy(_rand(K))
    z = F.conv2d(x, w, b, stride=s, padding=p, groups=g)
    yref = torch.relu(z) if relu else z
    y = oracle.conv_forward(x.numpy(), w.numpy(), b.numpy(), s, p, g, relu)
    np.testing.assert_allclose(y, yref.numpy(), rtol=1e-12, atol=1e-12)

    gt = torch.from_numpy(_rand(*yref.shape))
    d = gt * (yref > 0) if relu else gt
    dx_ref = torch.nn.grad.conv2d_input(x.shape, w, d, stride=s, padding=p, groups=g)
    dw_ref = torch.nn.grad.conv2d_weight(x, w.shape, d, stride=s, padding=p, groups=g)
    dx, dw, db = oracle.conv_backward(x.numpy(), w.numpy(), gt.numpy(), top=y, stride=s, pad=p,
                                      group=g, relu=relu)
    np.testing.assert_allclose(dx, dx_ref.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dw, dw_ref.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(db, d.sum(dim=(0, 2, 3)).numpy(), rtol=1e-12, atol=1e-12)


def test_group_is_independent_convs():
    x = _rand(2, 6, 9, 9)
    w = _rand(4, 3, 3, 3)
    b = _rand(4)
    y = oracle.conv_forward(x, w, b, 1, 1, 2)
    y0 = oracle.conv_forward(x[:, :3], w[:2], b[:2], 1, 1, 1)
    y1 = oracle.conv_forward(x[:, 3:], w[2:], b[2:], 1, 1, 1)
    np.testing.assert_array_equal(y, np.concatenate([y0, y1], axis=1))
    g = _rand(*y.shape)
    dx, dw, db = oracle.conv_backward(x, w, g, stride=1, pad=1, group=2)
    a = oracle.conv_backward(x[:, :3], w[:2], g[:, :2], stride=1, pad=1)
    c = oracle.conv_backward(x[:, 3:], w[2:], g[:, 2:], stride=1, pad=1)
    np.testing.assert_array_equal(dx, np.concatenate([a[0], c[0]], axis=1))
    np.testing.assert_array_equal(dw, np.concatenate([a[1], c[1]], axis=0))
    np.testing.assert_array_equal(db, np.concatenate([a[2], c[2]]))


def test_stride_is_subsampled_stride1():
    x = _rand(2, 3, 17, 15)
    w = _rand(4, 3, 5, 3)
    y1 = oracle.conv_forward(x, w, stride=1)
    for s in (2, 3, 4):
        ys = oracle.conv_forward(x, w, stride=s)
        np.testing.assert_array_equal(ys, y1[:, :, ::s, ::s][:, :, :ys.shape[2], :ys.shape[3]])


def test_pad_is_explicit_zero_pad():
    x = _rand(2, 3, 7, 8)
    w = _rand(4, 3, 3, 5)
    for p in (1, 2, 3):
        xp = np.pad(x, ((0, 0), (0, 0), (p, p), (p, p)))
        np.testing.assert_allclose(oracle.conv_forward(x, w, pad=p), oracle.conv_forward(xp, w),
                                   rtol=0, atol=1e-14)
        g = _rand(*oracle.conv_forward(xp, w).shape)
        dx, dw, _ = oracle.conv_backward(x, w, g, pad=p)
        dxp, dwp, _ = oracle.conv_backward(xp, w, g)
        np.testing.assert_allclose(dx, dxp[:, :, p:-p, p:-p], rtol=0, atol=1e-13)
        np.testing.assert_allclose(dw, dwp, rtol=1e-13, atol=1e-13)


# -------------------------------------------------------------- invariants
def test_linearity_and_bias_shift():
    x1, x2 = _rand(2, 4, 9, 9), _rand(2, 4, 9, 9)
    w1, w2 = _rand(6, 2, 3, 3), _rand(6, 2, 3, 3)
    a, b = 1.7, -0.3
    f = lambda x, w: oracle.conv_forward(x, w, None, 2, 1, 2)
    np.testing.assert_allclose(f(a * x1 + b * x2, w1), a * f(x1, w1) + b * f(x2, w1), atol=1e-12)
    np.testing.assert_allclose(f(x1, a * w1 + b * w2), a * f(x1, w1) + b * f(x1, w2), atol=1e-12)
    bias = _rand(6)
    yb = oracle.conv_forward(x1, w1, bias, 2, 1, 2)
    np.testing.assert_allclose(yb - f(x1, w1), np.broadcast_to(bias[None, :, None, None], yb.shape),
                               atol=1e-13)


@pytest.mark.parametrize("case", CASES)
def test_adjoint_identities(case):
    # <F_W(X), R> = <X, dgrad(R)> and <F_X(W), R> = <W, wgrad(R)>, db = sum R
    N, C, H, W, K, kh, kw, s, p, g = case
    x, w = _rand(N, C, H, W), _rand(K, C // g, kh, kw)
    y = oracle.conv_forward(x, w, None, s, p, g)
    r = _rand(*y.shape)
    dx, dw, db = oracle.conv_backward(x, w, r, stride=s, pad=p, group=g)
    lhs = float(np.sum(y * r))
    np.testing.assert_allclose(lhs, float(np.sum(x * dx)), rtol=1e-11)
    np.testing.assert_allclose(lhs, float(np.sum(w * dw)), rtol=1e-11)
    np.testing.assert_allclose(db, r.sum(axis=(0, 2, 3)), rtol=1e-12, atol=1e-12)


# ------------------------------------------------------- finite differences
def _loss(x, w, b, g, s, p, grp, relu):
    return float(np.sum(oracle.conv_forward(x, w, b, s, p, grp, relu) * g))


@pytest.mark.parametrize("relu", [False, True])
def test_finite_difference_gradients(relu):
    x = _rand(2, 4, 7, 6)
    w = _rand(4, 2, 3, 2)
    b = _rand(4)
    s, p, grp = 2, 1, 2
    y = oracle.conv_forward(x, w, b, s, p, grp, relu)
    g = _rand(*y.shape)
    dx, dw, db = oracle.conv_backward(x, w, g, top=y, stride=s, pad=p, group=grp, relu=relu)
    h = 1e-6
    rng = np.random.default_rng(7)

    def fd(arr, idx, fn):
        old = arr[idx]
        arr[idx] = old + h
        lp = fn()
        arr[idx] = old - h
        lm = fn()
        arr[idx] = old
        return (lp - lm) / (2 * h)

    fn = lambda: _loss(x, w, b, g, s, p, grp, relu)
    for arr, grad in ((x, dx), (w, dw), (b, db)):
        for _ in range(12):
            idx = tuple(int(rng.integers(0, d)) for d in arr.shape)
            # with relu, skip points whose perturbation crosses a kink
            if relu:
                old = arr[idx]
                arr[idx] = old + h
                yp = oracle.conv_forward(x, w, b, s, p, grp, False)
                arr[idx] = old - h
                ym = oracle.conv_forward(x, w, b, s, p, grp, False)
                arr[idx] = old
                if np.any((yp > 0) != (ym > 0)):
                    continue
            np.testing.assert_allclose(fd(arr, idx, fn), grad[idx], rtol=1e-6, atol=1e-7)


def test_empty_batch():
    x = np.zeros((0, 3, 8, 8))
    w = _rand(4, 3, 3, 3)
    y = oracle.conv_forward(x, w, _rand(4))
    assert y.shape == (0, 4, 6, 6)
    dx, dw, db = oracle.conv_backward(x, w, np.zeros(y.shape))
    assert dx.shape == x.shape
    np.testing.assert_array_equal(dw, 0.0)
    np.testing.assert_array_equal(db, 0.0)


def test_invalid_arguments():
    with pytest.raises(ValueError):
        oracle.conv_forward(_rand(1, 3, 8, 8), _rand(4, 2, 3, 3), group=2)  # C % group
    with pytest.raises(ValueError):
        oracle.conv_forward(_rand(1, 4, 8, 8), _rand(3, 2, 3, 3), group=2)  # K % group
    with pytest.raises(ValueError):
        oracle.conv_forward(_rand(1, 3, 2, 2), _rand(4, 3, 5, 5))  # output < 1
    with pytest.raises(ValueError):
        oracle.conv_backward(_rand(1, 3, 8, 8), _rand(4, 3, 3, 3), _rand(1, 4, 6, 6), top=None,
                             relu=True)  # relu needs top
