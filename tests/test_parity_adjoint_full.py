"""Whole-tensor checks of every CaffeNet layer at full batch on the GPU.

The forward map F(X, W) (no bias, no ReLU) is linear in X and in W; the data
gradient is the adjoint of X -> F(X, W) and the weight gradient the adjoint of
W -> F(X, W), so for any top gradient R

    <F(X, W), R> = <X, dgrad(R)> = <W, wgrad(R)>.

With R = Y = F(X, W) the identities hold image by image and filter by filter
as sums of squares (convolution acts on each image alone, and output channel
k depends only on filter k):

    <X_n, dgrad(Y)_n> = ||Y_n||^2        for every image n,
    <W_k, wgrad(Y)_k> = ||Y_k||^2        for every filter k,

and a launch tile that was skipped or written wrong anywhere in dX or dW
moves its image's or filter's sum by its share of that sum, far above the
tolerance.  The bf16 form uses R = bf16(Y) (the library rounds the top
gradient to bf16 before the products; R is then exact) and compares with
<Y, R> image by image and filter by filter.  Every sum is taken in float64
over all elements of the tensors the GPU produced; nothing is sampled.
"""
import numpy as np
import pytest
import torch

import paper_1408_5093_amd as cc
from paper_1408_5093_amd import workloads as wl

pytestmark = pytest.mark.gpu

# fp32 accumulation of up to ~10^4 products per output: relative error of a
# positive sum of squares well below 1e-5
TOL = 1e-4


def _inputs(L, N, seed, bf16):
    g = torch.Generator(device="cuda").manual_seed(seed)
    x = torch.randn((N, L.C, L.H, L.W), device="cuda", generator=g)
    if L.C != 3:
        x = x.abs()
    w = torch.randn((L.K, L.C // L.g, L.k, L.k), device="cuda", generator=g) * 0.01
    if bf16:
        x, w = x.to(torch.bfloat16), w.to(torch.bfloat16)
    return x, w


def _check(L, N, bf16, seed):
    print(f"adjoint {L.name} N={N} bf16={bf16}", flush=True)
    x, w = _inputs(L, N, seed, bf16)
    y = cc.conv_forward(x, w, None, L.s, L.p, L.g, relu=False)
    r = y.to(torch.bfloat16).float() if bf16 else y
    dx, dw, _ = cc.conv_backward(x, w, r, None, L.s, L.p, L.g, relu=False, need=("dx", "dw"))
    torch.cuda.synchronize()
    yr = y.double() * r.double()
    assert torch.isfinite(dx).all() and torch.isfinite(dw).all()
    # image by image: <X_n, dX_n> = <Y_n, R_n>
    lhs = (x.double() * dx.double()).sum(dim=(1, 2, 3))
    rhs = yr.sum(dim=(1, 2, 3))
    err = ((lhs - rhs).abs() / rhs.abs()).max().item()
    assert err <= TOL, f"{L.name} data gradient: image identity off by {err:.2e}"
    # filter by filter: <W_k, dW_k> = <Y_k, R_k>
    lhs = (w.double() * dw.double()).sum(dim=(1, 2, 3))
    rhs = yr.sum(dim=(0, 2, 3))
    err = ((lhs - rhs).abs() / rhs.abs()).max().item()
    assert err <= TOL, f"{L.name} weight gradient: filter identity off by {err:.2e}"
    del x, w, y, r, dx, dw, yr
    torch.cuda.empty_cache()


@pytest.mark.parametrize("l", range(5), ids=[L.name for L in wl.CAFFENET])
def test_caffenet_layer_adjoint_f32_n256(l):
    _check(wl.CAFFENET[l], 256, False, 100 + l)


@pytest.mark.parametrize("l", range(5), ids=[L.name for L in wl.CAFFENET])
def test_caffenet_layer_adjoint_bf16_n512(l):
    _check(wl.CAFFENET[l], 512, True, 200 + l)


def test_identity_catches_a_skipped_tile():
    """The check itself: zeroing one 128 x 128 block of a correct conv2
    weight gradient (filters 128..255, taps 0..127 of group 1) moves those
    filters' sums far beyond the tolerance."""
    L = wl.CAFFENET[1]
    x, w = _inputs(L, 32, 7, False)
    y = cc.conv_forward(x, w, None, L.s, L.p, L.g, relu=False)
    _, dw, _ = cc.conv_backward(x, w, y, None, L.s, L.p, L.g, relu=False, need=("dw",))
    dwf = dw.view(L.K, -1).clone()
    dwf[128:256, 0:128] = 0
    lhs = (w.double().view(L.K, -1) * dwf.double()).sum(dim=1)
    rhs = (y.double() ** 2).sum(dim=(0, 2, 3))
    err = ((lhs - rhs).abs() / rhs).max().item()
    print(f"skipped tile moves the filter identity by {err:.2e}")
    assert err > 10 * TOL
