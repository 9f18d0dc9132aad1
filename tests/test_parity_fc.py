"""GPU parity of the inner-product (fully connected) layer against the CPU
oracle, through the same C ABI: a 1x1 convolution of a 1x1 image with one
group runs as dense split-K GEMMs on the convolution's MFMA core.

Bar: max|gpu - oracle| / max|oracle| <= 1e-4 per output tensor (fp32).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1408_5093_amd as cc
from paper_1408_5093_amd import workloads as wl
from helpers import TOL_F32, assert_close
from layer_check import check_layer_sampled

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def _np(t):
    torch.cuda.synchronize()
    return t.detach().float().cpu().numpy()


def run_fc(N, C, K, relu, bias=True, seed=0, flags=0):
    print(f"inner product N={N} C={C} K={K} relu={relu} bias={bias} flags={flags}", flush=True)
    rng = np.random.default_rng([79, seed, N, C, K, int(relu), flags])
    x = rng.standard_normal((N, C, 1, 1)).astype(np.float32)
    if flags & cc.BACKWARD_MASK_BOTTOM_DIFF:
        x = np.maximum(x, 0)  # a ReLU output
    w = (rng.standard_normal((K, C, 1, 1)) / np.sqrt(C)).astype(np.float32)
    b = (rng.standard_normal(K) * 0.5).astype(np.float32) if bias else None
    y_ref = oracle.conv_forward(x, w, b, relu=relu)
    y = cc.conv_forward(_t(x), _t(w), _t(b) if bias else None, 1, 0, 1, relu)
    assert_close(_np(y), y_ref, TOL_F32, "forward")

    top = y_ref.astype(np.float32)
    gd = rng.standard_normal(top.shape).astype(np.float32)
    masked_in = bool(flags & cc.BACKWARD_TOP_DIFF_MASKED)
    if masked_in and relu:
        gd = (gd * (top > 0)).astype(np.float32)
    dx_ref, dw_ref, db_ref = oracle.conv_backward(x, w, gd, top=top, relu=relu)
    if flags & cc.BACKWARD_MASK_BOTTOM_DIFF:
        dx_ref = dx_ref * (x > 0)
    dx, dw, db = cc.conv_backward(_t(x), _t(w), _t(gd), None if masked_in else _t(top), 1, 0, 1,
                                  relu, flags=flags)
    assert_close(_np(dx), dx_ref, TOL_F32, "data gradient")
    assert_close(_np(dw), dw_ref, TOL_F32, "weight gradient")
    assert_close(_np(db), db_ref, TOL_F32, "bias gradient")


FC_SWEEP = [
    # N, C, K
    (1, 1, 1),
    (3, 7, 5),
    (5, 16, 33),
    (64, 800, 500),    # LeNet ip1
    (64, 500, 10),     # LeNet ip2
    (37, 100, 130),    # ragged rows, columns and reduction
    (130, 300, 257),
    (2, 2048, 64),     # deep reduction, many splits
    (300, 48, 20),
    (256, 1024, 1000), # 128-row tiles with a ragged last column tile
    (96, 1022, 130),   # C % 4 != 0: the forward goes through X^T and W^T
]


@pytest.mark.parametrize("case", FC_SWEEP)
@pytest.mark.parametrize("relu", [False, True])
def test_inner_product_sweep(case, relu):
    run_fc(*case, relu=relu, bias=relu or case[0] % 2 == 1)


@pytest.mark.parametrize("flags", [1, 2, 3])
def test_inner_product_backward_flags(flags):
    run_fc(40, 72, 96, True, flags=flags)


@pytest.mark.parametrize("N", [64, 2048])
def test_inner_product_accumulate(N):
    # N = 64: one split, the GEMM writes the weight gradient itself unless
    # accumulating; N = 2048: split-K partials and their reduction
    rng = np.random.default_rng([80, N])
    C, K = 512, 1024
    x = rng.standard_normal((N, C, 1, 1)).astype(np.float32)
    w = rng.standard_normal((K, C, 1, 1)).astype(np.float32)
    g = rng.standard_normal((N, K, 1, 1)).astype(np.float32)
    _, dw_ref, db_ref = oracle.conv_backward(x, w, g, need=("dw", "db"))
    dw0 = rng.standard_normal(w.shape).astype(np.float32)
    db0 = rng.standard_normal(K).astype(np.float32)
    dwt, dbt = _t(dw0), _t(db0)
    cc.conv_backward(_t(x), _t(w), _t(g), None, 1, 0, 1, False, need=("dw", "db"), accumulate=1,
                     outs=(None, dwt, dbt))
    assert_close(_np(dwt), dw_ref + dw0, TOL_F32, "accumulated dW")
    assert_close(_np(dbt), db_ref + db0, TOL_F32, "accumulated db")
    dw, db = cc.conv_backward_weights(_t(x), w.shape, _t(g), None, 1, 0, 1, False)
    assert_close(_np(dw), dw_ref, TOL_F32, "dW")
    assert_close(_np(db), db_ref, TOL_F32, "db")


def test_inner_product_separate_entry_points():
    rng = np.random.default_rng(81)
    N, C, K = 96, 300, 200
    x = rng.standard_normal((N, C, 1, 1)).astype(np.float32)
    w = rng.standard_normal((K, C, 1, 1)).astype(np.float32)
    b = rng.standard_normal(K).astype(np.float32)
    top = oracle.conv_forward(x, w, b, relu=True).astype(np.float32)
    g = rng.standard_normal(top.shape).astype(np.float32)
    dx_ref, dw_ref, db_ref = oracle.conv_backward(x, w, g, top=top, relu=True)
    dx = cc.conv_backward_data(x.shape, _t(w), _t(g), _t(top), 1, 0, 1, True)
    dw, db = cc.conv_backward_weights(_t(x), w.shape, _t(g), _t(top), 1, 0, 1, True)
    assert_close(_np(dx), dx_ref, TOL_F32, "data gradient")
    assert_close(_np(dw), dw_ref, TOL_F32, "weight gradient")
    assert_close(_np(db), db_ref, TOL_F32, "bias gradient")


def test_inner_product_empty_batch():
    x = torch.empty((0, 64, 1, 1), device=DEV)
    w = torch.randn((32, 64, 1, 1), device=DEV)
    y = cc.conv_forward(x, w, torch.zeros(32, device=DEV), 1, 0, 1, True)
    assert y.shape == (0, 32, 1, 1)
    g = torch.empty(y.shape, device=DEV)
    dx, dw, db = cc.conv_backward(x, w, g, y, 1, 0, 1, True)
    torch.cuda.synchronize()
    assert dx.shape == x.shape
    assert torch.all(dw == 0) and torch.all(db == 0)


def test_inner_product_bitwise_determinism():
    rng = np.random.default_rng(82)
    x = _t(rng.standard_normal((128, 2048, 1, 1)))
    w = _t(rng.standard_normal((512, 2048, 1, 1)) * 0.02)
    b = _t(rng.standard_normal(512))
    outs = []
    for _ in range(2):
        y = cc.conv_forward(x, w, b, 1, 0, 1, True)
        g = torch.ones_like(y) * 0.5
        outs.append((y,) + cc.conv_backward(x, w, g, y, 1, 0, 1, True))
    torch.cuda.synchronize()
    for a, b_ in zip(*outs):
        assert torch.equal(a, b_)


def test_inner_product_no_writes_outside_outputs():
    rng = np.random.default_rng(83)
    N, C, K = 70, 300, 130
    x = _t(rng.standard_normal((N, C, 1, 1)))
    w = _t(rng.standard_normal((K, C, 1, 1)))
    band, canary = 4096, -12345.0

    def guarded(n):
        buf = torch.full((band + n + band,), canary, device=DEV)
        return buf, buf[band:band + n]

    ybuf, yv = guarded(N * K)
    y = yv.view(N, K, 1, 1)
    cc.conv_forward(x, w, None, 1, 0, 1, True, out=y)
    dxbuf, dxv = guarded(x.numel())
    dwbuf, dwv = guarded(w.numel())
    dbbuf, dbv = guarded(K)
    g = _t(rng.standard_normal((N, K, 1, 1)))
    cc.conv_backward(x, w, g, y, 1, 0, 1, True, outs=(dxv.view(x.shape), dwv.view(w.shape), dbv))
    torch.cuda.synchronize()
    for buf in (ybuf, dxbuf, dwbuf, dbbuf):
        assert torch.all(buf[:band] == canary) and torch.all(buf[-band:] == canary)


@pytest.mark.parametrize("l", [0, 1, 2])
def test_caffenet_fc_full_size(l):
    """fc6..fc8 at N=256: sampled images for the forward pass and the data
    gradient, sampled filters for the weight gradient, every bias gradient."""
    N = 256
    inp = wl.caffenet_fc_layer(l, N)
    L = wl.CAFFENET_FC[l]
    x, w = _t(inp["x"]), _t(inp["W"])
    y = cc.conv_forward(x, w, _t(inp["b"]), 1, 0, 1, L.relu)
    dx, dw, db = cc.conv_backward(x, w, _t(inp["top_diff"]), y, 1, 0, 1, L.relu)
    check_layer_sampled(L, inp["x"], inp["W"], inp["b"], _np(y), inp["top_diff"], _np(dx),
                        _np(dw), _np(db), images=[0, 129, N - 1], filters=[0, L.K // 2, L.K - 1],
                        what=L.name)
