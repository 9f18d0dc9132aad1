"""caffe_conv_backward_pool_lrn: a convolution layer's backward pass from the
gradient of the LRN that follows its max-pool, in one call.

Checked three ways on the same seeded inputs:
- against the unfused GPU path (caffe_lrn_pool_backward, then
  caffe_conv_backward on its float output): the staged bf16 top gradient is
  the same, so dX and dW agree bit for bit; the bias gradient sums the same
  float values in another fixed order;
- the glue part against the oracle: lrn_backward, then maxpool_backward, with
  the ReLU's backward (route only to positive winners);
- the convolution part against the oracle on the operands the GPU multiplied
  (bf16: the rounded inputs, weights and top gradient).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1408_5093_amd as cc
from helpers import TOL_F32, assert_close

pytestmark = pytest.mark.gpu
DEV = "cuda"

# (N, C, H, W, K, k, s, p, g, bf16, relu_input): the pool is 3x3/2 and the LRN
# local_size 5 (CaffeNet's glue)
CASES = [
    (3, 8, 15, 15, 32, 3, 1, 1, 1, True, True),    # staged in bf16, ReLU folded into the pool
    (2, 8, 13, 17, 64, 3, 1, 1, 2, True, False),   # staged, grouped, ReLU mask from top
    (2, 6, 14, 14, 40, 3, 1, 1, 2, True, True),    # K/g = 20: through the float gradient
    (2, 8, 15, 15, 32, 3, 1, 1, 1, False, True),   # float operands
    (2, 3, 59, 59, 32, 11, 4, 0, 1, True, True),   # conv1's stride-4 geometry, staged
    (2, 16, 27, 27, 64, 5, 1, 2, 2, True, True),   # conv2's geometry, staged
    (2, 16, 27, 27, 64, 5, 1, 2, 2, "f32", True),  # the same from a float bottom
    (2, 8, 13, 17, 64, 3, 1, 1, 2, "f32", False),  # float bottom, ReLU mask from top
]
POOL = dict(kernel=3, stride=2, pad=0)
LRN = dict(size=5, alpha=1e-4, beta=0.75, k=1.0)


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("case", CASES)
def test_backward_pool_lrn(case):
    N, C, H, W, K, k, s, p, g, bf16, relu_input = case
    print(f"backward_pool_lrn {case}", flush=True)
    rng = np.random.default_rng([1408, 5093, 90, sum(case[:9])])
    # bf16 == "f32": bf16 weights and a float bottom the library rounds
    # (CAFFE_BF16_F32_BOTTOM)
    f32_bottom = bf16 == "f32"
    op = torch.bfloat16 if bf16 else torch.float32
    x = torch.from_numpy(rng.standard_normal((N, C, H, W)).astype(np.float32)).to(DEV)
    x = x if f32_bottom else x.to(op)
    w = torch.from_numpy((rng.standard_normal((K, C // g, k, k)) * 0.2).astype(np.float32))
    w = w.to(DEV).to(op)
    b = torch.from_numpy(rng.standard_normal(K).astype(np.float32) * 0.1).to(DEV)
    top = cc.conv_forward(x, w, b, s, p, g, relu=True)
    flags_pool = cc.POOL_RELU_INPUT if relu_input else 0
    pooled, mask, lrn_top = cc.pool_lrn_forward(top, flags=flags_pool, **POOL, **LRN)
    gl = torch.from_numpy(rng.standard_normal(lrn_top.shape).astype(np.float32)).to(DEV)

    dt = cc.CAFFE_BF16_F32_BOTTOM if f32_bottom else cc.CAFFE_BF16 if bf16 else cc.CAFFE_F32
    d = cc.conv_desc(x.shape, w.shape, s, p, g, True, dt)
    pd = cc.pool_desc(top.shape, POOL["kernel"], POOL["stride"], POOL["pad"])
    ld = cc.lrn_desc(pooled.shape, **LRN)
    flags = cc.BACKWARD_TOP_DIFF_MASKED if relu_input else 0
    dx = torch.full(x.shape, float("nan"), device=DEV)
    dw = torch.full(w.shape, float("nan"), device=DEV)
    db = torch.full((K,), float("nan"), device=DEV)
    ws = cc.Workspace().get(cc.conv_workspace_size(d, cc.PASS_BACKWARD_POOL_LRN))
    ws.fill_(0x7E)  # (large finite bf16 values: a staging border left unzeroed shows)
    cc.caffe_conv_backward_pool_lrn(d, pd, ld, pooled, lrn_top, gl, mask,
                                    None if relu_input else top, x, w, dx, dw, db, 0, flags, ws)

    # the unfused GPU path
    gtop = cc.lrn_pool_backward(top.shape, pooled, lrn_top, gl, mask, **POOL, **LRN)
    if not relu_input:
        gtop = gtop * (top > 0)
    dx2, dw2, db2 = cc.conv_backward(x, w, gtop, None, s, p, g, relu=True,
                                     flags=cc.BACKWARD_TOP_DIFF_MASKED)
    torch.cuda.synchronize()
    assert torch.equal(dx, dx2), "data gradient differs from the unfused path"
    assert torch.equal(dw, dw2), "weight gradient differs from the unfused path"
    assert_close(_np(db), _np(db2), 1e-6, "bias gradient vs the unfused path")

    # the glue against the oracle (route only to positive winners: the ReLU)
    topn = _np(top)
    gref = oracle.lrn_backward(_np(pooled), _np(gl), LRN["size"], LRN["alpha"], LRN["beta"],
                               LRN["k"])
    gref = oracle.maxpool_backward(topn, gref, POOL["kernel"], POOL["stride"]) * (topn > 0)
    gg = _np(gtop)
    assert_close(gg, gref, TOL_F32, "glue backward vs the oracle")
    # the convolution against the oracle on the operands the GPU multiplied
    gmul = _np(gtop.to(torch.bfloat16)) if bf16 else gg
    xm = _np(x.to(torch.bfloat16)) if f32_bottom else _np(x)   # the bottom multiplied
    dx_r, dw_r, _ = oracle.conv_backward(xm, _np(w), gmul, stride=s, pad=p, group=g)
    _, _, db_r = oracle.conv_backward(xm, _np(w), gg, stride=s, pad=p, group=g, need=("db",))
    assert_close(_np(dx), dx_r, TOL_F32, "data gradient vs the oracle")
    assert_close(_np(dw), dw_r, TOL_F32, "weight gradient vs the oracle")
    assert_close(_np(db), db_r, TOL_F32, "bias gradient vs the oracle")


@pytest.mark.parametrize("case", CASES)
def test_backward_pool_lrn_byte_mask(case):
    """The max-pool's winners recorded as bytes (each one's offset in its
    window, CAFFE_POOL_MASK_OFFSETS) and read so by the fused backward
    (CAFFE_BACKWARD_POOL_MASK_OFFSETS): the same pooled blob and every
    gradient bit for bit against the 32-bit plane-index mask."""
    N, C, H, W, K, k, s, p, g, bf16, relu_input = case
    print(f"backward_pool_lrn byte mask {case}", flush=True)
    rng = np.random.default_rng([1408, 5093, 92, sum(case[:9])])
    f32_bottom = bf16 == "f32"
    op = torch.bfloat16 if bf16 else torch.float32
    x = torch.from_numpy(rng.standard_normal((N, C, H, W)).astype(np.float32)).to(DEV)
    x = x if f32_bottom else x.to(op)
    w = torch.from_numpy((rng.standard_normal((K, C // g, k, k)) * 0.2).astype(np.float32))
    w = w.to(DEV).to(op)
    b = torch.from_numpy(rng.standard_normal(K).astype(np.float32) * 0.1 - 0.2).to(DEV)
    top = cc.conv_forward(x, w, b, s, p, g, relu=True)
    dt = cc.CAFFE_BF16_F32_BOTTOM if f32_bottom else cc.CAFFE_BF16 if bf16 else cc.CAFFE_F32
    d = cc.conv_desc(x.shape, w.shape, s, p, g, True, dt)
    fl_pool = cc.POOL_RELU_INPUT if relu_input else 0
    fl = cc.BACKWARD_TOP_DIFF_MASKED if relu_input else 0
    outs = []
    for byte in (False, True):
        pooled, mask, lrn_top = cc.pool_lrn_forward(
            top, flags=fl_pool | (cc.POOL_MASK_OFFSETS if byte else 0), **POOL, **LRN)
        assert mask.dtype == (torch.uint8 if byte else torch.int32)
        gl = torch.from_numpy(np.random.default_rng(7).standard_normal(
            tuple(lrn_top.shape)).astype(np.float32)).to(DEV)
        pd = cc.pool_desc(top.shape, POOL["kernel"], POOL["stride"], POOL["pad"])
        ld = cc.lrn_desc(pooled.shape, **LRN)
        dx = torch.full(x.shape, float("nan"), device=DEV)
        dw = torch.full(w.shape, float("nan"), device=DEV)
        db = torch.full((K,), float("nan"), device=DEV)
        ws = cc.Workspace().get(cc.conv_workspace_size(d, cc.PASS_BACKWARD_POOL_LRN))
        cc.caffe_conv_backward_pool_lrn(d, pd, ld, pooled, lrn_top, gl, mask,
                                        None if relu_input else top, x, w, dx, dw, db, 0,
                                        fl | (cc.BACKWARD_POOL_MASK_OFFSETS if byte else 0), ws)
        torch.cuda.synchronize()
        outs.append((pooled, dx, dw, db))
    for name, a, c in zip(("pooled", "dx", "dw", "db"), *outs):
        assert torch.equal(a, c), name


def test_backward_pool_lrn_rejects_mismatched_pool():
    """The pool must describe the layer's top: checked on the host, nothing
    launched."""
    d = cc.conv_desc((2, 8, 15, 15), (32, 8, 3, 3), 1, 1, 1, True, cc.CAFFE_BF16)
    pd = cc.pool_desc((2, 16, 15, 15), 3, 2)
    ld = cc.lrn_desc((2, 16, 7, 7))
    P = torch.empty(16, device=DEV)
    with pytest.raises(cc.CaffeError):
        cc.caffe_conv_backward_pool_lrn(d, pd, ld, P, P, P, P.view(torch.int32), None, None,
                                        None, None, None, None, 0, cc.BACKWARD_TOP_DIFF_MASKED,
                                        None)
