"""GPU parity of the convolution layer (C ABI -> gfx950 kernels) against the
CPU oracle on identical seeded inputs.

Bar: max|gpu - oracle| / max|oracle| <= 1e-4 per output tensor (fp32).  The
backward pass gets the same `top` (the oracle's forward output rounded to
fp32) on both sides, so the ReLU mask [top > 0] is identical.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1408_5093_amd as cc
from helpers import TOL_F32, assert_close

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _t(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV, dtype)


def _np(t):
    torch.cuda.synchronize()
    return t.detach().float().cpu().numpy()


def run_case(N, C, H, W, K, kh, kw, sh, sw, ph, pw, g, relu, bias=True, seed=0, tol=TOL_F32):
    print(f"case N={N} C={C} H={H} W={W} K={K} k={kh}x{kw} s={sh},{sw} p={ph},{pw} g={g} "
          f"relu={relu} bias={bias}", flush=True)
    rng = np.random.default_rng([77, seed, N, C, H, W, K, kh, kw, sh, sw, ph, pw, g, int(relu)])
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    w = (rng.standard_normal((K, C // g, kh, kw)) * 0.3).astype(np.float32)
    b = (rng.standard_normal(K) * 0.5).astype(np.float32) if bias else None
    y_ref = oracle.conv_forward(x, w, b, (sh, sw), (ph, pw), g, relu)
    y = cc.conv_forward(_t(x), _t(w), _t(b) if bias else None, (sh, sw), (ph, pw), g, relu)
    assert_close(_np(y), y_ref, tol, "forward")

    top = y_ref.astype(np.float32)
    gd = rng.standard_normal(top.shape).astype(np.float32)
    dx_ref, dw_ref, db_ref = oracle.conv_backward(x, w, gd, top=top, stride=(sh, sw),
                                                  pad=(ph, pw), group=g, relu=relu)
    dx, dw, db = cc.conv_backward(_t(x), _t(w), _t(gd), _t(top), (sh, sw), (ph, pw), g, relu)
    assert_close(_np(dx), dx_ref, tol, "data gradient")
    assert_close(_np(dw), dw_ref, tol, "weight gradient")
    assert_close(_np(db), db_ref, tol, "bias gradient")
    return y, dx, dw, db


# geometry sweep: strides 1-4, pads 0-3, kernels 1-11, groups 1-4, ragged sizes
SWEEP = [
    # N, C, H, W, K, kh, kw, sh, sw, ph, pw, g
    (2, 3, 17, 19, 5, 3, 3, 1, 1, 1, 1, 1),
    (1, 1, 9, 9, 1, 1, 1, 1, 1, 0, 0, 1),
    (3, 7, 19, 19, 150, 3, 3, 1, 1, 1, 1, 1),     # 2 row tiles, ragged columns
    (2, 8, 15, 13, 12, 5, 5, 1, 1, 2, 2, 2),
    (2, 3, 35, 35, 16, 11, 11, 4, 4, 0, 0, 1),    # conv1-like
    (2, 3, 37, 33, 10, 11, 11, 4, 4, 2, 1, 1),    # conv1-like, padded, ragged
    (1, 12, 11, 11, 20, 3, 3, 2, 2, 1, 1, 4),
    (2, 6, 10, 14, 9, 2, 3, 3, 2, 1, 2, 3),       # stride > kernel rows
    (1, 4, 8, 8, 6, 3, 3, 1, 1, 3, 3, 2),         # pad = kernel
    (2, 5, 7, 6, 7, 7, 6, 1, 1, 0, 0, 1),         # kernel = image (1x1 output)
    (3, 96, 13, 13, 70, 5, 5, 1, 1, 2, 2, 2),
    (1, 2, 40, 3, 4, 1, 3, 1, 1, 0, 1, 1),
    (2, 16, 9, 9, 200, 1, 1, 1, 1, 0, 0, 1),      # 1x1 conv, 2 row tiles
    (1, 4, 23, 23, 48, 4, 4, 3, 3, 1, 1, 1),
    (2, 9, 12, 12, 33, 5, 5, 2, 2, 2, 2, 3),
]


@pytest.mark.parametrize("case", SWEEP)
@pytest.mark.parametrize("relu", [False, True])
def test_sweep(case, relu):
    run_case(*case, relu=relu, bias=(case[0] % 2 == 0) or relu)


def test_tile_shapes_each_chooser_branch():
    # output channels per group hitting each tile height: 20 (48-row tile), 50 (64),
    # 96 (96), 128 (128), 192 (96 x 2), 256 (128 x 2), plus a 3-row-tile case
    for K, g in [(20, 1), (50, 1), (96, 1), (128, 1), (384, 2), (256, 1), (300, 1)]:
        run_case(2, 2 * g, 9, 10, K, 3, 3, 1, 1, 1, 1, g, True)


def test_data_gradient_phase_stacked_row_heights():
    # C/group * stride^2 rows: 3*16 = 48 (conv1), 1*4, 5*9, 8*16 = 128
    for C, s, k in [(3, 4, 11), (1, 2, 5), (5, 3, 7), (8, 4, 5)]:
        run_case(2, C, 29, 31, 6, k, k, s, s, 1, 2, 1, True)


@pytest.mark.parametrize("C", [4, 8])  # 8: 4 channels per group, the quad-order weight gradient
def test_empty_batch(C):
    x = torch.empty((0, C, 9, 9), device=DEV)
    w = torch.randn((6, C // 2, 3, 3), device=DEV)
    y = cc.conv_forward(x, w, torch.zeros(6, device=DEV), 1, 1, 2, True)
    assert y.shape == (0, 6, 9, 9)
    g = torch.empty(y.shape, device=DEV)
    dx, dw, db = cc.conv_backward(x, w, g, y, 1, 1, 2, True)
    torch.cuda.synchronize()
    assert dx.shape == x.shape
    assert torch.all(dw == 0) and torch.all(db == 0)


def test_accumulate_adds():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 4, 11, 11)).astype(np.float32)
    w = rng.standard_normal((8, 4, 3, 3)).astype(np.float32)
    g = rng.standard_normal((2, 8, 11, 11)).astype(np.float32)
    _, dw_ref, db_ref = oracle.conv_backward(x, w, g, stride=1, pad=1)
    dw0 = rng.standard_normal(w.shape).astype(np.float32)
    db0 = rng.standard_normal(8).astype(np.float32)
    dwt, dbt = _t(dw0), _t(db0)
    cc.conv_backward(_t(x), _t(w), _t(g), None, 1, 1, 1, False, need=("dw", "db"), accumulate=1,
                     outs=(None, dwt, dbt))
    assert_close(_np(dwt), dw_ref + dw0, TOL_F32, "accumulated dW")
    assert_close(_np(dbt), db_ref + db0, TOL_F32, "accumulated db")


def test_separate_entry_points_match_combined():
    rng = np.random.default_rng(9)
    x = _t(rng.standard_normal((2, 6, 13, 13)))
    w = _t(rng.standard_normal((10, 3, 3, 3)) * 0.2)
    y = cc.conv_forward(x, w, None, 1, 1, 2, True)
    g = _t(rng.standard_normal(y.shape))
    dx, dw, db = cc.conv_backward(x, w, g, y, 1, 1, 2, True)
    dx2 = cc.conv_backward_data(x.shape, w, g, y, 1, 1, 2, True)
    dw2, db2 = cc.conv_backward_weights(x, w.shape, g, y, 1, 1, 2, True)
    torch.cuda.synchronize()
    assert torch.equal(dx, dx2) and torch.equal(dw, dw2) and torch.equal(db, db2)


def test_bitwise_determinism():
    rng = np.random.default_rng(11)
    x = _t(rng.standard_normal((4, 16, 27, 27)))
    w = _t(rng.standard_normal((32, 8, 5, 5)) * 0.1)
    b = _t(rng.standard_normal(32))
    outs = []
    for _ in range(2):
        y = cc.conv_forward(x, w, b, 1, 2, 2, True)
        g = torch.ones_like(y) * 0.5
        outs.append((y,) + cc.conv_backward(x, w, g, y, 1, 2, 2, True))
    torch.cuda.synchronize()
    for a, b_ in zip(*outs):
        assert torch.equal(a, b_)


def test_no_writes_outside_outputs():
    # canary bands around every output buffer must survive forward + backward
    rng = np.random.default_rng(13)
    N, C, H, W, K = 3, 6, 14, 15, 20
    x = _t(rng.standard_normal((N, C, H, W)))
    w = _t(rng.standard_normal((K, C // 2, 3, 3)))
    band = 4096
    canary = -12345.0

    def guarded(n):
        buf = torch.full((band + n + band,), canary, device=DEV)
        return buf, buf[band:band + n]

    ybuf, yv = guarded(N * K * H * W)
    y = yv.view(N, K, H, W)
    d = cc.conv_desc(x.shape, w.shape, 1, 1, 2, True)
    cc.caffe_conv_forward(d, x, w, None, y,
                          cc.Workspace().get(cc.conv_workspace_size(d, cc.PASS_FORWARD)))
    dxbuf, dxv = guarded(x.numel())
    dwbuf, dwv = guarded(w.numel())
    dbbuf, dbv = guarded(K)
    g = _t(rng.standard_normal((N, K, H, W)))
    cc.conv_backward(x, w, g, y, 1, 1, 2, True,
                     outs=(dxv.view(x.shape), dwv.view(w.shape), dbv))
    torch.cuda.synchronize()
    for buf in (ybuf, dxbuf, dwbuf, dbbuf):
        assert torch.all(buf[:band] == canary) and torch.all(buf[-band:] == canary)


def test_backward_flags_fused_relu():
    """CAFFE_BACKWARD_TOP_DIFF_MASKED: top_diff comes masked and top is not
    read; CAFFE_BACKWARD_MASK_BOTTOM_DIFF: bottom_diff = adjoint(D) [bottom > 0]."""
    rng = np.random.default_rng(21)
    N, C, H, W, K = 2, 8, 13, 13, 24
    x = np.maximum(rng.standard_normal((N, C, H, W)), 0).astype(np.float32)  # a ReLU output
    w = (rng.standard_normal((K, C // 2, 3, 3)) * 0.3).astype(np.float32)
    b = rng.standard_normal(K).astype(np.float32)
    y_ref = oracle.conv_forward(x, w, b, 1, 1, 2, True)
    top = y_ref.astype(np.float32)
    gd = rng.standard_normal(top.shape).astype(np.float32)
    dx_ref, dw_ref, db_ref = oracle.conv_backward(x, w, gd, top=top, stride=1, pad=1, group=2,
                                                  relu=True)
    gmasked = (gd * (top > 0)).astype(np.float32)
    for flags in (cc.BACKWARD_TOP_DIFF_MASKED, cc.BACKWARD_MASK_BOTTOM_DIFF,
                  cc.BACKWARD_TOP_DIFF_MASKED | cc.BACKWARD_MASK_BOTTOM_DIFF):
        masked_in = flags & cc.BACKWARD_TOP_DIFF_MASKED
        g_in = gmasked if masked_in else gd
        top_in = None if masked_in else _t(top)
        dx, dw, db = cc.conv_backward(_t(x), _t(w), _t(g_in), top_in, 1, 1, 2, True, flags=flags)
        want_dx = dx_ref * (x > 0) if flags & cc.BACKWARD_MASK_BOTTOM_DIFF else dx_ref
        assert_close(_np(dx), want_dx, TOL_F32, f"dx flags={flags}")
        assert_close(_np(dw), dw_ref, TOL_F32, f"dw flags={flags}")
        assert_close(_np(db), db_ref, TOL_F32, f"db flags={flags}")
    # bias gradient alone from a masked top gradient
    dx, dw, db = cc.conv_backward(_t(x), _t(w), _t(gmasked), None, 1, 1, 2, True, need=("db",),
                                  flags=cc.BACKWARD_TOP_DIFF_MASKED)
    assert_close(_np(db), db_ref, TOL_F32, "db only, masked")


# ------------------------------------------------ split-K forward / data gradient
SPLIT_CASES = [
    (2, 32, 9, 9, 64, 3, 3, 1, 1, 1, 1, 1),       # reduction-blocked / tap-major walks
    (1, 48, 11, 10, 96, 5, 5, 1, 1, 2, 2, 2),     # groups, 48 channels per group
    (2, 3, 35, 35, 16, 11, 11, 4, 4, 0, 0, 1),    # conv1-like: 11x11/4, phase-stacked gradient
    (3, 7, 19, 19, 150, 3, 3, 1, 1, 1, 1, 1),     # generic gather, 2 row tiles, ragged columns
    (2, 9, 12, 12, 33, 5, 5, 2, 2, 2, 2, 3),      # stride-2 phases, 3 groups
]


@pytest.mark.parametrize("case", SPLIT_CASES)
@pytest.mark.parametrize("splits", [2, 5])
@pytest.mark.parametrize("blocked", ["1", "0"])
def test_split_k(case, splits, blocked, overrides):
    """Forced split counts (profiling overrides) on both reduction orders:
    each split starts its walk mid-reduction, the reduce applies the
    epilogue."""
    overrides.setenv("CAFFE_CONV_FWD_SPLITS", str(splits))
    overrides.setenv("CAFFE_CONV_DGRAD_SPLITS", str(splits))
    overrides.setenv("CAFFE_CONV_BLOCKED", blocked)
    run_case(*case, relu=True, bias=True)
    run_case(*case, relu=False, bias=False, seed=1)


@pytest.mark.parametrize("case", SPLIT_CASES)
@pytest.mark.parametrize("splits,units", [(2, 1), (3, 2)])
def test_tail_split(case, splits, units, overrides):
    """Tail splits (the last column tiles of the last group cut into
    reduction ranges, their partials finished by a reduce over that region),
    forced by the profiling overrides as if the device had `units` compute
    units: the forward and data gradient match the oracle with and without
    bias, ReLU and the blocked order."""
    overrides.setenv("CAFFE_CONV_TAIL_SPLITS", str(splits))
    overrides.setenv("CAFFE_CONV_TAIL_UNITS", str(units))
    run_case(*case, relu=True, bias=True)
    overrides.setenv("CAFFE_CONV_BLOCKED", "0")
    run_case(*case, relu=False, bias=False, seed=1)


@pytest.mark.parametrize("case", [
    # N, C, H, W, K, k, pad, group, blocks (the split target): which weight-
    # gradient kernel runs follows from the shape (3x3 / 5x5 LDS-DMA, any-tap)
    (12, 64, 13, 13, 128, 3, 1, 2, 48),    # 2 groups x 8 splits
    (6, 48, 14, 11, 96, 5, 2, 1, 80),      # one group, 7 splits (the most), ragged
    (5, 3, 23, 23, 32, 7, 0, 1, 0),        # the any-tap kernel, default splits
])
def test_wgrad_unit_order(case, overrides):
    """The fp32 weight gradient with each (group, split) unit's tiles on one
    XCD against the linear order at the same split count: the same partials
    in the same order, so the same bits; and the oracle."""
    N, C, H, W, K, k, pad, g, blocks = case
    print(f"wgrad unit order {case}", flush=True)
    rng = np.random.default_rng([80, *case])
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    w = rng.standard_normal((K, C // g, k, k)).astype(np.float32)
    gd = rng.standard_normal((N, K, H + 2 * pad - k + 1, W + 2 * pad - k + 1)).astype(np.float32)
    if blocks:
        overrides.setenv("CAFFE_CONV_WGRAD_BLOCKS", str(blocks))
    dws = []
    for order in ("1", "0"):
        overrides.setenv("CAFFE_CONV_WGRAD_UNIT_ORDER", order)
        _, dw, _ = cc.conv_backward(_t(x), _t(w), _t(gd), None, 1, pad, g, need=("dw",))
        torch.cuda.synchronize()
        dws.append(dw)
    assert torch.equal(dws[0], dws[1])
    _, dw_ref, _ = oracle.conv_backward(x, w, gd, stride=1, pad=pad, group=g, need=("dw",))
    assert_close(_np(dws[0]), dw_ref, TOL_F32, "weight gradient")


def test_split_k_masked_bottom_and_default_plan(overrides):
    # the bottom mask applied by the data-gradient reduce; then a shape whose
    # own plan splits (one image, a long reduction)
    overrides.setenv("CAFFE_CONV_DGRAD_SPLITS", "3")
    rng = np.random.default_rng(31)
    x = np.maximum(rng.standard_normal((2, 16, 10, 10)), 0).astype(np.float32)
    w = rng.standard_normal((32, 16, 3, 3)).astype(np.float32)
    g = rng.standard_normal((2, 32, 10, 10)).astype(np.float32)
    dx_ref, _, _ = oracle.conv_backward(x, w, g, stride=1, pad=1, need=("dx",))
    dx, _, _ = cc.conv_backward(_t(x), _t(w), _t(g), None, 1, 1, 1, False, need=("dx",),
                                flags=cc.BACKWARD_MASK_BOTTOM_DIFF)
    assert_close(_np(dx), dx_ref * (x > 0), TOL_F32, "masked data gradient")
    overrides.delenv("CAFFE_CONV_DGRAD_SPLITS")
    run_case(1, 64, 6, 6, 64, 5, 5, 1, 1, 2, 2, 1, True)


# Weight gradients in the quad tap order (Cg % 4 == 0, 3x3 or 5x5 kernels):
# several tap tiles with a ragged tail, each row tile height, groups, strides,
# pads up to the kernel size and a ragged column count.
QUAD_CASES = [
    # N, C, H, W, K, kh, kw, sh, sw, ph, pw, g
    (2, 36, 11, 9, 70, 3, 3, 1, 1, 1, 1, 1),      # R = 324: 3 tap tiles, ragged rows
    (3, 8, 13, 12, 192, 3, 3, 2, 2, 1, 1, 2),     # stride 2, Kg = 96 (96-row tile)
    (2, 16, 9, 10, 128, 5, 5, 1, 1, 2, 2, 1),     # 128-row tile
    (1, 24, 7, 7, 128, 5, 5, 1, 1, 4, 4, 2),      # pad = kernel - 1, Kg = 64
    (5, 4, 6, 5, 10, 3, 3, 1, 1, 0, 0, 1),        # unpadded, 60 columns
    (2, 12, 8, 9, 21, 3, 3, 1, 2, 3, 0, 3),       # uneven stride and pad, 3 groups
]


@pytest.mark.parametrize("case", QUAD_CASES)
def test_weight_gradient_quad_order(case, overrides):
    """The quad-order kernel (register-staged copies) against the oracle, and
    bit for bit against the channel-major kernel (same sums, same order; only
    the tile columns are permuted)."""
    overrides.setenv("CAFFE_CONV_WGRAD_QUAD", "1")
    overrides.setenv("CAFFE_CONV_WGRAD_DMA", "0")
    N, C, H, W, K, kh, kw, sh, sw, ph, pw, g = case
    rng = np.random.default_rng([91, N, C, H, W, K])
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    w = (rng.standard_normal((K, C // g, kh, kw)) * 0.3).astype(np.float32)
    top = np.maximum(rng.standard_normal((N, K, (H + 2 * ph - kh) // sh + 1,
                                          (W + 2 * pw - kw) // sw + 1)), 0).astype(np.float32)
    gd = rng.standard_normal(top.shape).astype(np.float32)
    _, dw_ref, db_ref = oracle.conv_backward(x, w, gd, top=top, stride=(sh, sw), pad=(ph, pw),
                                             group=g, relu=True, need=("dw", "db"))
    args = (_t(x), _t(w), _t(gd), _t(top), (sh, sw), (ph, pw), g, True)
    _, dw, db = cc.conv_backward(*args, need=("dw", "db"))
    assert_close(_np(dw), dw_ref, TOL_F32, "weight gradient")
    assert_close(_np(db), db_ref, TOL_F32, "bias gradient")
    overrides.setenv("CAFFE_CONV_WGRAD_QUAD", "0")
    _, dw0, db0 = cc.conv_backward(*args, need=("dw", "db"))
    torch.cuda.synchronize()
    assert torch.equal(dw, dw0) and torch.equal(db, db0)


@pytest.mark.parametrize("case", [
    (2, 3, 35, 35, 16, 11, 11, 4, 4, 0, 0, 1),    # every window inside: table offsets
    (2, 5, 23, 21, 40, 4, 4, 3, 3, 1, 1, 1),      # padded: inner waves on the table
    (3, 6, 9, 9, 10, 3, 3, 1, 1, 0, 0, 2),        # groups, ragged columns
])
def test_forward_tap_table(case, overrides):
    """The channel-major forward with its tap-offset table against the
    oracle, and bit for bit against the scalar tap walk."""
    N, C, H, W, K, kh, kw, sh, sw, ph, pw, g = case
    rng = np.random.default_rng([93, N, C, H, W, K])
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    w = (rng.standard_normal((K, C // g, kh, kw)) * 0.3).astype(np.float32)
    b = rng.standard_normal(K).astype(np.float32)
    y_ref = oracle.conv_forward(x, w, b, (sh, sw), (ph, pw), g, True)
    overrides.setenv("CAFFE_CONV_TAP_TABLE", "1")
    y = cc.conv_forward(_t(x), _t(w), _t(b), (sh, sw), (ph, pw), g, True)
    assert_close(_np(y), y_ref, TOL_F32, "forward")
    overrides.setenv("CAFFE_CONV_TAP_TABLE", "0")
    y0 = cc.conv_forward(_t(x), _t(w), _t(b), (sh, sw), (ph, pw), g, True)
    torch.cuda.synchronize()
    assert torch.equal(y, y0)


@pytest.mark.parametrize("tile", [-1, 1, 3])
def test_data_gradient_192_rows_masked(tile, overrides):
    """192 gathered rows per group (conv4/conv5's data gradient): the default
    tile choice, the 96-row and the 64-row tiles, with the bottom mask."""
    overrides.setenv("CAFFE_CONV_DGRAD_TILE", str(tile))
    rng = np.random.default_rng(23)
    N, C, H, W, K, g = 2, 384, 7, 6, 32, 2
    x = np.maximum(rng.standard_normal((N, C, H, W)), 0).astype(np.float32)
    w = (rng.standard_normal((K, C // g, 3, 3)) * 0.1).astype(np.float32)
    gd = rng.standard_normal((N, K, H, W)).astype(np.float32)
    dx_ref, _, _ = oracle.conv_backward(x, w, gd, stride=1, pad=1, group=g, need=("dx",))
    dx, _, _ = cc.conv_backward(_t(x), _t(w), _t(gd), None, 1, 1, g, False, need=("dx",),
                                flags=cc.BACKWARD_MASK_BOTTOM_DIFF)
    assert_close(_np(dx), dx_ref * (x > 0), TOL_F32, "masked data gradient")


@pytest.mark.parametrize("case", QUAD_CASES)
def test_weight_gradient_dma_copies(case, overrides):
    """The quad-order GEMM with LDS-DMA copies (the default where the quad
    order applies) against the oracle, against the register-staged kernel to
    rounding (it sums each stage's columns in another order), and bit for bit
    from one run to the next; split-K ranges of one stage and of many."""
    N, C, H, W, K, kh, kw, sh, sw, ph, pw, g = case
    rng = np.random.default_rng([92, N, C, H, W, K])
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    w = (rng.standard_normal((K, C // g, kh, kw)) * 0.3).astype(np.float32)
    top = np.maximum(rng.standard_normal((N, K, (H + 2 * ph - kh) // sh + 1,
                                          (W + 2 * pw - kw) // sw + 1)), 0).astype(np.float32)
    gd = rng.standard_normal(top.shape).astype(np.float32)
    _, dw_ref, db_ref = oracle.conv_backward(x, w, gd, top=top, stride=(sh, sw), pad=(ph, pw),
                                             group=g, relu=True, need=("dw", "db"))
    args = (_t(x), _t(w), _t(gd), _t(top), (sh, sw), (ph, pw), g, True)
    for blocks in ("2048", "16"):
        overrides.setenv("CAFFE_CONV_WGRAD_BLOCKS", blocks)
        overrides.setenv("CAFFE_CONV_WGRAD_DMA", "1")
        _, dw, db = cc.conv_backward(*args, need=("dw", "db"))
        _, dw2, db2 = cc.conv_backward(*args, need=("dw", "db"))
        overrides.setenv("CAFFE_CONV_WGRAD_DMA", "0")
        _, dw0, db0 = cc.conv_backward(*args, need=("dw", "db"))
        torch.cuda.synchronize()
        assert_close(_np(dw), dw_ref, TOL_F32, f"weight gradient ({blocks} blocks)")
        assert_close(_np(db), db_ref, TOL_F32, f"bias gradient ({blocks} blocks)")
        assert torch.equal(dw, dw2) and torch.equal(db, db2)
        assert_close(_np(dw), _np(dw0), 1e-5, "DMA vs register-staged copies")
