"""GPU parity of the bf16-operand convolution (bf16 bottom and weights, fp32
accumulation and results) against the CPU oracle, through the C ABI.

Two bars per output tensor, max|gpu - ref| / max|ref|:
* 1e-4 against the oracle fed the very values the GPU multiplied -- the
  bf16-rounded bottom and weights and, for the gradients, the bf16-rounded
  (masked) top gradient.  Products of bf16 values are exact in fp32, so only
  the order of the fp32 sums differs from the oracle's fp64 sums.
* 2e-2 against the oracle on the unrounded fp32 operands: the tolerance the
  bf16 variant is held to.
The bias gradient sums the unrounded fp32 top gradient, so it is held to
1e-4 against the oracle on that gradient.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1408_5093_amd as cc
from paper_1408_5093_amd import workloads as wl
from paper_1408_5093_amd.net import ConvStack
from helpers import TOL_BF16, TOL_F32, assert_close
from layer_check import check_layer_sampled
from test_parity_conv import SWEEP

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _t(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(dtype)


def _np(t):
    torch.cuda.synchronize()
    return t.detach().float().cpu().numpy()


def run_case(N, C, H, W, K, kh, kw, sh, sw, ph, pw, g, relu, bias=True, seed=0, flags=0):
    print(f"bf16 case N={N} C={C} H={H} W={W} K={K} k={kh}x{kw} s={sh},{sw} p={ph},{pw} g={g} "
          f"relu={relu} flags={flags}", flush=True)
    rng = np.random.default_rng([78, seed, N, C, H, W, K, kh, kw, sh, sw, ph, pw, g, int(relu)])
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    if flags & cc.BACKWARD_MASK_BOTTOM_DIFF:
        x = np.maximum(x, 0)  # a ReLU output
    w = (rng.standard_normal((K, C // g, kh, kw)) * 0.3).astype(np.float32)
    b = (rng.standard_normal(K) * 0.5).astype(np.float32) if bias else None
    xr, wr = wl.round_bf16(x), wl.round_bf16(w)
    geom = dict(stride=(sh, sw), pad=(ph, pw), group=g)
    xb, wb = _t(xr, torch.bfloat16), _t(wr, torch.bfloat16)

    y = _np(cc.conv_forward(xb, wb, _t(b) if bias else None, (sh, sw), (ph, pw), g, relu))
    y_ref_r = oracle.conv_forward(xr, wr, b, (sh, sw), (ph, pw), g, relu)
    assert_close(y, y_ref_r, TOL_F32, "forward (rounded operands)")
    assert_close(y, oracle.conv_forward(x, w, b, (sh, sw), (ph, pw), g, relu), TOL_BF16,
                 "forward (fp32 operands)")

    top = y_ref_r.astype(np.float32)
    gd = rng.standard_normal(top.shape).astype(np.float32)
    masked_in = bool(flags & cc.BACKWARD_TOP_DIFF_MASKED)
    if masked_in and relu:
        gd = (gd * (top > 0)).astype(np.float32)
    gr = wl.round_bf16(gd)
    dx, dw, db = cc.conv_backward(xb, wb, _t(gd), None if masked_in else _t(top), (sh, sw),
                                  (ph, pw), g, relu, flags=flags)
    dx, dw, db = _np(dx), _np(dw), _np(db)
    keep = (xr > 0) if flags & cc.BACKWARD_MASK_BOTTOM_DIFF else 1.0
    dx_r, dw_r, _ = oracle.conv_backward(xr, wr, gr, top=top, relu=relu, need=("dx", "dw"), **geom)
    _, _, db_ref = oracle.conv_backward(xr, wr, gd, top=top, relu=relu, need=("db",), **geom)
    assert_close(dx, dx_r * keep, TOL_F32, "data gradient (rounded operands)")
    assert_close(dw, dw_r, TOL_F32, "weight gradient (rounded operands)")
    assert_close(db, db_ref, TOL_F32, "bias gradient")
    dx_f, dw_f, _ = oracle.conv_backward(x, w, gd, top=top, relu=relu, need=("dx", "dw"), **geom)
    assert_close(dx, dx_f * keep, TOL_BF16, "data gradient (fp32 operands)")
    assert_close(dw, dw_f, TOL_BF16, "weight gradient (fp32 operands)")


@pytest.mark.parametrize("case", SWEEP)
@pytest.mark.parametrize("relu", [False, True])
def test_sweep_bf16(case, relu):
    run_case(*case, relu=relu, bias=(case[0] % 2 == 0) or relu)


def test_tile_shapes_each_chooser_branch_bf16():
    # forward rows Kg: 48-, 64-, 96-, 128-row tiles and several row tiles;
    # data-gradient rows Cg * s^2 alike
    for K, g in [(20, 1), (50, 1), (96, 1), (128, 1), (384, 2), (300, 1)]:
        run_case(2, 2 * g, 9, 10, K, 3, 3, 1, 1, 1, 1, g, True)
    for C, s, k in [(3, 4, 11), (1, 2, 5), (5, 3, 7), (8, 4, 5), (40, 1, 3)]:
        run_case(2, C, 29, 31, 6, k, k, s, s, 1, 2, 1, True)


def test_narrow_channel_packing_bf16():
    # one group of at most 4 channels staged as Cgp = 1, 2 or 4 channels with
    # 8 / Cgp taps per 16-byte chunk when the horizontal stride allows it
    # (kernel widths that are not multiples of the taps per chunk, vertical
    # strides that differ from the horizontal one); 3 channels with an odd
    # horizontal stride keep 8-channel chunks
    for C, sh, sw, kh, kw in [(3, 4, 4, 11, 11), (4, 1, 2, 3, 3), (2, 3, 4, 5, 7),
                              (1, 2, 8, 4, 9), (3, 2, 1, 5, 5), (2, 1, 2, 1, 1)]:
        run_case(2, C, 23, 37, 10, kh, kw, sh, sw, 1, 2, 1, True)


def test_channel_padding_and_long_reductions_bf16():
    # channels per group that are not multiples of 8 (zero padding), and
    # channel counts spanning several 32-deep stages per tap
    for C, K, g in [(9, 10, 1), (18, 30, 3), (64, 72, 1), (200, 40, 2)]:
        run_case(2, C, 11, 12, K, 3, 3, 1, 1, 1, 1, g, True)


@pytest.mark.parametrize("flags", [1, 2, 3])
def test_backward_flags_bf16(flags):
    run_case(2, 8, 13, 13, 24, 3, 3, 1, 1, 1, 1, 2, True, flags=flags)


@pytest.mark.parametrize("case", [(2, 3, 29, 31, 16, 11, 11, 4, 4, 0, 0, 1, True),
                                  (2, 8, 13, 13, 24, 3, 3, 1, 1, 1, 1, 2, True),
                                  (3, 20, 9, 10, 30, 5, 5, 1, 1, 2, 2, 1, False)])
def test_backward_reuses_forward_staging_bf16(case):
    """BACKWARD_BOTTOM_STAGED: a backward on the workspace the forward
    staged its input into gives bitwise the gradients of a plain backward on
    a fresh workspace (the same kernels in the same order read the same
    staged copy); in fp32 mode the flag changes nothing."""
    N, C, H, W, K, kh, kw, sh, sw, ph, pw, g, relu = case
    print(f"staged bottom case {case}", flush=True)
    rng = np.random.default_rng([79, N, C, K, kh])
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    w = (rng.standard_normal((K, C // g, kh, kw)) * 0.3).astype(np.float32)
    b = (rng.standard_normal(K) * 0.5).astype(np.float32)
    for op in (torch.bfloat16, torch.float32):
        dt = cc.CAFFE_BF16 if op == torch.bfloat16 else cc.CAFFE_F32
        d = cc.conv_desc(x.shape, w.shape, (sh, sw), (ph, pw), g, relu, dt)
        Ho, Wo = cc.conv_out_shape(d)
        xb, wb, bt = _t(x, op), _t(w, op), _t(b)
        gd = _t(rng.standard_normal((N, K, Ho, Wo)))
        need = max(cc.conv_workspace_size(d, cc.PASS_FORWARD),
                   cc.conv_workspace_size(d, cc.PASS_BACKWARD))
        buf = cc.Workspace(DEV).get(need)
        top = torch.empty((N, K, Ho, Wo), dtype=torch.float32, device=DEV)
        cc.caffe_conv_forward(d, xb, wb, bt, top, buf)
        ref = cc.conv_backward(xb, wb, gd, top if relu else None, (sh, sw), (ph, pw), g, relu)
        outs = tuple(torch.empty_like(t) for t in ref)
        cc.caffe_conv_backward(d, gd, top if relu else None, xb, wb, *outs, 0,
                               cc.BACKWARD_BOTTOM_STAGED, buf)
        torch.cuda.synchronize()
        for name, u, v in zip(("dx", "dw", "db"), outs, ref):
            assert torch.equal(u, v), (op, name)


def test_empty_batch_bf16():
    x = torch.empty((0, 4, 9, 9), device=DEV, dtype=torch.bfloat16)
    w = torch.randn((6, 2, 3, 3), device=DEV).to(torch.bfloat16)
    y = cc.conv_forward(x, w, torch.zeros(6, device=DEV), 1, 1, 2, True)
    assert y.shape == (0, 6, 9, 9)
    g = torch.empty(y.shape, device=DEV)
    dx, dw, db = cc.conv_backward(x, w, g, y, 1, 1, 2, True)
    torch.cuda.synchronize()
    assert dx.shape == x.shape
    assert torch.all(dw == 0) and torch.all(db == 0)


def test_accumulate_bf16():
    rng = np.random.default_rng(6)
    x = wl.round_bf16(rng.standard_normal((2, 4, 11, 11)).astype(np.float32))
    w = wl.round_bf16(rng.standard_normal((8, 4, 3, 3)).astype(np.float32))
    g = rng.standard_normal((2, 8, 11, 11)).astype(np.float32)
    _, dw_ref, _ = oracle.conv_backward(x, w, wl.round_bf16(g), stride=1, pad=1, need=("dw",))
    _, _, db_ref = oracle.conv_backward(x, w, g, stride=1, pad=1, need=("db",))
    dw0 = rng.standard_normal(w.shape).astype(np.float32)
    db0 = rng.standard_normal(8).astype(np.float32)
    dwt, dbt = _t(dw0), _t(db0)
    cc.conv_backward(_t(x, torch.bfloat16), _t(w, torch.bfloat16), _t(g), None, 1, 1, 1, False,
                     need=("dw", "db"), accumulate=1, outs=(None, dwt, dbt))
    assert_close(_np(dwt), dw_ref + dw0, TOL_F32, "accumulated dW")
    assert_close(_np(dbt), db_ref + db0, TOL_F32, "accumulated db")


def test_bitwise_determinism_bf16():
    rng = np.random.default_rng(12)
    x = _t(rng.standard_normal((4, 16, 27, 27)), torch.bfloat16)
    w = _t(rng.standard_normal((32, 8, 5, 5)) * 0.1, torch.bfloat16)
    b = _t(rng.standard_normal(32))
    outs = []
    for _ in range(2):
        y = cc.conv_forward(x, w, b, 1, 2, 2, True)
        g = torch.ones_like(y) * 0.5
        outs.append((y,) + cc.conv_backward(x, w, g, y, 1, 2, 2, True))
    torch.cuda.synchronize()
    for a, b_ in zip(*outs):
        assert torch.equal(a, b_)


def test_no_writes_outside_outputs_bf16():
    rng = np.random.default_rng(14)
    N, C, H, W, K = 3, 6, 14, 15, 20
    x = _t(rng.standard_normal((N, C, H, W)), torch.bfloat16)
    w = _t(rng.standard_normal((K, C // 2, 3, 3)), torch.bfloat16)
    band, canary = 4096, -12345.0

    def guarded(n):
        buf = torch.full((band + n + band,), canary, device=DEV)
        return buf, buf[band:band + n]

    ybuf, yv = guarded(N * K * H * W)
    y = yv.view(N, K, H, W)
    d = cc.conv_desc(x.shape, w.shape, 1, 1, 2, True, cc.CAFFE_BF16)
    cc.caffe_conv_forward(d, x, w, None, y, cc.Workspace().get(
        cc.conv_workspace_size(d, cc.PASS_FORWARD)))
    dxbuf, dxv = guarded(x.numel())
    dwbuf, dwv = guarded(w.numel())
    dbbuf, dbv = guarded(K)
    g = _t(rng.standard_normal((N, K, H, W)))
    cc.conv_backward(x, w, g, y, 1, 1, 2, True, outs=(dxv.view(x.shape), dwv.view(w.shape), dbv))
    torch.cuda.synchronize()
    for buf in (ybuf, dxbuf, dwbuf, dbbuf):
        assert torch.all(buf[:band] == canary) and torch.all(buf[-band:] == canary)


def caffenet_glue():
    return {0: [("pool", wl.CAFFENET_POOL), ("lrn", wl.CAFFENET_LRN)],
            1: [("pool", wl.CAFFENET_POOL), ("lrn", wl.CAFFENET_LRN)]}


def test_caffenet_bf16_training_step_full_size():
    """The CaffeNet conv1-5 step at N=512 with bf16 operands, layer by layer
    on the tensors the GPU consumed (sampled images and filters)."""
    N = 512
    inp = wl.caffenet_step(N, wl.CAFFENET_STEP_BF16)
    # (unfused staging: the glue's float gradient is stored, so the check can
    # read each layer's top gradient; the fused step is compared with this one
    # in test_caffenet_bf16_step_fused_staging_matches)
    net = ConvStack(wl.CAFFENET, N, inp["W"], inp["b"], glue=caffenet_glue(), bf16=True,
                    fuse_staging=False, chain_staging=False)
    x = torch.from_numpy(inp["x"]).to(DEV)
    g = torch.from_numpy(inp["top_diff"]).to(DEV)
    net.forward(x)
    net.backward(g)
    torch.cuda.synchronize()
    images = [0, N - 1]
    for l, L in enumerate(wl.CAFFENET):
        xl = _np(net.bottom[l])          # the fp32 input
        xr = wl.round_bf16(xl)           # the bf16 operand the layer multiplies
        wr = _np(net.W[l])
        gl = _np(net.layer_top_diff(l, g))
        top = _np(net.top[l])
        dx, dw, db = _np(net.dbottom[l]), _np(net.dW[l]), _np(net.db[l])
        mask = (xr > 0) if net.mask_bottom[l] else None
        check_layer_sampled(L, xr, wr, inp["b"][l], top, wl.round_bf16(gl), dx, dw, db,
                            images=images, filters=[0, L.K - 1], what=f"bf16 step {L.name}",
                            dx_mask=mask, db_top_diff=gl)
        check_layer_sampled(L, xl, inp["W"][l], inp["b"][l], top, gl, dx, dw, db,
                            images=images, filters=[L.K // 2], tol=TOL_BF16,
                            what=f"bf16 step {L.name} vs fp32 operands",
                            dx_mask=(xl > 0) if net.mask_bottom[l] else None)


def test_backward_side_stream_fork_bf16(overrides):
    """A combined bf16 backward runs its weight gradient on the library's
    second stream: bitwise the gradients of the one-stream order, on the
    caller's stream once the call returns (three calls in a row)."""
    rng = np.random.default_rng(83)
    N, C, H, W, K, g = 3, 16, 11, 12, 40, 2
    x = _t(rng.standard_normal((N, C, H, W)), torch.bfloat16)
    w = _t(rng.standard_normal((K, C // g, 3, 3)) * 0.3, torch.bfloat16)
    y = cc.conv_forward(x, w, _t(rng.standard_normal(K)), 1, 1, g, True)
    gds = [_t(rng.standard_normal(y.shape)) for _ in range(3)]
    out = {}
    for fork in ("1", "0"):
        overrides.setenv("CAFFE_BACKWARD_FORK", fork)
        out[fork] = [cc.conv_backward(x, w, gd, y, 1, 1, g, True) for gd in gds]
    torch.cuda.synchronize()
    for a, b in zip(out["1"], out["0"]):
        for u, v in zip(a, b):
            assert torch.equal(u, v)


@pytest.mark.parametrize("bf16", [True, False])
def test_backward_weight_stream(bf16):
    """caffe_conv_backward_ex: the weight and bias gradients ordered on a
    second stream of the caller's, not joined -- bitwise the gradients of
    caffe_conv_backward, over three calls in a row on one workspace with the
    streams joined only at the end."""
    rng = np.random.default_rng(89)
    N, C, H, W, K, g = 3, 16, 11, 12, 40, 2
    op = torch.bfloat16 if bf16 else torch.float32
    x = _t(rng.standard_normal((N, C, H, W)), op)
    w = _t(rng.standard_normal((K, C // g, 3, 3)) * 0.3, op)
    y = cc.conv_forward(x, w, _t(rng.standard_normal(K)), 1, 1, g, True)
    d = cc.conv_desc(x.shape, w.shape, 1, 1, g, True, cc.CAFFE_BF16 if bf16 else cc.CAFFE_F32)
    gds = [_t(rng.standard_normal(y.shape)) for _ in range(3)]
    ws = cc.Workspace().get(cc.conv_workspace_size(d, cc.PASS_BACKWARD))
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    outs = {}
    for mode in ("one", "two"):
        res = []
        for gd in gds:
            dx = torch.empty(x.shape, device=DEV)
            dw = torch.empty(w.shape, device=DEV)
            db = torch.empty(K, device=DEV)
            if mode == "two":
                # (the workspace is reused: the previous call's weight side first)
                main.wait_stream(side)
            cc.caffe_conv_backward(d, gd, y, x, w, dx, dw, db, 0, 0, ws,
                                   weight_stream=side if mode == "two" else None)
            res.append((dx, dw, db))
        main.wait_stream(side)
        torch.cuda.synchronize()
        outs[mode] = res
    for a, b in zip(outs["one"], outs["two"]):
        for u, v in zip(a, b):
            assert torch.equal(u, v)


def test_caffenet_bf16_step_weight_stream_matches():
    """The bf16 step at N=512 with every layer's weight and bias gradients
    on the network's second stream (the default) against the one-stream step:
    every gradient bit for bit, over two steps."""
    N = 512
    inp = wl.caffenet_step(N, wl.CAFFENET_STEP_BF16)
    x = torch.from_numpy(inp["x"]).to(DEV)
    g = torch.from_numpy(inp["top_diff"]).to(DEV)
    nets = [ConvStack(wl.CAFFENET, N, inp["W"], inp["b"], glue=caffenet_glue(), bf16=True,
                      split_backward=f) for f in (True, False)]
    assert nets[0].weight_side and not nets[1].weight_side
    for _ in range(2):
        for net in nets:
            net.forward(x)
            net.backward(g)
        torch.cuda.synchronize()
        a, b = nets
        for l in range(len(wl.CAFFENET)):
            if not a.stage_into[l]:  # (a staged data gradient is not stored)
                assert torch.equal(a.dbottom[l], b.dbottom[l]), f"layer {l} data gradient"
            assert torch.equal(a.dW[l], b.dW[l]), f"layer {l} weight gradient"
            assert torch.equal(a.db[l], b.db[l]), f"layer {l} bias gradient"


def test_caffenet_bf16_step_fused_staging_matches():
    """The bf16 step at N=512 with conv1's and conv2's top gradients staged
    by the fused glue backward (the default) against the unfused step: every
    data and weight gradient bit for bit (the staged bf16 gradient is the
    same), every bias gradient within 1e-6, over two steps."""
    N = 512
    inp = wl.caffenet_step(N, wl.CAFFENET_STEP_BF16)
    x = torch.from_numpy(inp["x"]).to(DEV)
    g = torch.from_numpy(inp["top_diff"]).to(DEV)
    nets = [ConvStack(wl.CAFFENET, N, inp["W"], inp["b"], glue=caffenet_glue(), bf16=True,
                      fuse_staging=f) for f in (True, False)]
    assert nets[0].fuse_staging[:2] == [True, True] and not any(nets[1].fuse_staging)
    for _ in range(2):
        for net in nets:
            net.forward(x)
            net.backward(g)
        torch.cuda.synchronize()
        a, b = nets
        for l in range(len(wl.CAFFENET)):
            if not a.stage_into[l]:
                assert torch.equal(a.dbottom[l], b.dbottom[l]), f"layer {l} data gradient"
            assert torch.equal(a.dW[l], b.dW[l]), f"layer {l} weight gradient"
            assert_close(_np(a.db[l]), _np(b.db[l]), 1e-6, f"layer {l} bias gradient")


@pytest.mark.parametrize("dt", ["bf16", "f32_bottom"])
@pytest.mark.parametrize("ga", [1, 2])
def test_backward_into_layer_below(dt, ga):
    """caffe_conv_backward_into: layer B's data gradient (masked by B's bottom,
    the ReLU output of layer A) staged straight into A's top-gradient staging,
    then A's backward with CAFFE_BACKWARD_TOP_STAGED -- against B storing its
    float data gradient and A staging it: A's data and weight gradients bit
    for bit, A's bias gradient within 1e-6, B's weight and bias gradients
    bit for bit; twice, the second time into a workspace that held other
    values."""
    rng = np.random.default_rng([97, ga, dt == "bf16"])
    mode = cc.CAFFE_BF16 if dt == "bf16" else cc.CAFFE_BF16_F32_BOTTOM
    N, C, H, W, KA, KB = 2, 16, 10, 9, 128, 40
    x = _t(rng.standard_normal((N, C, H, W)), torch.bfloat16)
    wa = _t(rng.standard_normal((KA, C // ga, 3, 3)) * 0.2, torch.bfloat16)
    wb = _t(rng.standard_normal((KB, KA // 2, 3, 3)) * 0.2, torch.bfloat16)
    ba, bb = _t(rng.standard_normal(KA) * 0.1), _t(rng.standard_normal(KB) * 0.1)
    da = cc.conv_desc(x.shape, wa.shape, 1, 1, ga, True, cc.CAFFE_BF16)
    ya = torch.empty((N, KA, H, W), device=DEV)
    wsa0 = cc.Workspace(DEV).get(max(cc.conv_workspace_size(da, p) for p in range(4)))
    cc.caffe_conv_forward(da, x, wa, ba, ya, wsa0)
    xb = ya.to(torch.bfloat16) if mode == cc.CAFFE_BF16 else ya
    db_ = cc.conv_desc(xb.shape, wb.shape, 1, 1, 2, True, mode)
    assert cc.conv_stage_below_supported(db_, da)
    yb = torch.empty((N, KB, H, W), device=DEV)
    wsb = cc.Workspace(DEV).get(max(cc.conv_workspace_size(db_, p) for p in range(4)))
    cc.caffe_conv_forward(db_, xb, wb, bb, yb, wsb)
    gd = _t(rng.standard_normal(yb.shape))
    nA = cc.conv_workspace_size(da, cc.PASS_BACKWARD)
    out = {}
    for way in ("stored", "staged", "staged"):
        wsa = torch.full((nA,), 0x7F, dtype=torch.uint8, device=DEV)
        # A's forward staging of its bottom (what BACKWARD_BOTTOM_STAGED reads)
        cc.caffe_conv_forward(da, x, wa, ba, ya, wsa)
        dwb, dbb = torch.empty(wb.shape, device=DEV), torch.empty(KB, device=DEV)
        dxa, dwa, dba = (torch.empty(x.shape, device=DEV), torch.empty(wa.shape, device=DEV),
                         torch.empty(KA, device=DEV))
        fb = cc.BACKWARD_MASK_BOTTOM_DIFF
        fa = cc.BACKWARD_BOTTOM_STAGED
        if way == "stored":
            dxb = torch.empty(xb.shape, device=DEV, dtype=torch.float32)
            cc.caffe_conv_backward(db_, gd, yb, xb, wb, dxb, dwb, dbb, 0, fb, wsb)
            cc.caffe_conv_backward(da, dxb, ya, x, wa, dxa, dwa, dba, 0,
                                   fa | cc.BACKWARD_TOP_DIFF_MASKED, wsa)
        else:
            cc.caffe_conv_backward_into(db_, gd, yb, xb, wb, dwb, dbb, 0, fb, wsb, da, wsa)
            cc.caffe_conv_backward(da, None, ya, x, wa, dxa, dwa, dba, 0,
                                   fa | cc.BACKWARD_TOP_STAGED, wsa)
        torch.cuda.synchronize()
        out.setdefault(way, []).append((dxa, dwa, dba, dwb, dbb))
    ref = out["stored"][0]
    for got in out["staged"]:
        assert torch.equal(got[0], ref[0]), "A data gradient"
        assert torch.equal(got[1], ref[1]), "A weight gradient"
        assert_close(_np(got[2]), _np(ref[2]), 1e-6, "A bias gradient")
        assert torch.equal(got[3], ref[3]) and torch.equal(got[4], ref[4]), "B gradients"


def test_caffenet_bf16_step_chained_staging_matches():
    """The bf16 step at N=512 with conv5's and conv4's data gradients staged
    straight into conv4's and conv3's top-gradient staging (the default)
    against the step that stores and stages them: the stored data gradients,
    every weight gradient bit for bit (the staged bf16 values are the same),
    the bias gradients within 1e-6 (their partial sums are taken in another
    order), over two steps."""
    N = 512
    inp = wl.caffenet_step(N, wl.CAFFENET_STEP_BF16)
    x = torch.from_numpy(inp["x"]).to(DEV)
    g = torch.from_numpy(inp["top_diff"]).to(DEV)
    nets = [ConvStack(wl.CAFFENET, N, inp["W"], inp["b"], glue=caffenet_glue(), bf16=True,
                      chain_staging=f) for f in (True, False)]
    assert nets[0].stage_into == [False, False, False, True, True]
    assert not any(nets[1].stage_into)
    for _ in range(2):
        for net in nets:
            net.forward(x)
            net.backward(g)
        torch.cuda.synchronize()
        a, b = nets
        for l in range(len(wl.CAFFENET)):
            if not a.stage_into[l]:
                assert torch.equal(a.dbottom[l], b.dbottom[l]), f"layer {l} data gradient"
            assert torch.equal(a.dW[l], b.dW[l]), f"layer {l} weight gradient"
            assert_close(_np(a.db[l]), _np(b.db[l]), 1e-6, f"layer {l} bias gradient")


@pytest.mark.parametrize("case", [
    # N, C, H, W, pool k/s, LRN size, next K, kernel, pad, group
    (2, 32, 13, 13, 3, 2, 5, 24, 3, 1, 2),     # grouped, 16 channels a group, 6x6 image
    (3, 48, 24, 19, 3, 2, 3, 40, 5, 2, 1),     # LRN size 3, ragged pixel count
    (1, 96, 55, 55, 3, 2, 5, 64, 5, 2, 2),     # the conv1 -> conv2 geometry, one image
])
def test_lrn_forward_into_next_staging(case):
    """A max-pool + LRN whose output is staged as the next bf16 convolution's
    bottom (caffe_pool_lrn_forward_into), then that convolution run on the
    staged bottom (CAFFE_FORWARD_BOTTOM_STAGED) and its weight gradient on
    the same staging (CAFFE_BACKWARD_BOTTOM_STAGED): every output bit for
    bit against the separate passes, also with CAFFE_POOL_LRN_STAGE_ONLY (the
    LRN's float output then left untouched).  The staging workspace starts
    filled with large finite values, so a border the fused pass fails to
    zero shows up in the convolution's output."""
    N, C, H, W, pk, ps, size, K, kk, pad, g = case
    print(f"lrn staging case {case}", flush=True)
    rng = np.random.default_rng([91, *case])
    x = _t(np.maximum(rng.standard_normal((N, C, H, W)), 0))
    prm = (pk, ps, 0, size, 1e-4 * 50, 0.75, 1.0)
    Hp, Wp = cc.pool_out_shape(cc.pool_desc((N, C, H, W), pk, ps, 0))
    nd = cc.conv_desc((N, C, Hp, Wp), (K, C // g, kk, kk), 1, pad, g, True,
                      cc.CAFFE_BF16_F32_BOTTOM)
    assert cc.pool_lrn_stage_supported(x.shape, *prm, nd)
    w = _t(rng.standard_normal((K, C // g, kk, kk)) * 0.2, torch.bfloat16)
    b = _t(rng.standard_normal(K) * 0.3)
    ws_n = max(cc.conv_workspace_size(nd, cc.PASS_FORWARD),
               cc.conv_workspace_size(nd, cc.PASS_BACKWARD))
    ws = [torch.full((ws_n,), 0x7E, dtype=torch.uint8, device=DEV) for _ in range(2)]
    outs = []
    ws.append(torch.full((ws_n,), 0x7E, dtype=torch.uint8, device=DEV))
    for mode in (0, 1, 2):  # separate staging, staged by the LRN, staged only
        staged = mode > 0
        y0 = torch.full((N, C, Hp, Wp), float("nan"), device=DEV)
        pooled, mask, y = cc.pool_lrn_forward(x, *prm, out=y0,
                                              stage_for=(nd, ws[mode]) if staged else None,
                                              flags=cc.POOL_LRN_STAGE_ONLY if mode == 2 else 0)
        if mode == 2:
            assert torch.isnan(y).all(), "the float output was written"
            y = outs[0][2]  # (the float bottom is not read: the staging is)
        Ho, Wo = cc.conv_out_shape(nd)
        top = torch.empty((N, K, Ho, Wo), device=DEV)
        cc.caffe_conv_forward(nd, y, w, b, top, ws[mode],
                              flags=cc.FORWARD_BOTTOM_STAGED if staged else 0)
        gd = _t(np.random.default_rng(5).standard_normal(top.shape))
        dW, db = torch.empty(w.shape, device=DEV), torch.empty(K, device=DEV)
        cc.caffe_conv_backward(nd, gd, top, y, w, None, dW, db, flags=cc.BACKWARD_BOTTOM_STAGED,
                               workspace=ws[mode])
        torch.cuda.synchronize()
        outs.append((pooled, mask, y, top, dW, db))
    for other in outs[1:]:
        for name, a, c in zip(("pooled", "mask", "lrn", "top", "dW", "db"), outs[0], other):
            assert torch.equal(a, c), name
    assert torch.isfinite(outs[1][3]).all()


def test_caffenet_bf16_step_byte_masks_match():
    """The bf16 step at N=512 with the max-pools after conv1 and conv2
    recording their winners as bytes (the default where the fused backward
    reads them) against 32-bit plane-index masks: every top and gradient
    the same bits."""
    N = 512
    inp = wl.caffenet_step(N, wl.CAFFENET_STEP_BF16)
    x = torch.from_numpy(inp["x"]).to(DEV)
    g = torch.from_numpy(inp["top_diff"]).to(DEV)
    nets = [ConvStack(wl.CAFFENET, N, inp["W"], inp["b"], glue=caffenet_glue(), bf16=True,
                      mask_offsets=f) for f in (True, False)]
    assert nets[0].mask_u8 == [True, True, False, False, False]
    assert not any(nets[1].mask_u8)
    for net in nets:
        net.forward(x)
        net.backward(g)
    torch.cuda.synchronize()
    a, b = nets
    for l in range(len(wl.CAFFENET)):
        assert torch.equal(a.top[l], b.top[l]), f"layer {l} top"
        if not a.stage_into[l]:
            assert torch.equal(a.dbottom[l], b.dbottom[l]), f"layer {l} data gradient"
        assert torch.equal(a.dW[l], b.dW[l]), f"layer {l} weight gradient"
        assert torch.equal(a.db[l], b.db[l]), f"layer {l} bias gradient"


def test_caffenet_bf16_step_lrn_staging_matches():
    """The bf16 step at N=512 with the LRN after conv1 and conv2 staging conv2's
    and conv3's bf16 bottoms as it forms its output (the default) against the
    step whose convolutions stage their own bottoms: every top, data, weight
    and bias gradient bit for bit (the staged values are the same roundings of
    the same floats), over two steps."""
    N = 512
    inp = wl.caffenet_step(N, wl.CAFFENET_STEP_BF16)
    x = torch.from_numpy(inp["x"]).to(DEV)
    g = torch.from_numpy(inp["top_diff"]).to(DEV)
    nets = [ConvStack(wl.CAFFENET, N, inp["W"], inp["b"], glue=caffenet_glue(), bf16=True,
                      lrn_staging=f) for f in (True, False)]
    assert nets[0].bottom_staged == [False, True, True, False, False]
    assert not any(nets[1].bottom_staged)
    for _ in range(2):
        for net in nets:
            net.forward(x)
            net.backward(g)
        torch.cuda.synchronize()
        a, b = nets
        for l in range(len(wl.CAFFENET)):
            assert torch.equal(a.top[l], b.top[l]), f"layer {l} top"
            if not a.stage_into[l]:
                assert torch.equal(a.dbottom[l], b.dbottom[l]), f"layer {l} data gradient"
            assert torch.equal(a.dW[l], b.dW[l]), f"layer {l} weight gradient"
            assert torch.equal(a.db[l], b.db[l]), f"layer {l} bias gradient"


@pytest.mark.parametrize("case", [
    # N, C, H, W, K, k, pad, group, blocks (the split target; 0: the default)
    (4, 256, 13, 13, 128, 3, 1, 1, 0),     # one split: one unit, seven empty ones exit
    (48, 256, 13, 13, 256, 3, 1, 2, 72),   # 2 groups x 8 splits: two units per XCD
    (24, 256, 13, 11, 192, 3, 1, 2, 108),  # 96-row tiles, 2 groups x 6 splits, ragged
])
def test_wgrad_unit_order_bf16(case, overrides):
    """The bf16 weight gradient with each (group, split) unit's tiles on one
    XCD against the linear tile order at the same split count: the same
    partial sums in the same order, so the same bits; and the oracle on the
    rounded operands."""
    N, C, H, W, K, k, pad, g, blocks = case
    print(f"bf16 wgrad unit order {case}", flush=True)
    rng = np.random.default_rng([79, *case])
    xr = wl.round_bf16(rng.standard_normal((N, C, H, W)).astype(np.float32))
    wr = wl.round_bf16((rng.standard_normal((K, C // g, k, k)) * 0.2).astype(np.float32))
    gd = wl.round_bf16(rng.standard_normal((N, K, H + 2 * pad - k + 1,
                                            W + 2 * pad - k + 1)).astype(np.float32))
    xb, wb = _t(xr, torch.bfloat16), _t(wr, torch.bfloat16)
    if blocks:
        overrides.setenv("CAFFE_CONV_WGRAD_BLOCKS", str(blocks))
    dws = []
    for order in ("1", "0"):
        overrides.setenv("CAFFE_BF16_WGRAD_UNIT_ORDER", order)
        _, dw, _ = cc.conv_backward(xb, wb, _t(gd), None, 1, pad, g, need=("dw",))
        torch.cuda.synchronize()
        dws.append(dw)
    assert torch.equal(dws[0], dws[1])
    _, dw_ref, _ = oracle.conv_backward(xr, wr, gd, stride=1, pad=pad, group=g, need=("dw",))
    assert_close(_np(dws[0]), dw_ref, TOL_F32, "weight gradient (rounded operands)")


@pytest.mark.parametrize("blocked", ["0", "1"])
def test_dgrad_channel_blocked_bf16(blocked, overrides):
    """The data gradient with the reduction in 64-channel blocks outer, taps
    inner (the default where the top gradient's channels per group are a
    multiple of 64) and in the tap-major order: each against the oracle,
    with several channel blocks, 3x3 and 5x5 taps, groups and the masked
    bottom gradient."""
    overrides.setenv("CAFFE_BF16_DGRAD_BLOCKED", blocked)
    run_case(2, 32, 13, 11, 128, 3, 3, 1, 1, 1, 1, 1, True)        # 2 blocks, 9 taps
    run_case(2, 48, 11, 12, 256, 5, 5, 1, 1, 2, 2, 2, False)       # 2 groups x 2 blocks
    run_case(3, 16, 9, 9, 192, 3, 3, 1, 1, 1, 1, 1, True, flags=cc.BACKWARD_MASK_BOTTOM_DIFF)


@pytest.mark.parametrize("tile", range(4))
def test_forced_gemm_tiles_bf16(tile, overrides):
    """Every bf16 GEMM tile, forced for the forward and the data gradient,
    on row counts that leave a partial row tile and columns that leave a
    partial column tile (several tiles each way)."""
    overrides.setenv("CAFFE_BF16_FWD_TILE", str(tile))
    overrides.setenv("CAFFE_BF16_DGRAD_TILE", str(tile))
    run_case(3, 16, 14, 15, 200, 3, 3, 1, 1, 1, 1, 1, True)   # 200 rows, 630 columns
    run_case(2, 24, 21, 22, 36, 5, 5, 1, 1, 2, 2, 2, False)   # grouped, 5x5 taps
    run_case(2, 3, 45, 47, 40, 11, 11, 4, 4, 0, 0, 1, True)   # stride 4, 48 phase rows


@pytest.mark.parametrize("case", [
    (2, 3, 45, 47, 40, 11, 11, 4, 4, 0, 0, 1, True),   # 3 channels: narrow staging
    (2, 16, 14, 15, 64, 3, 3, 1, 1, 1, 1, 2, True),    # grouped, padded
    (3, 20, 9, 10, 30, 5, 5, 1, 1, 2, 2, 1, False),    # channels not a multiple of 8
])
def test_float_bottom_rounded_by_the_library(case):
    """CAFFE_BF16_F32_BOTTOM: a float bottom that the library rounds while
    staging gives bitwise what CAFFE_BF16 gives on the bottom rounded by
    torch (nearest-even): top, and every gradient with the bottom mask and
    with and without the forward's staged copy.  Some bottom values sit
    exactly half-way between two bf16 values and some round to +-0, so the
    rounding and the mask's sign rule are both exercised."""
    N, C, H, W, K, kh, kw, sh, sw, ph, pw, g, relu = case
    print(f"float bottom case {case}", flush=True)
    rng = np.random.default_rng([84, N, C, K, kh])
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    bits = x.view(np.uint32)
    bits[:, :, 0, :] = (bits[:, :, 0, :] & 0xFFFF0000) | 0x8000   # ties
    x[:, :, 1, :4] = np.array([1e-39, -1e-39, 2e-45, -2e-45], np.float32)  # to +-0 / denormals
    w = (rng.standard_normal((K, C // g, kh, kw)) * 0.3).astype(np.float32)
    b = (rng.standard_normal(K) * 0.5).astype(np.float32)
    xf = _t(x)
    xb = xf.to(torch.bfloat16)
    wb = _t(w, torch.bfloat16)
    bt = _t(b)
    outs = []
    for dt, xin in ((cc.CAFFE_BF16, xb), (cc.CAFFE_BF16_F32_BOTTOM, xf)):
        d = cc.conv_desc(x.shape, w.shape, (sh, sw), (ph, pw), g, relu, dt)
        Ho, Wo = cc.conv_out_shape(d)
        need = max(cc.conv_workspace_size(d, p) for p in range(4))
        buf = cc.Workspace(DEV).get(need)
        top = torch.empty((N, K, Ho, Wo), device=DEV)
        cc.caffe_conv_forward(d, xin, wb, bt, top, buf)
        gd = _t(np.random.default_rng(85).standard_normal((N, K, Ho, Wo)))
        res = [top.clone()]
        for flags in (cc.BACKWARD_MASK_BOTTOM_DIFF,
                      cc.BACKWARD_MASK_BOTTOM_DIFF | cc.BACKWARD_BOTTOM_STAGED):
            dx = torch.empty(x.shape, device=DEV)
            dw = torch.empty(w.shape, device=DEV)
            db = torch.empty(K, device=DEV)
            cc.caffe_conv_backward(d, gd, top if relu else None, xin, wb, dx, dw, db, 0, flags,
                                   buf)
            res += [dx, dw, db]
        torch.cuda.synchronize()
        outs.append(res)
    for a, c in zip(*outs):
        assert torch.equal(a, c)


@pytest.mark.parametrize("tile", range(2))
def test_forced_wgrad_tiles_bf16(tile, overrides):
    """Every bf16 weight-gradient tile, forced, on channel counts that leave
    partial row and column tiles (narrow packing included)."""
    overrides.setenv("CAFFE_BF16_WGRAD_TILE", str(tile))
    run_case(3, 16, 14, 15, 200, 3, 3, 1, 1, 1, 1, 1, True)   # 200 rows, 144 columns
    run_case(2, 24, 21, 22, 36, 5, 5, 1, 1, 2, 2, 2, False)   # grouped, 300 columns
    run_case(2, 3, 45, 47, 40, 11, 11, 4, 4, 0, 0, 1, True)   # narrow: 528 columns
