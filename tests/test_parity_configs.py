"""Parity at the full workload sizes, in the launch configuration the
benchmark times (the same descriptors, the same ConvStack chain).

* LeNet conv pair (N=64): every output is compared with the oracle.
* CaffeNet at N=256: the oracle recomputes sampled outputs -- whole images
  for the forward pass and the data gradient (each image is independent),
  whole filters for the weight gradient (each filter's gradient is a sum
  over the full batch), every bias gradient -- from the very tensors the GPU
  consumed (layer by layer on shared inputs).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1408_5093_amd as cc
from paper_1408_5093_amd import workloads as wl
from paper_1408_5093_amd.net import ConvStack
from helpers import TOL_F32, assert_close
from layer_check import check_layer_sampled

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _np(t):
    torch.cuda.synchronize()
    return t.detach().float().cpu().numpy()


def test_lenet_pair_full():
    inp = wl.lenet_pair(64)
    net = ConvStack(wl.LENET, 64, inp["W"], inp["b"], glue={0: [("pool", wl.LENET_POOL)]})
    x = torch.from_numpy(inp["x"]).to(DEV)
    g = torch.from_numpy(inp["top_diff"]).to(DEV)
    net.forward(x)
    net.backward(g)
    L1, L2 = wl.LENET
    x1 = inp["x"]
    top1 = _np(net.top[0])
    y1_ref = oracle.conv_forward(x1, inp["W"][0], inp["b"][0], 1, 0, 1, False)
    assert_close(top1, y1_ref, TOL_F32, "conv1 forward")
    pool = net.stages[0][0]
    x2 = _np(pool["y"])
    np.testing.assert_array_equal(x2, oracle.maxpool_forward(top1, 2, 2).astype(np.float32))
    y2_ref = oracle.conv_forward(x2, inp["W"][1], inp["b"][1], 1, 0, 1, False)
    assert_close(_np(net.top[1]), y2_ref, TOL_F32, "conv2 forward")
    dx2_ref, dw2_ref, db2_ref = oracle.conv_backward(x2, inp["W"][1], inp["top_diff"])
    assert_close(_np(net.dbottom[1]), dx2_ref, TOL_F32, "conv2 data gradient")
    assert_close(_np(net.dW[1]), dw2_ref, TOL_F32, "conv2 weight gradient")
    assert_close(_np(net.db[1]), db2_ref, TOL_F32, "conv2 bias gradient")
    g1 = _np(pool["dx"])
    assert_close(g1, oracle.maxpool_backward(top1, _np(net.dbottom[1]), 2, 2), TOL_F32,
                 "pool backward")
    dx1_ref, dw1_ref, db1_ref = oracle.conv_backward(x1, inp["W"][0], g1)
    assert_close(_np(net.dbottom[0]), dx1_ref, TOL_F32, "conv1 data gradient")
    assert_close(_np(net.dW[0]), dw1_ref, TOL_F32, "conv1 weight gradient")
    assert_close(_np(net.db[0]), db1_ref, TOL_F32, "conv1 bias gradient")


def test_caffenet_conv1_forward_full_size():
    inp = wl.caffenet_conv1_fwd(256)
    L = wl.CAFFENET[0]
    y = cc.conv_forward(torch.from_numpy(inp["x"]).to(DEV), torch.from_numpy(inp["W"]).to(DEV),
                        torch.from_numpy(inp["b"]).to(DEV), L.s, L.p, L.g, L.relu)
    check_layer_sampled(L, inp["x"], inp["W"], inp["b"], _np(y), None, None, None, None,
                        images=[0, 131, 255], filters=[], what="conv1")


@pytest.mark.parametrize("l", [1, 2, 3, 4])
def test_caffenet_conv25_forward_full_size(l):
    inp = wl.caffenet_conv25_layer(l, 256)
    L = wl.CAFFENET[l]
    y = cc.conv_forward(torch.from_numpy(inp["x"]).to(DEV), torch.from_numpy(inp["W"]).to(DEV),
                        torch.from_numpy(inp["b"]).to(DEV), L.s, L.p, L.g, L.relu)
    check_layer_sampled(L, inp["x"], inp["W"], inp["b"], _np(y), None, None, None, None,
                        images=[0, 77, 255], filters=[], what=L.name)


def caffenet_glue():
    return {0: [("pool", wl.CAFFENET_POOL), ("lrn", wl.CAFFENET_LRN)],
            1: [("pool", wl.CAFFENET_POOL), ("lrn", wl.CAFFENET_LRN)]}


def test_caffenet_training_step_full_size():
    N = 256
    inp = wl.caffenet_step(N)
    net = ConvStack(wl.CAFFENET, N, inp["W"], inp["b"], glue=caffenet_glue())
    _run_and_check_step(net, wl.CAFFENET, inp, images=[0, 255])


def test_caffenet_network_step_full_size():
    """conv1-5, pool5 and the fc6-fc8 inner products at N=256: every layer
    and glue stage on the tensors the GPU consumed, sampled as above."""
    N = 256
    inp = wl.caffenet_net_step(N)
    net = ConvStack(wl.CAFFENET_NET, N, inp["W"], inp["b"], glue=wl.CAFFENET_NET_GLUE)
    _run_and_check_step(net, wl.CAFFENET_NET, inp, images=[0, 200])


def _tile_filters(L):
    """One filter in every 64 rows of every group (the weight-gradient row
    tiles are 64, 96 or 128 rows) and each group's last filter."""
    Kg = L.K // L.g
    if L.H == 1 and L.W == 1:  # inner products: first and last
        return [0, L.K - 1]
    return sorted({t * Kg + m for t in range(L.g) for m in list(range(0, Kg, 64)) + [Kg - 1]})


def _run_and_check_step(net, layers, inp, images):
    x = torch.from_numpy(inp["x"]).to(DEV)
    g = torch.from_numpy(inp["top_diff"]).to(DEV)
    net.forward(x)
    net.backward(g)
    torch.cuda.synchronize()
    for l, L in enumerate(layers):
        xl = _np(net.bottom[l])
        gl = _np(net.layer_top_diff(l, g))
        check_layer_sampled(L, xl, inp["W"][l], inp["b"][l], _np(net.top[l]), gl,
                            _np(net.dbottom[l]), _np(net.dW[l]), _np(net.db[l]), images=images,
                            filters=_tile_filters(L), what=f"step {L.name}",
                            dx_mask=(xl > 0) if net.mask_bottom[l] else None)
        for st in net.stages[l]:
            xin = _np(st["x"])[images]
            p = st["prm"]
            if st["kind"] == "pool":
                ref = oracle.maxpool_forward(xin, p["kernel"], p["stride"])
                np.testing.assert_array_equal(_np(st["y"])[images], ref.astype(np.float32))
                if net.fused[l]:
                    # pool + LRN backward in one pass: the pooled gradient is
                    # the LRN backward of what the LRN received
                    lst = net.stages[l][1]
                    r = lst["prm"]
                    dy = oracle.lrn_backward(_np(lst["x"])[images],
                                             _np(_glue_dy(net, l, lst))[images], r["size"],
                                             r["alpha"], r["beta"], r["k"])
                else:
                    dy = _np(_glue_dy(net, l, st))[images]
                gref = oracle.maxpool_backward(xin, dy, p["kernel"], p["stride"])
                if net.pool_flags[l] and st is net.stages[l][0]:
                    gref = gref * (xin > 0)  # the fused backward of conv's ReLU
            elif net.fused[l]:
                ref = oracle.lrn_forward(xin, p["size"], p["alpha"], p["beta"], p["k"])
                assert_close(_np(st["y"])[images], ref, TOL_F32, f"{L.name} LRN forward")
                continue  # no separate LRN gradient
            else:
                ref = oracle.lrn_forward(xin, p["size"], p["alpha"], p["beta"], p["k"])
                assert_close(_np(st["y"])[images], ref, TOL_F32, f"{L.name} LRN forward")
                gref = oracle.lrn_backward(xin, _np(_glue_dy(net, l, st))[images], p["size"],
                                           p["alpha"], p["beta"], p["k"])
            assert_close(_np(st["dx"])[images], gref, TOL_F32, f"{L.name} {st['kind']} backward")


def _glue_dy(net, l, st):
    """Gradient the glue stage st (after layer l) received in the backward sweep."""
    stages = net.stages[l]
    i = next(j for j, s in enumerate(stages) if s is st)
    if i + 1 < len(stages):
        return stages[i + 1]["dx"]
    return net.dbottom[l + 1].view(st["y"].shape)


def test_caffenet_step_side_stream_matches_one_stream():
    """The fp32 backward with the weight gradients on a side stream gives the
    single-stream results bit for bit (same kernels, same inputs), over three
    steps in a row."""
    N = 8
    inp = wl.caffenet_step(N)
    x = torch.from_numpy(inp["x"]).to(DEV)
    g = torch.from_numpy(inp["top_diff"]).to(DEV)
    nets = [ConvStack(wl.CAFFENET, N, inp["W"], inp["b"], glue=caffenet_glue(),
                      split_backward=split) for split in (True, False)]
    for _ in range(3):
        for net in nets:
            net.forward(x)
            net.backward(g)
        torch.cuda.synchronize()
        a, b = nets
        for l in range(len(wl.CAFFENET)):
            assert torch.equal(a.top[l], b.top[l])
            assert torch.equal(a.dW[l], b.dW[l]) and torch.equal(a.db[l], b.db[l])
            assert torch.equal(a.dbottom[l], b.dbottom[l])


def test_caffenet_step_byte_masks_match():
    """The fp32 step with the fused max-pools recording their winners as
    bytes (the default: the fused glue backward reads them) against 32-bit
    plane-index masks: every top and gradient the same bits."""
    N = 32
    inp = wl.caffenet_step(N, wl.CAFFENET_STEP)
    x = torch.from_numpy(inp["x"]).to(DEV)
    g = torch.from_numpy(inp["top_diff"]).to(DEV)
    nets = [ConvStack(wl.CAFFENET, N, inp["W"], inp["b"], glue=caffenet_glue(),
                      mask_offsets=f) for f in (True, False)]
    assert nets[0].mask_u8 == [True, True, False, False, False]
    assert nets[0].stages[0][0]["mask"].dtype == torch.uint8
    assert not any(nets[1].mask_u8)
    for net in nets:
        net.forward(x)
        net.backward(g)
    torch.cuda.synchronize()
    a, b = nets
    for l in range(len(wl.CAFFENET)):
        assert torch.equal(a.top[l], b.top[l]), f"layer {l} top"
        assert torch.equal(a.dbottom[l], b.dbottom[l]), f"layer {l} data gradient"
        assert torch.equal(a.dW[l], b.dW[l]), f"layer {l} weight gradient"
        assert torch.equal(a.db[l], b.db[l]), f"layer {l} bias gradient"
