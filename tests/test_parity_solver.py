"""GPU parity of the softmax loss, the SGD update and whole LeNet training
iterations against the CPU oracle, through the C ABI.

Bar: max|gpu - oracle| / max|oracle| <= 1e-4 per output tensor (fp32).  The
training iterations are checked step by step on the tensors the GPU
consumed: each layer, the loss on the GPU's scores, and the update on the
GPU's pre-update weights, gradients and momentum histories (so a max-pool's
choice of winner is made on identical inputs on both sides).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1408_5093_amd as cc
from paper_1408_5093_amd import workloads as wl
from paper_1408_5093_amd.net import ConvStack, SGDTrainer
from helpers import TOL_F32, assert_close
from layer_check import check_layer_sampled

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _t(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV, dtype)


def _np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("N,K", [(1, 1), (3, 10), (64, 10), (5, 130), (100, 3), (256, 1000),
                                 (2, 4097), (300, 64)])
def test_softmax_loss(N, K):
    print(f"softmax loss N={N} K={K}", flush=True)
    rng = np.random.default_rng([90, N, K])
    z = (rng.standard_normal((N, K)) * 4).astype(np.float32)
    y = rng.integers(0, K, N).astype(np.int32)
    for lw in (1.0, 0.37):
        loss, sample, prob, diff = cc.softmax_loss(_t(z), _t(y, torch.int32), loss_weight=lw,
                                                   prob=True)
        l_ref, s_ref, p_ref, d_ref = oracle.softmax_loss(z, y, lw)
        assert_close(_np(loss), [l_ref], TOL_F32, "loss")
        assert_close(_np(sample), s_ref, TOL_F32, "per-sample loss")
        assert_close(_np(prob), p_ref, TOL_F32, "probabilities")
        assert_close(_np(diff), d_ref, TOL_F32, "score gradient")


def test_softmax_loss_scores_blob_and_large_scores():
    # an N x K x 1 x 1 blob, scores around 1e3 (the maximum is subtracted)
    rng = np.random.default_rng(91)
    z = (rng.standard_normal((16, 10, 1, 1)) * 3 + 1000).astype(np.float32)
    y = rng.integers(0, 10, 16).astype(np.int32)
    loss, sample, _, diff = cc.softmax_loss(_t(z), _t(y, torch.int32))
    l_ref, s_ref, _, d_ref = oracle.softmax_loss(z, y)
    assert np.isfinite(_np(loss)).all()
    assert_close(_np(loss), [l_ref], TOL_F32, "loss")
    assert_close(_np(diff).reshape(16, 10), d_ref, TOL_F32, "score gradient")


def test_softmax_loss_empty_batch_and_bad_label():
    loss, sample, _, _ = cc.softmax_loss(torch.empty((0, 10), device=DEV),
                                         torch.empty(0, dtype=torch.int32, device=DEV))
    assert _np(loss)[0] == 0.0
    z = torch.zeros((4, 10), device=DEV)
    y = torch.tensor([0, 1, 10, 3], dtype=torch.int32, device=DEV)  # 10 is out of range
    loss, sample, _, diff = cc.softmax_loss(z, y)
    s = _np(sample)
    assert np.isnan(_np(loss)[0]) and np.isnan(s[2]) and np.isfinite(s[[0, 1, 3]]).all()
    # the bad sample's gradient row has no -1 term: p / N = 0.1 / 4
    np.testing.assert_allclose(_np(diff)[2], np.full(10, 0.025), rtol=1e-6)


def test_softmax_loss_bitwise_determinism():
    rng = np.random.default_rng(92)
    z = _t(rng.standard_normal((512, 1000)))
    y = _t(rng.integers(0, 1000, 512), torch.int32)
    a = cc.softmax_loss(z, y, prob=True)
    b = cc.softmax_loss(z, y, prob=True)
    torch.cuda.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u, v)


@pytest.mark.parametrize("count", [1, 3, 4, 7, 1001, 4096, (1 << 20) + 3])
def test_sgd_update(count):
    rng = np.random.default_rng([93, count])
    w = rng.standard_normal(count).astype(np.float32)
    g = rng.standard_normal(count).astype(np.float32)
    v = (rng.standard_normal(count) * 0.1).astype(np.float32)
    for lr, mom, wd in [(0.01, 0.9, 5e-4), (0.1, 0.0, 0.0), (0.05, 0.5, 0.0)]:
        wt, gt, vt = _t(w), _t(g), _t(v)
        cc.sgd_update(wt, gt, vt, lr, mom, wd)
        w_ref, v_ref = oracle.sgd_step(w, g, v, lr, mom, wd)
        assert_close(_np(wt), w_ref, TOL_F32, "weights")
        assert_close(_np(vt), v_ref, TOL_F32, "momentum history")
        assert_close(_np(gt), g, 0.0, "gradient untouched")


def _lenet_trainer(N=64, batches=3):
    inp = wl.lenet_train(N, batches)
    net = ConvStack(wl.LENET_NET, N, inp["W"], inp["b"], glue=wl.LENET_NET_GLUE)
    sol = {k: v for k, v in wl.LENET_SOLVER.items()}
    mom, wd = sol.pop("momentum"), sol.pop("weight_decay")
    return inp, net, SGDTrainer(net, momentum=mom, weight_decay=wd, **sol)


def test_lenet_training_iterations():
    """Three LeNet iterations at N=64 (three batches), each checked step by
    step against the oracle on the GPU's own tensors."""
    N = 64
    inp, net, tr = _lenet_trainer(N, 3)
    images = [0, 17, N - 1]
    for it in range(3):
        print(f"lenet iteration {it}", flush=True)
        x = _t(inp["x"][it])
        y = _t(inp["labels"][it], torch.int32)
        W0 = [_np(w) for w in net.W]
        b0 = [_np(b) for b in net.b]
        vW0 = [_np(v) for v in tr.vW]
        vb0 = [_np(v) for v in tr.vb]
        loss = tr.forward_backward(x, y)
        # the loss on the GPU's scores
        scores = _np(net.top[-1])
        l_ref, _, _, d_ref = oracle.softmax_loss(scores, inp["labels"][it])
        assert_close(_np(loss), [l_ref], TOL_F32, f"iteration {it} loss")
        assert_close(_np(tr.scores_diff).reshape(N, -1), d_ref, TOL_F32, f"iteration {it} dz")
        # every layer on its own inputs
        for l, L in enumerate(wl.LENET_NET):
            xl = _np(net.bottom[l])
            gl = _np(net.layer_top_diff(l, tr.scores_diff))
            dx = _np(net.dbottom[l]) if l > 0 else None
            check_layer_sampled(L, xl, W0[l], b0[l], _np(net.top[l]), gl, dx, _np(net.dW[l]),
                                _np(net.db[l]), images=images, filters=list(range(L.K))[:3],
                                what=f"iteration {it} {L.name}",
                                dx_mask=(xl > 0) if net.mask_bottom[l] else None)
        for l in range(len(wl.LENET_NET)):
            for st in net.stages[l]:  # one max-pool after each conv
                xin = _np(st["x"])
                np.testing.assert_array_equal(_np(st["y"]), oracle.maxpool_forward(xin, 2, 2))
                dy = _np(net.dbottom[l + 1].view(st["y"].shape))
                assert_close(_np(st["dx"]), oracle.maxpool_backward(xin, dy, 2, 2), TOL_F32,
                             f"iteration {it} pool {l} backward")
        # the update on the GPU's pre-update state and gradients
        dW = [_np(w) for w in net.dW]
        db = [_np(b) for b in net.db]
        lr = tr.update()
        lr_ref = oracle.learning_rate("inv", np.float32(0.01), it, gamma=np.float32(1e-4),
                                      power=np.float32(0.75))
        assert abs(lr - lr_ref) <= 1e-6 * lr_ref
        for l in range(len(wl.LENET_NET)):
            w_ref, v_ref = oracle.sgd_step(W0[l], dW[l], vW0[l], lr, 0.9, 5e-4)
            assert_close(_np(net.W[l]), w_ref, TOL_F32, f"iteration {it} W{l}")
            assert_close(_np(tr.vW[l]), v_ref, TOL_F32, f"iteration {it} vW{l}")
            b_ref, vb_ref = oracle.sgd_step(b0[l], db[l], vb0[l], lr, 0.9, 5e-4)
            assert_close(_np(net.b[l]), b_ref, TOL_F32, f"iteration {it} b{l}")
            assert_close(_np(tr.vb[l]), vb_ref, TOL_F32, f"iteration {it} vb{l}")


def test_lenet_training_fits_a_batch():
    """Repeated steps on one fixed batch drive its loss well below its
    starting value (ln 10 for an untrained net)."""
    inp, net, tr = _lenet_trainer(64, 1)
    x = _t(inp["x"][0])
    y = _t(inp["labels"][0], torch.int32)
    losses = [float(_np(tr.step(x, y))[0]) for _ in range(60)]
    assert abs(losses[0] - np.log(10)) < 0.5
    assert losses[-1] < 0.5 * losses[0], losses[::10]


def test_lenet_training_graph_replays_match_eager():
    """The captured iteration, replayed with eager work and synchronizations
    between replays, gives bitwise the weights, histories and losses of the
    eager iterations from the same start (trainer state after every replay)."""
    N = 64
    inp, net_e, tr_e = _lenet_trainer(N, 3)
    _, net_g, tr_g = _lenet_trainer(N, 3)
    xs = [_t(a) for a in inp["x"]]
    ys = [_t(a, torch.int32) for a in inp["labels"]]
    xg, yg = xs[0].clone(), ys[0].clone()      # the graph's static batch buffers
    tr_g.capture(xg, yg)
    for it in range(3):
        print(f"graph replay {it}", flush=True)
        le = tr_e.step(xs[it], ys[it])
        xg.copy_(xs[it])
        yg.copy_(ys[it])
        lg = tr_g.replay()
        torch.cuda.synchronize()
        _ = torch.randn(1000, device=DEV).sum().item()   # eager work between replays
        assert torch.equal(le, lg), (le, lg)
        for a, b in zip(net_e.W + net_e.b + tr_e.vW + tr_e.vb,
                        net_g.W + net_g.b + tr_g.vW + tr_g.vb):
            assert torch.equal(a, b)
