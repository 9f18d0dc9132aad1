"""Pins for the max-pooling and LRN oracles (layer types listed in the
paper's Sec. 3.2): hand-worked examples, torch float64 CPU routines, and
finite differences."""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

RNG = np.random.default_rng(1408)


def test_worked_examples(golden_dir):
    data = json.load(open(os.path.join(golden_dir, "glue_worked_examples.json")))
    for c in data["maxpool"]:
        x = np.array(c["x"], float)
        y = oracle.maxpool_forward(x, c["k"], c["s"], c["p"])
        np.testing.assert_array_equal(y, np.array(c["y"], float), err_msg=c["name"])
        dx = oracle.maxpool_backward(x, np.array(c["top_diff"], float), c["k"], c["s"], c["p"])
        np.testing.assert_array_equal(dx, np.array(c["dx"], float), err_msg=c["name"])
    for c in data["lrn"]:
        x = np.array(c["x"], float)
        kw = dict(size=c["size"], alpha=c["alpha"], beta=c["beta"], k=c["k"])
        np.testing.assert_allclose(oracle.lrn_forward(x, **kw), np.array(c["y"]), rtol=1e-15)
        np.testing.assert_allclose(oracle.lrn_backward(x, np.array(c["top_diff"], float), **kw),
                                   np.array(c["dx"]), rtol=1e-14)


@pytest.mark.parametrize("shape,k,s", [((2, 3, 55, 55), 3, 2), ((2, 4, 24, 24), 2, 2),
                                       ((1, 2, 13, 11), 3, 2), ((1, 1, 9, 9), 3, 3)])
def test_maxpool_matches_torch(shape, k, s):
    x = RNG.standard_normal(shape)
    xt = torch.from_numpy(x).requires_grad_(True)
    yt = F.max_pool2d(xt, k, s)
    np.testing.assert_array_equal(oracle.maxpool_forward(x, k, s), yt.detach().numpy())
    g = RNG.standard_normal(yt.shape)
    yt.backward(torch.from_numpy(g))
    # continuous random inputs: no ties, so the routed gradient is unique
    np.testing.assert_allclose(oracle.maxpool_backward(x, g, k, s), xt.grad.numpy(), rtol=1e-14,
                               atol=1e-15)


@pytest.mark.parametrize("shape", [(2, 7, 5, 4), (1, 12, 3, 3), (2, 3, 2, 2)])
def test_lrn_matches_torch(shape):
    x = RNG.standard_normal(shape) * 3
    xt = torch.from_numpy(x).requires_grad_(True)
    yt = F.local_response_norm(xt, size=5, alpha=1e-2, beta=0.75, k=1.0)
    np.testing.assert_allclose(oracle.lrn_forward(x, 5, 1e-2, 0.75, 1.0), yt.detach().numpy(),
                               rtol=1e-13, atol=1e-14)
    g = RNG.standard_normal(shape)
    yt.backward(torch.from_numpy(g))
    np.testing.assert_allclose(oracle.lrn_backward(x, g, 5, 1e-2, 0.75, 1.0), xt.grad.numpy(),
                               rtol=1e-11, atol=1e-13)


def test_lrn_finite_difference():
    x = RNG.standard_normal((1, 8, 2, 3)) * 5
    g = RNG.standard_normal(x.shape)
    args = (5, 0.3, 0.75, 2.0)
    dx = oracle.lrn_backward(x, g, *args)
    h = 1e-6
    for idx in [(0, 0, 0, 0), (0, 3, 1, 2), (0, 7, 1, 1), (0, 5, 0, 2)]:
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        fd = (np.sum(oracle.lrn_forward(xp, *args) * g) - np.sum(oracle.lrn_forward(xm, *args) * g)) / (2 * h)
        np.testing.assert_allclose(fd, dx[idx], rtol=1e-6, atol=1e-8)


def test_maxpool_finite_difference():
    x = RNG.standard_normal((1, 2, 7, 7))
    g = RNG.standard_normal((1, 2, 3, 3))
    dx = oracle.maxpool_backward(x, g, 3, 2)
    h = 1e-7
    for idx in [(0, 0, 2, 2), (0, 1, 4, 3), (0, 0, 6, 6), (0, 1, 0, 1)]:
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        fd = (np.sum(oracle.maxpool_forward(xp, 3, 2) * g) - np.sum(oracle.maxpool_forward(xm, 3, 2) * g)) / (2 * h)
        np.testing.assert_allclose(fd, dx[idx], rtol=1e-6, atol=1e-8)
