"""Pins of the solver oracle (softmax loss, SGD step, learning-rate schedules)
against closed forms, hand-worked values, torch float64 CPU routines and
finite differences.  Each pin is also run against deliberately wrong
variants of the oracle (a dropped 1/N, a sign error, a missing term, ...),
which must fail it."""
import math

import numpy as np
import pytest
import torch

import oracle


# ------------------------------------------------------------ softmax loss
def pin_softmax_hand_example(fn):
    # two classes, scores (0, ln 3), label 1: p = (1/4, 3/4), loss = ln(4/3),
    # dz = (1/4, -1/4)
    loss, sample, p, dz = fn(np.array([[0.0, math.log(3.0)]]), np.array([1]))
    assert abs(loss - math.log(4.0 / 3.0)) < 1e-14
    np.testing.assert_allclose(p, [[0.25, 0.75]], rtol=0, atol=1e-15)
    np.testing.assert_allclose(dz, [[0.25, -0.25]], rtol=0, atol=1e-15)
    np.testing.assert_allclose(sample, [math.log(4.0 / 3.0)], rtol=1e-14)


def pin_softmax_uniform_scores(fn):
    # equal scores: loss = ln K for every label; dz = (1/K - [k == y]) / N
    N, K = 5, 7
    z = np.full((N, K), 3.25)
    y = np.array([0, 6, 3, 3, 1])
    loss, _, p, dz = fn(z, y)
    assert abs(loss - math.log(K)) < 1e-13
    ref = (np.full((N, K), 1.0 / K) - np.eye(K)[y]) / N
    np.testing.assert_allclose(dz, ref, rtol=0, atol=1e-15)


def pin_softmax_torch(fn):
    rng = np.random.default_rng(3)
    N, K = 9, 13
    z = rng.standard_normal((N, K)) * 3
    y = rng.integers(0, K, N)
    loss, sample, p, dz = fn(z, y)
    zt = torch.tensor(z, dtype=torch.float64, requires_grad=True)
    lt = torch.nn.functional.cross_entropy(zt, torch.tensor(y), reduction="mean")
    lt.backward()
    assert abs(loss - lt.item()) < 1e-12
    np.testing.assert_allclose(dz, zt.grad.numpy(), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(p, torch.softmax(torch.tensor(z), 1).numpy(), rtol=1e-12)
    ref_s = torch.nn.functional.cross_entropy(torch.tensor(z), torch.tensor(y), reduction="none")
    np.testing.assert_allclose(sample, ref_s.numpy(), rtol=1e-12)


def pin_softmax_finite_differences(fn):
    rng = np.random.default_rng(4)
    N, K = 3, 5
    z = rng.standard_normal((N, K))
    y = np.array([4, 0, 2])
    _, _, _, dz = fn(z, y)
    h = 1e-6
    for n in range(N):
        for k in range(K):
            zp, zm = z.copy(), z.copy()
            zp[n, k] += h
            zm[n, k] -= h
            fd = (fn(zp, y)[0] - fn(zm, y)[0]) / (2 * h)
            assert abs(fd - dz[n, k]) < 1e-8, (n, k, fd, dz[n, k])


def pin_softmax_shift_and_large_scores(fn):
    # adding a constant to a sample's scores changes nothing; scores of 1e3
    # stay finite
    rng = np.random.default_rng(5)
    z = rng.standard_normal((4, 6))
    y = np.array([1, 2, 3, 4])
    a = fn(z, y)
    b = fn(z + np.array([[1000.0], [-700.0], [0.5], [250.0]]), y)
    assert abs(a[0] - b[0]) < 1e-10
    np.testing.assert_allclose(a[3], b[3], rtol=0, atol=1e-12)
    assert all(np.all(np.isfinite(t)) for t in b[1:])


SOFTMAX_PINS = [pin_softmax_hand_example, pin_softmax_uniform_scores, pin_softmax_torch,
                pin_softmax_finite_differences, pin_softmax_shift_and_large_scores]


@pytest.mark.parametrize("pin", SOFTMAX_PINS)
def test_softmax_pins(pin):
    pin(oracle.softmax_loss)


def test_softmax_loss_weight_and_empty_batch():
    rng = np.random.default_rng(6)
    z = rng.standard_normal((4, 3))
    y = np.array([0, 1, 2, 0])
    l1, _, _, d1 = oracle.softmax_loss(z, y)
    l2, _, _, d2 = oracle.softmax_loss(z, y, loss_weight=2.5)
    assert abs(l2 - 2.5 * l1) < 1e-13
    np.testing.assert_allclose(d2, 2.5 * d1, rtol=1e-14)
    loss, sample, p, dz = oracle.softmax_loss(np.zeros((0, 10)), np.zeros(0, np.int64))
    assert loss == 0.0 and sample.shape == (0,) and dz.shape == (0, 10)
    with pytest.raises(ValueError):
        oracle.softmax_loss(z, np.array([0, 1, 3, 0]))


# ------------------------------------------------------------ SGD step
def pin_sgd_hand_example(fn):
    # w = 2, g = 0.5, v = 0.1, lr = 0.1, momentum 0.9, decay 0.01:
    # v' = 0.09 + 0.1 (0.5 + 0.02) = 0.142, w' = 1.858
    w, v = fn(np.array([2.0]), np.array([0.5]), np.array([0.1]), 0.1, 0.9, 0.01)
    np.testing.assert_allclose(v, [0.142], rtol=1e-14)
    np.testing.assert_allclose(w, [1.858], rtol=1e-14)


def pin_sgd_plain_descent(fn):
    rng = np.random.default_rng(7)
    w0, g = rng.standard_normal(6), rng.standard_normal(6)
    w, v = fn(w0, g, np.zeros(6), 0.05, 0.0, 0.0)
    np.testing.assert_allclose(w, w0 - 0.05 * g, rtol=1e-14)


def pin_sgd_constant_gradient_series(fn):
    # constant g, no decay: v_t = lr g (1 - mu^t) / (1 - mu) and
    # w_t = w_0 - lr g (t - mu (1 - mu^t) / (1 - mu)) / (1 - mu)
    lr, mu, g = 0.1, 0.9, np.array([0.3, -1.2])
    w, v = np.array([1.0, 2.0]), np.zeros(2)
    w0 = w.copy()
    for t in range(1, 8):
        w, v = fn(w, g, v, lr, mu, 0.0)
        np.testing.assert_allclose(v, lr * g * (1 - mu ** t) / (1 - mu), rtol=1e-12)
        s = (t - mu * (1 - mu ** t) / (1 - mu)) / (1 - mu)
        np.testing.assert_allclose(w, w0 - lr * g * s, rtol=1e-12)


def pin_sgd_weight_decay_only(fn):
    # g = 0, no momentum: w_t = w_0 (1 - lr decay)^t
    w, v = np.array([3.0, -1.5]), np.zeros(2)
    for t in range(1, 5):
        w, v = fn(w, np.zeros(2), v, 0.2, 0.0, 0.05)
        np.testing.assert_allclose(w, np.array([3.0, -1.5]) * (1 - 0.2 * 0.05) ** t, rtol=1e-13)


SGD_PINS = [pin_sgd_hand_example, pin_sgd_plain_descent, pin_sgd_constant_gradient_series,
            pin_sgd_weight_decay_only]


@pytest.mark.parametrize("pin", SGD_PINS)
def test_sgd_pins(pin):
    pin(oracle.sgd_step)


# ------------------------------------------------------------ schedules
def test_learning_rate_schedules():
    lr = oracle.learning_rate
    assert lr("fixed", 0.01, 12345) == 0.01
    assert lr("step", 0.01, 99, gamma=0.1, stepsize=100) == 0.01
    assert abs(lr("step", 0.01, 100, gamma=0.1, stepsize=100) - 1e-3) < 1e-18
    assert abs(lr("step", 0.01, 250, gamma=0.1, stepsize=100) - 1e-4) < 1e-18
    assert abs(lr("exp", 0.5, 3, gamma=0.5) - 0.0625) < 1e-18
    assert lr("inv", 0.01, 0, gamma=1e-4, power=0.75) == 0.01
    # (1 + 1e-4 * 10000)^-0.75 = 2^-0.75
    assert abs(lr("inv", 0.01, 10000, gamma=1e-4, power=0.75) - 0.01 * 2 ** -0.75) < 1e-16
    with pytest.raises(ValueError):
        lr("poly", 0.01, 1)


# ------------------------------------------------------------ the pins catch mistakes
def _softmax_variants():
    f = oracle.softmax_loss

    def no_mean(z, y, w=1.0):       # sum instead of mean over the batch
        l, s, p, d = f(z, y, w)
        return l * len(y), s, p, d * len(y)

    def wrong_sign(z, y, w=1.0):    # gradient onehot - p
        l, s, p, d = f(z, y, w)
        return l, s, p, -d

    def no_max_shift(z, y, w=1.0):  # exp without the max subtracted (overflows)
        z = np.asarray(z, np.float64)
        e = np.exp(z)
        p = e / e.sum(1, keepdims=True)
        n = len(y)
        s = -np.log(p[np.arange(n), y])
        d = p.copy()
        d[np.arange(n), y] -= 1
        return s.mean() * w, s, p, d * w / n

    def label_off_by_one(z, y, w=1.0):
        return f(z, (np.asarray(y) + 1) % np.asarray(z).reshape(len(y), -1).shape[1], w)

    return [no_mean, wrong_sign, no_max_shift, label_off_by_one]


def _sgd_variants():
    f = oracle.sgd_step
    return [
        lambda w, g, v, lr, mu, wd: f(w, g, v, lr, mu, -wd),             # decay sign
        lambda w, g, v, lr, mu, wd: f(w, g, v * 0, lr, mu, wd),          # momentum dropped
        lambda w, g, v, lr, mu, wd: (lambda r: (r[0], r[1] / lr if lr else r[1]))(
            f(w, g, v, lr, mu, wd)),                                     # lr outside the history
        lambda w, g, v, lr, mu, wd: f(w, -np.asarray(g), v, lr, mu, wd),  # ascent
    ]


@pytest.mark.parametrize("i", range(4))
def test_softmax_pins_catch_a_planted_mistake(i):
    bad = _softmax_variants()[i]
    failed = 0
    for pin in SOFTMAX_PINS:
        try:
            with np.errstate(all="ignore"):
                pin(bad)
        except (AssertionError, FloatingPointError, ValueError):
            failed += 1
    assert failed >= 1


@pytest.mark.parametrize("i", range(4))
def test_sgd_pins_catch_a_planted_mistake(i):
    bad = _sgd_variants()[i]
    failed = 0
    for pin in SGD_PINS:
        try:
            pin(bad)
        except AssertionError:
            failed += 1
    assert failed >= 1
