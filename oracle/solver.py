"""Softmax loss and stochastic gradient descent, plain numpy in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).  These are the loss
layer and the training algorithm of the paper's Sec. 3.2 (softmax loss among
the layer types) and Sec. 3.4 (training by stochastic gradient descent over
mini-batches, with learning-rate decay schedules and momentum).  The paper
gives no formulas; the standard definitions are written out here:

* softmax loss of a mini-batch of N score vectors z_n (K classes each) with
  labels y_n:  p_{n,k} = exp(z_{n,k}) / sum_j exp(z_{n,j}),
  loss = -(1/N) sum_n log p_{n,y_n};  d loss / d z_{n,k} = (p_{n,k} - [k == y_n]) / N.
* one SGD step with momentum mu and L2 weight decay lambda at learning rate
  lr:  v <- mu v + lr (g + lambda w);  w <- w - v.
* learning-rate schedules at iteration t (0 for the first update):
  fixed lr0;  step lr0 gamma^floor(t / stepsize);  exp lr0 gamma^t;
  inv lr0 (1 + gamma t)^(-power).
"""
import numpy as np


def softmax_loss(z, labels, loss_weight=1.0):
    """z: (N, K) scores (any trailing 1x1 dims are flattened), labels: (N,)
    ints in [0, K).  Returns (loss, per-sample losses, p, dz), float64."""
    z = np.asarray(z, dtype=np.float64)
    N = z.shape[0]
    K = int(np.prod(z.shape[1:]))
    z = z.reshape(N, K)
    y = np.asarray(labels).reshape(N).astype(np.int64)
    if N and (y.min() < 0 or y.max() >= K):
        raise ValueError("labels must lie in [0, K)")
    # probabilities p_{n,k} = exp(z_{n,k}) / sum_j exp(z_{n,j}), computed with
    # the row maximum subtracted (the same ratio, no overflow)
    e = np.exp(z - z.max(axis=1, keepdims=True)) if N else np.zeros_like(z)
    p = e / e.sum(axis=1, keepdims=True) if N else e
    # -log p_{n,y_n} = log sum_j exp(z_{n,j}) - z_{n,y_n}
    m = z.max(axis=1) if N else np.zeros(0)
    lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1)) if N else np.zeros(0)
    sample = lse - z[np.arange(N), y]
    loss = loss_weight * sample.sum() / N if N else 0.0
    dz = p.copy()
    dz[np.arange(N), y] -= 1.0
    dz *= loss_weight / N if N else 0.0
    return loss, sample, p, dz


def sgd_step(w, g, v, lr, momentum=0.0, weight_decay=0.0):
    """One update: v <- momentum v + lr (g + weight_decay w); w <- w - v.
    Returns (new w, new v), float64."""
    w = np.asarray(w, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    v_new = momentum * v + lr * (g + weight_decay * w)
    return w - v_new, v_new


def learning_rate(policy, base_lr, it, gamma=0.0, power=0.0, stepsize=1):
    """Learning rate at iteration `it` (0 for the first update)."""
    if policy == "fixed":
        return float(base_lr)
    if policy == "step":
        return float(base_lr) * float(gamma) ** (it // int(stepsize))
    if policy == "exp":
        return float(base_lr) * float(gamma) ** it
    if policy == "inv":
        return float(base_lr) * (1.0 + float(gamma) * it) ** (-float(power))
    raise ValueError(f"unknown learning-rate policy {policy!r}")
