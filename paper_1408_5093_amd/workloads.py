"""Seeded synthetic workloads: layer shapes and input generators.

This module holds shapes and random draws only -- none of the layer's
arithmetic -- so that the HIP path and the CPU oracle can be fed the very
same inputs.  Every tensor is drawn in float64 from
``numpy.random.default_rng([1408, 5093, workload_id, tensor_id])`` and then
rounded once to float32 (and, for the bfloat16 workload, to bfloat16 with
round-to-nearest-even).  Neither MNIST nor ImageNet is used: the draws only
mimic their shapes and value ranges (mean-subtracted pixels ~ N(0, 50),
post-ReLU activations ~ |N(0, 1)|, MNIST-like pixels ~ U[0, 1)).

Geometry.  The CaffeNet conv1-5 stack (the AlexNet-style reference model the
paper ships) at batch N, and the two conv layers of the LeNet MNIST example
of the paper's Fig. 1.
"""
from dataclasses import dataclass

import numpy as np

SEED = (1408, 5093)


@dataclass(frozen=True)
class ConvLayer:
    name: str
    C: int
    H: int
    W: int
    K: int
    k: int
    s: int
    p: int
    g: int
    relu: bool

    def out_hw(self):
        Ho = (self.H + 2 * self.p - self.k) // self.s + 1
        Wo = (self.W + 2 * self.p - self.k) // self.s + 1
        return Ho, Wo

    def flops(self, N):
        """Multiply-adds x 2 of one pass (forward, data grad or weight grad)."""
        Ho, Wo = self.out_hw()
        return 2 * N * self.K * Ho * Wo * (self.C // self.g) * self.k * self.k


CAFFENET = (
    ConvLayer("conv1", 3, 227, 227, 96, 11, 4, 0, 1, True),
    ConvLayer("conv2", 96, 27, 27, 256, 5, 1, 2, 2, True),
    ConvLayer("conv3", 256, 13, 13, 384, 3, 1, 1, 1, True),
    ConvLayer("conv4", 384, 13, 13, 384, 3, 1, 1, 2, True),
    ConvLayer("conv5", 384, 13, 13, 256, 3, 1, 1, 2, True),
)
# Glue after conv1 and conv2: 3x3 stride-2 max pooling, then LRN (size 5).
CAFFENET_POOL = dict(kernel=3, stride=2, pad=0)
CAFFENET_LRN = dict(size=5, alpha=1e-4, beta=0.75, k=1.0)

LENET = (
    ConvLayer("conv1", 1, 28, 28, 20, 5, 1, 0, 1, False),
    ConvLayer("conv2", 20, 12, 12, 50, 5, 1, 0, 1, False),
)
LENET_POOL = dict(kernel=2, stride=2, pad=0)

# The inner-product (fully connected) layers that follow the conv stacks:
# CaffeNet fc6-fc8 on pool5's 256 x 6 x 6 output and LeNet ip1-ip2 on pool2's
# 50 x 4 x 4 output.  An inner product is the 1x1 convolution of a 1x1 image
# whose channels are the flattened (c, h, w) input.
CAFFENET_FC = (
    ConvLayer("fc6", 256 * 6 * 6, 1, 1, 4096, 1, 1, 0, 1, True),
    ConvLayer("fc7", 4096, 1, 1, 4096, 1, 1, 0, 1, True),
    ConvLayer("fc8", 4096, 1, 1, 1000, 1, 1, 0, 1, False),
)
# The whole CaffeNet chain of the paper's reference model: conv1-5, max-pool
# after conv5, fc6-fc8 (dropout, a training-time mask, is not part of it).
CAFFENET_NET = CAFFENET + CAFFENET_FC
CAFFENET_NET_GLUE = {0: [("pool", CAFFENET_POOL), ("lrn", CAFFENET_LRN)],
                     1: [("pool", CAFFENET_POOL), ("lrn", CAFFENET_LRN)],
                     4: [("pool", CAFFENET_POOL)]}

LENET_FC = (
    ConvLayer("ip1", 50 * 4 * 4, 1, 1, 500, 1, 1, 0, 1, True),
    ConvLayer("ip2", 500, 1, 1, 10, 1, 1, 0, 1, False),
)
# The whole LeNet of Fig. 1: conv1, pool, conv2, pool, ip1 + ReLU, ip2, then
# the softmax loss; trained by SGD with momentum 0.9, weight decay 5e-4 and
# the "inv" schedule lr = 0.01 (1 + 1e-4 t)^-0.75.
LENET_NET = LENET + LENET_FC
LENET_NET_GLUE = {0: [("pool", LENET_POOL)], 1: [("pool", LENET_POOL)]}
LENET_SOLVER = dict(policy="inv", base_lr=0.01, gamma=1e-4, power=0.75, momentum=0.9,
                    weight_decay=5e-4)

# Workload ids (the third seed word).
LENET_PAIR = 1          # LeNet conv pair, N=64
CAFFENET_CONV1_FWD = 2  # conv1 forward, N=256
CAFFENET_CONV25_FWD = 3 # conv2..5 forward, N=256, inputs drawn per layer
CAFFENET_STEP = 4       # conv1-5 forward + backward with pool/LRN glue, N=256
CAFFENET_STEP_BF16 = 5  # the same at N=512 with bfloat16 operands
CAFFENET_FC_LAYER = 6   # one inner-product layer fc6..fc8, N=256, inputs drawn per layer
CAFFENET_NET_STEP = 7   # conv1-5 + pool5 + fc6-fc8 forward + backward, N=256
LENET_TRAIN = 8         # LeNet training iterations (softmax loss + SGD), N=64


def rng(workload, tensor_id):
    return np.random.default_rng([SEED[0], SEED[1], int(workload), int(tensor_id)])


def normal(workload, tensor_id, shape, std, mean=0.0):
    return (rng(workload, tensor_id).standard_normal(shape) * std + mean).astype(np.float32)


def half_normal(workload, tensor_id, shape, std=1.0):
    return np.abs(rng(workload, tensor_id).standard_normal(shape) * std).astype(np.float32)


def uniform(workload, tensor_id, shape, lo, hi):
    return rng(workload, tensor_id).uniform(lo, hi, shape).astype(np.float32)


def xavier_uniform(workload, tensor_id, shape):
    """U(-a, a) with a = sqrt(3 / fan_in), fan_in = C/group * kh * kw."""
    fan_in = int(np.prod(shape[1:]))
    a = np.sqrt(3.0 / fan_in)
    return uniform(workload, tensor_id, shape, -a, a)


def to_bf16_bits(a):
    """float32 array -> uint16 bfloat16 bit patterns, round to nearest even."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = (u & 0x7F800000) == 0x7F800000
    nan &= (u & 0x007FFFFF) != 0
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    r[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return r


def bf16_bits_to_f32(b):
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_bf16(a):
    """float32 values rounded to the nearest bfloat16 (as float32)."""
    return bf16_bits_to_f32(to_bf16_bits(a))


# Tensor ids: 0 = input image batch; 10 + l = weights of layer l; 20 + l =
# bias of layer l; 30 = top gradient; 40 + l = per-layer input (forward-only
# workloads).
def lenet_pair(N=64):
    w = LENET_PAIR
    x = uniform(w, 0, (N, 1, 28, 28), 0.0, 1.0)
    Ws = [xavier_uniform(w, 10 + l, (L.K, L.C // L.g, L.k, L.k)) for l, L in enumerate(LENET)]
    bs = [normal(w, 20 + l, (L.K,), 0.01) for l, L in enumerate(LENET)]
    Ho, Wo = LENET[1].out_hw()
    g = normal(w, 30, (N, LENET[1].K, Ho, Wo), 1.0)
    return dict(x=x, W=Ws, b=bs, top_diff=g)


def caffenet_conv1_fwd(N=256):
    w = CAFFENET_CONV1_FWD
    L = CAFFENET[0]
    return dict(x=normal(w, 0, (N, 3, 227, 227), 50.0),
                W=normal(w, 10, (L.K, L.C // L.g, L.k, L.k), 0.01),
                b=np.zeros((L.K,), np.float32))


def caffenet_conv25_layer(l, N=256):
    """Inputs of layer l (1..4 -> conv2..conv5) for the forward-only workload."""
    w = CAFFENET_CONV25_FWD
    L = CAFFENET[l]
    return dict(x=half_normal(w, 40 + l, (N, L.C, L.H, L.W)),
                W=normal(w, 10 + l, (L.K, L.C // L.g, L.k, L.k), 0.01),
                b=np.full((L.K,), 0.1, np.float32))


def caffenet_step(N=256, workload=CAFFENET_STEP):
    """Weights, biases, input batch and top gradient of the conv1-5 training step."""
    x = normal(workload, 0, (N, 3, 227, 227), 50.0)
    Ws = [normal(workload, 10 + l, (L.K, L.C // L.g, L.k, L.k), 0.01)
          for l, L in enumerate(CAFFENET)]
    bs = [np.full((L.K,), 0.0 if l == 0 else 0.1, np.float32) for l, L in enumerate(CAFFENET)]
    Ho, Wo = CAFFENET[4].out_hw()
    g = normal(workload, 30, (N, CAFFENET[4].K, Ho, Wo), 1e-3)
    return dict(x=x, W=Ws, b=bs, top_diff=g)


def caffenet_fc_layer(l, N=256):
    """Input, weights, bias and top gradient of inner-product layer l (0..2 ->
    fc6..fc8): post-ReLU activations in, Gaussian weights (std 0.005 for
    fc6-fc7, 0.01 for fc8, as the reference model initialises them)."""
    w = CAFFENET_FC_LAYER
    L = CAFFENET_FC[l]
    return dict(x=half_normal(w, 40 + l, (N, L.C, 1, 1)),
                W=normal(w, 10 + l, (L.K, L.C, 1, 1), 0.01 if l == 2 else 0.005),
                b=np.full((L.K,), 0.1 if l < 2 else 0.0, np.float32),
                top_diff=normal(w, 30 + l, (N, L.K, 1, 1), 1e-3))


def caffenet_net_step(N=256):
    """Weights, biases, input batch and fc8 top gradient of the whole-network
    CaffeNet step (conv weights N(0, 0.01); fc6-fc7 N(0, 0.005), fc8
    N(0, 0.01); biases 0.1, 0 for conv1 and fc8)."""
    w = CAFFENET_NET_STEP
    x = normal(w, 0, (N, 3, 227, 227), 50.0)
    Ws, bs = [], []
    for l, L in enumerate(CAFFENET_NET):
        std = 0.005 if L.name in ("fc6", "fc7") else 0.01
        Ws.append(normal(w, 10 + l, (L.K, L.C // L.g, L.k, L.k), std))
        bs.append(np.full((L.K,), 0.0 if L.name in ("conv1", "fc8") else 0.1, np.float32))
    g = normal(w, 30, (N, CAFFENET_NET[-1].K, 1, 1), 1e-3)
    return dict(x=x, W=Ws, b=bs, top_diff=g)


def lenet_train(N=64, batches=1):
    """Weights (Xavier-uniform), zero biases, `batches` input batches
    (MNIST-like pixels U[0, 1)) and int32 labels uniform over the 10 classes."""
    w = LENET_TRAIN
    Ws = [xavier_uniform(w, 10 + l, (L.K, L.C // L.g, L.k, L.k)) for l, L in enumerate(LENET_NET)]
    bs = [np.zeros((L.K,), np.float32) for L in LENET_NET]
    xs = [uniform(w, 100 + i, (N, 1, 28, 28), 0.0, 1.0) for i in range(batches)]
    ys = [rng(w, 200 + i).integers(0, 10, N).astype(np.int32) for i in range(batches)]
    return dict(W=Ws, b=bs, x=xs, labels=ys)
