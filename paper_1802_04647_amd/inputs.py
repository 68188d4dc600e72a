"""Seeded synthetic inputs for the conv2d layer and the LeNet/ResNet-shaped workloads.

This module only draws random numbers and arranges them in the DML matrix layout
(an [N, C, H, W] tensor is an N x (C*H*W) row-major matrix).  It holds none of
the layer arithmetic, so both the GPU library's tests and the oracle can consume
its arrays.  Draws are float64 (numpy PCG64); fp32 mode rounds the same draws to
float32 with round-to-nearest-even (``to_dtype``).

Workloads (shapes follow the paper's LeNet and ResNet examples; the paper names
no dataset, so every input is synthetic):

* ``conv_small``   N=4, C=1, 8x8, F=2 3x3 s1 p1
* ``lenet_conv1``  N=64, C=1, 28x28 (~80% exact zeros), F=32 5x5 s1 p2
* ``lenet_conv2``  N=64, C=32, 14x14 (relu(N(0,1))), F=64 5x5 s1 p2, then 2x2/2 max-pool
* ``lenet_train``  one SGD-momentum step of a LeNet-style net, batch 64
* ``resnet_conv``  N=256, C=64, 56x56 (relu(N(0,1))), F=64 3x3 s1 p1
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

BASE_SEED = 180204647


def streams(k: int, count: int = 6):
    """Independent generators for workload k: X, mask, W, dout, labels, spare."""
    ss = np.random.SeedSequence(BASE_SEED + k)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(count)]


def to_dtype(a: np.ndarray, dtype: str) -> np.ndarray:
    """Round a float64 draw to the mode's storage type ('f64' or 'f32')."""
    if dtype == "f64":
        return np.ascontiguousarray(a, dtype=np.float64)
    if dtype == "f32":
        return np.ascontiguousarray(a, dtype=np.float32)
    raise ValueError(f"unknown dtype {dtype!r}")


def he_normal(rng, rows: int, fan_in: int) -> np.ndarray:
    """Weights ~ N(0, std = sqrt(2 / fan_in)), shape rows x fan_in."""
    return rng.standard_normal((rows, fan_in)) * math.sqrt(2.0 / fan_in)


def relu_normal(rng, shape) -> np.ndarray:
    """max(0, N(0,1)) draws: about half exact zeros."""
    z = rng.standard_normal(shape)
    z[z < 0.0] = 0.0
    return z


def sparse_uniform(rng_mask, rng_val, shape, keep: float) -> np.ndarray:
    """Bernoulli(keep) mask times U[0,1): about (1-keep) exact zeros, i.i.d."""
    m = rng_mask.random(shape) < keep
    v = rng_val.random(shape)
    return np.where(m, v, 0.0)


@dataclass(frozen=True)
class ConvShape:
    N: int
    C: int
    Hin: int
    Win: int
    F: int
    Hf: int
    Wf: int
    stride: int
    pad: int

    @property
    def Hout(self) -> int:
        return (self.Hin + 2 * self.pad - self.Hf) // self.stride + 1

    @property
    def Wout(self) -> int:
        return (self.Win + 2 * self.pad - self.Wf) // self.stride + 1

    @property
    def K(self) -> int:
        return self.C * self.Hf * self.Wf

    def flops_per_pass(self) -> float:
        """Dense algorithmic work of one conv pass: 2*N*F*Hout*Wout*C*Hf*Wf."""
        return 2.0 * self.N * self.F * self.Hout * self.Wout * self.K

    def args(self):
        return (self.N, self.C, self.Hin, self.Win, self.F, self.Hf, self.Wf, self.stride,
                self.pad)


SHAPES = {
    "conv_small": ConvShape(4, 1, 8, 8, 2, 3, 3, 1, 1),
    "lenet_conv1": ConvShape(64, 1, 28, 28, 32, 5, 5, 1, 2),
    "lenet_conv2": ConvShape(64, 32, 14, 14, 64, 5, 5, 1, 2),
    "resnet_conv": ConvShape(256, 64, 56, 56, 64, 3, 3, 1, 1),
}

WORKLOAD_INDEX = {"conv_small": 1, "lenet_conv1": 2, "lenet_conv2": 3, "lenet_train": 4,
                  "resnet_conv": 5}


def conv_layer_inputs(name: str, N: int | None = None):
    """X, W, b, dout (float64) for a single-conv workload; N may be reduced for tests.

    ``dout`` has the conv output's shape.  For ``lenet_conv2`` it is instead the
    upstream gradient of the pooled output (N x F*7*7); the caller routes it
    through the pool backward to get the conv's dout.
    """
    s = SHAPES[name]
    k = WORKLOAD_INDEX[name]
    n = s.N if N is None else N
    g_x, g_mask, g_w, g_dout, _, _ = streams(k)
    P_in = s.C * s.Hin * s.Win
    P_out = s.F * s.Hout * s.Wout
    if name == "conv_small":
        X = g_x.uniform(-1.0, 1.0, (n, P_in))
        W = he_normal(g_w, s.F, s.K)
        b = np.full((s.F,), 0.1)
        dout = g_dout.uniform(-1.0, 1.0, (n, P_out))
    elif name == "lenet_conv1":
        X = sparse_uniform(g_mask, g_x, (n, P_in), keep=0.2)
        W = he_normal(g_w, s.F, s.K)
        b = np.zeros((s.F,))
        dout = g_dout.standard_normal((n, P_out))
    elif name == "lenet_conv2":
        X = relu_normal(g_x, (n, P_in))
        W = he_normal(g_w, s.F, s.K)
        b = np.zeros((s.F,))
        Hp, Wp = s.Hout // 2, s.Wout // 2
        dout = g_dout.standard_normal((n, s.F * Hp * Wp))
    elif name == "resnet_conv":
        X = relu_normal(g_x, (n, P_in))
        W = he_normal(g_w, s.F, s.K)
        b = np.zeros((s.F,))
        dout = g_dout.standard_normal((n, P_out))
    else:
        raise KeyError(name)
    return X, W, b, dout


# LeNet-style training step: conv(1->32,5x5,p2)-relu-pool2 -> conv(32->64,5x5,p2)-relu-pool2
# -> affine 3136->512 relu -> affine 512->10 -> softmax + cross-entropy.
LENET = dict(N=64, classes=10, lr=0.01, mu=0.9,
             conv1=ConvShape(64, 1, 28, 28, 32, 5, 5, 1, 2),
             conv2=ConvShape(64, 32, 14, 14, 64, 5, 5, 1, 2),
             fc1=(3136, 512), fc2=(512, 10))


def lenet_train_inputs(N: int = 64):
    """Batch X (N x 784, ~80% zeros), one-hot Y (N x 10), and the 8 initial parameters."""
    g_x, g_mask, g_w, _, g_lab, _ = streams(WORKLOAD_INDEX["lenet_train"])
    X = sparse_uniform(g_mask, g_x, (N, 784), keep=0.2)
    labels = g_lab.integers(0, 10, size=N)
    Y = np.zeros((N, 10))
    Y[np.arange(N), labels] = 1.0
    W1 = he_normal(g_w, 32, 25)
    W2 = he_normal(g_w, 64, 800)
    # affine weights are D x M; fan_in = D
    W3 = g_w.standard_normal((3136, 512)) * math.sqrt(2.0 / 3136)
    W4 = g_w.standard_normal((512, 10)) * math.sqrt(2.0 / 512)
    params = dict(W1=W1, b1=np.zeros(32), W2=W2, b2=np.zeros(64),
                  W3=W3, b3=np.zeros(512), W4=W4, b4=np.zeros(10))
    return X, Y, params


def random_conv_case(seed: int, shape: ConvShape, zero_frac: float = 0.0, bias: float | None = None):
    """Generic seeded case for parity sweeps: X (with i.i.d. zeros), W, b, dout."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(BASE_SEED ^ (seed * 7919 + 13))))
    s = shape
    X = g.standard_normal((s.N, s.C * s.Hin * s.Win))
    if zero_frac > 0:
        X[g.random(X.shape) < zero_frac] = 0.0
    W = g.standard_normal((s.F, s.K)) * math.sqrt(2.0 / s.K)
    b = g.standard_normal(s.F) * 0.1 if bias is None else np.full(s.F, float(bias))
    dout = g.standard_normal((s.N, s.F * s.Hout * s.Wout))
    return X, W, b, dout


def rng(seed: int):
    """A plain seeded generator for ad-hoc test data."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(BASE_SEED ^ seed)))


def structured_zero_conv_case(seed: int, shape: ConvShape):
    """X, W, b, dout, mask source with structured zeros (the supplementary input
    of the zero-skip path): besides ~30% i.i.d. zeros, X has a zero band over
    the top third of every image and every third channel zero; dout and the
    mask source (relu of a normal draw) have zero bands over the bottom half of
    the even-numbered filters and every fourth filter zero.  Whole matrix-core
    fragments of these inputs are zero, which i.i.d. zeros almost never give."""
    s = shape
    X, W, b, dout = random_conv_case(seed, s, zero_frac=0.3)
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(BASE_SEED ^ (seed * 104729 + 7))))
    X = X.reshape(s.N, s.C, s.Hin, s.Win)
    X[:, :, : max(1, s.Hin // 3), :] = 0.0
    X[:, ::3] = 0.0
    mask = relu_normal(g, (s.N, s.F, s.Hout, s.Wout))
    dout = dout.reshape(s.N, s.F, s.Hout, s.Wout)
    for a in (dout, mask):
        a[:, ::2, s.Hout // 2:, :] = 0.0
        a[:, 1::4] = 0.0
    return (X.reshape(s.N, -1).copy(), W, b, dout.reshape(s.N, -1).copy(),
            mask.reshape(s.N, -1).copy())
