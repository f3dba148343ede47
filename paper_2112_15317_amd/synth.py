"""Seeded synthetic inputs for the worker-share workloads.

This module only draws random numbers: it holds none of the arithmetic of
the layers being computed.  Both the GPU library's callers and the tests'
CPU oracle consume the arrays it returns, so the two sides always see the
same values.

Every tensor comes from its own stream
``Generator(PCG64(SeedSequence([seed, tensor_id])))`` with a fixed
``tensor_id`` (see ``TID``), so any tensor can be regenerated on its own.

Distributions (stand-ins for CIFAR-10 / ImageNet images and for trained
state, which are not used):
  * images, upstream gradients: N(0, 1) (per-channel-normalised pixels);
  * conv weights: He-normal, std = sqrt(2 / (9 * C_in)) (fan-in);
  * FC weights: Xavier-uniform on the *full* layer, bound
    sqrt(6 / (fan_in + fan_out)); a worker's shard is a column slice;
  * gathered FC activations and remote stand-ins: max(N(0,1), 0), the
    distribution of a ReLU output;
  * biases: zero unless a test asks for N(0, 1) values.
"""
from __future__ import annotations

import math

import numpy as np


class TID:
    """Fixed tensor ids of the seeded streams."""
    IMAGES = 0
    DY_TOP = 1
    CONV_W = 100          # + layer index
    CONV_B = 200          # + layer index
    FC_W = 300            # + FC layer index (full matrix)
    FC_B = 400            # + FC layer index
    X0_REMOTE = 500       # gathered rows of the other replicas (FC0 input)
    X1_REMOTE = 501       # feature columns of the other shards (FC1 input)
    FC_DY = 502           # upstream gradient of the last FC shard
    LABELS = 503          # class labels of the gathered rows
    LOGITS_REMOTE = 504   # the other shards' columns of the last FC output
    FC_X = 600            # standalone FC-shard input
    COLS_REMOTE = 700     # + FC layer index (>= 2): other shards' columns of its input
    MISC = 900            # + anything a test needs


def generator(seed: int, tensor_id: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tensor_id])))


def normal(shape, seed: int, tensor_id: int, std: float = 1.0) -> np.ndarray:
    """float32 array ~ N(0, std^2)."""
    g = generator(seed, tensor_id)
    return (g.standard_normal(shape) * std).astype(np.float32)


def relu_normal(shape, seed: int, tensor_id: int) -> np.ndarray:
    """float32 array ~ max(N(0,1), 0)."""
    g = generator(seed, tensor_id)
    return np.maximum(g.standard_normal(shape), 0.0).astype(np.float32)


def he_normal_conv3x3(k: int, c: int, seed: int, tensor_id: int) -> np.ndarray:
    """KCRS float32 weights, std = sqrt(2 / (9 c))."""
    return normal((k, c, 3, 3), seed, tensor_id, std=math.sqrt(2.0 / (9.0 * c)))


def xavier_uniform(fan_in: int, fan_out: int, seed: int, tensor_id: int) -> np.ndarray:
    """Full [fan_in, fan_out] float32 matrix ~ U(-a, a), a = sqrt(6/(in+out))."""
    a = math.sqrt(6.0 / (fan_in + fan_out))
    g = generator(seed, tensor_id)
    return g.uniform(-a, a, size=(fan_in, fan_out)).astype(np.float32)


def labels(m: int, classes: int, seed: int, tensor_id: int) -> np.ndarray:
    """int32 array of m class labels ~ U{0, ..., classes - 1}."""
    return generator(seed, tensor_id).integers(0, classes, size=m).astype(np.int32)


def zeros(shape) -> np.ndarray:
    return np.zeros(shape, dtype=np.float32)


def to_bf16(a: np.ndarray):
    """CPU torch bfloat16 tensor holding a's float32 values rounded to
    nearest-even (torch's own conversion)."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
