"""Seeded synthetic tensors for the calibration workloads.

Both the GPU path (tests, bench) and the CPU oracle draw their inputs from
here, so they see the same bytes.  The module only draws random numbers; it
holds none of the quantizer's arithmetic.

Every tensor is identified by (seed, name): the generator is
``numpy.random.default_rng([seed, crc32(name)])``, so a tensor does not depend
on which other tensors were drawn before it.  Shapes are given in the
canonical PyTorch layouts (NCHW activations, OIHW / [out][in] weights); each
consumer permutes to its own layout.

Distributions (standard deviations, numpy convention):
  images            N(0, 1)
  FC weights (cfg1) N(0, 0.05); FC activations ReLU(N(0, 1))
  conv/FC weights   He-normal: N(0, sqrt(2 / fan_in)), fan_in = in * kh * kw
  biases            N(0, 0.01)
  BN gamma          U(0.5, 1.5); BN beta N(0, 0.1); running mean 0, var 1
"""
import zlib

import numpy as np


def rng_for(seed: int, name: str) -> np.random.Generator:
    return np.random.default_rng([int(seed) & 0xFFFFFFFF, zlib.crc32(name.encode())])


def normal(seed, name, shape, std=1.0, mean=0.0):
    g = rng_for(seed, name)
    return (g.standard_normal(size=shape, dtype=np.float32) * np.float32(std)
            + np.float32(mean)).astype(np.float32)


def relu_normal(seed, name, shape):
    return np.maximum(normal(seed, name, shape), np.float32(0.0))


def he_normal(seed, name, shape):
    fan_in = int(np.prod(shape[1:]))
    return normal(seed, name, shape, std=float(np.sqrt(2.0 / fan_in)))


def uniform(seed, name, shape, lo, hi):
    g = rng_for(seed, name)
    return g.uniform(lo, hi, size=shape).astype(np.float32)


def integers(seed, name, shape, lo, hi):
    """Integers in [lo, hi] inclusive (int64)."""
    g = rng_for(seed, name)
    return g.integers(lo, hi + 1, size=shape, dtype=np.int64)


def choice(seed, name, options, count):
    g = rng_for(seed, name)
    return [int(v) for v in g.choice(np.asarray(options), size=count)]
