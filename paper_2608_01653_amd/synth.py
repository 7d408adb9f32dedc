"""Seeded synthetic inputs shared by the HIP path's tests/bench and the CPU oracle.

This module only draws random numbers: it holds none of the method's arithmetic
(no transform, no quantizer, no convolution), so both sides can consume the same
arrays without sharing any computation.

Distributions follow the learned-image-coding workloads described in Sec. IV-A
(heavy-tailed activations with a few channel-localized outliers and sparse large
responses) and Sec. V-A (RGB images of the Kodak size 512x768 and 2K-class CLIC
images, which these synthetic tensors stand in for).

Every generator uses one ``numpy.random.default_rng(seed)`` (PCG64) and draws in a
fixed order, so results are reproducible run to run and machine to machine.
"""
from __future__ import annotations

import numpy as np

NU_ACT = 3.0      # Student-t degrees of freedom for activations
NU_W = 4.0        # Student-t degrees of freedom for weights
W_STD = 0.05      # weight standard deviation
BIAS_STD = 0.05   # bias standard deviation
N_OFFSET_CH = 8   # channels that carry a +3 sigma mean offset


def heavy_tailed_activations(rng: np.random.Generator, shape) -> np.ndarray:
    """fp32 NHWC activations: Student-t(3) times per-channel log-normal(0,1) scales,
    with ``N_OFFSET_CH`` channels shifted by +3 standard deviations.

    Draw order: channel scales, t samples, offset channel choice.
    The standard deviation of a unit Student-t(nu) is sqrt(nu/(nu-2)), sqrt(3) here.
    """
    shape = tuple(int(v) for v in shape)
    c = shape[-1]
    scale = rng.lognormal(0.0, 1.0, c)
    t = rng.standard_t(NU_ACT, shape)
    nofs = min(N_OFFSET_CH, c)
    chans = rng.choice(c, nofs, replace=False)
    offset = np.zeros(c)
    offset[chans] = 3.0 * np.sqrt(NU_ACT / (NU_ACT - 2.0)) * scale[chans]
    return (t * scale + offset).astype(np.float32)


def student_t_weights(rng: np.random.Generator, shape) -> np.ndarray:
    """fp32 weights: 0.05 times a unit-variance Student-t(4) (std of t4 is sqrt(2))."""
    t = rng.standard_t(NU_W, tuple(int(v) for v in shape))
    return (W_STD * t / np.sqrt(NU_W / (NU_W - 2.0))).astype(np.float32)


def bias(rng: np.random.Generator, cout: int) -> np.ndarray:
    return rng.normal(0.0, BIAS_STD, int(cout)).astype(np.float32)


def rgb_uniform(rng: np.random.Generator, shape) -> np.ndarray:
    """fp32 NHWC image in [0, 1)."""
    return rng.random(tuple(int(v) for v in shape), dtype=np.float32)


def dyadic_integers(rng: np.random.Generator, shape, lim: int = 1024) -> np.ndarray:
    """Integer-valued fp32 in [-lim, lim]: every partial sum of a <=128-point signed
    sum is exact in fp32, so any summation order gives identical results."""
    return rng.integers(-lim, lim + 1, tuple(int(v) for v in shape)).astype(np.float32)


def int8_codes(rng: np.random.Generator, shape, lim: int = 127) -> np.ndarray:
    """Random symmetric INT8 codes in [-lim, lim]."""
    return rng.integers(-lim, lim + 1, tuple(int(v) for v in shape)).astype(np.int8)


def weight_shape(cin: int, cout: int, k: int, transposed: bool):
    """PyTorch weight layout: OIHW for a convolution, IOHW for a transposed one."""
    return (cin, cout, k, k) if transposed else (cout, cin, k, k)


def layer_params(rng: np.random.Generator, cin: int, cout: int, k: int,
                 transposed: bool = False, with_bias: bool = True):
    """Weights (drawn first) then bias, for one layer."""
    w = student_t_weights(rng, weight_shape(cin, cout, k, transposed))
    b = bias(rng, cout) if with_bias else None
    return w, b
