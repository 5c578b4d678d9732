"""Oracle of the calibration loop -- TEST INFRASTRUCTURE ONLY (like the rest
of this package: only the tests, the smoke check and the benchmark's
CPU-baseline leg use it).

Adam with bias correction as published by Kingma and Ba (2015): for step
t = 1, 2, ...
    m = beta1 m + (1 - beta1) g
    v = beta2 v + (1 - beta2) g^2
    p = p - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
driven by the oracle's exact per-lane gradients, as in the paper's Kalman
maximum-likelihood calibration (Section "From buckets to phases"), where an
Adam optimiser fits a model's parameters with the interpreter's gradients.
Plain numpy in fp64, one operation at a time in the order above; beta^t is
Python's ``**`` (the C library's pow)."""
from __future__ import annotations

import numpy as np

from . import run


def adam_step(p, g, m, v, t: int, lr: float, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8):
    """One Adam step on arrays of equal shape, in place; returns p."""
    c1 = 1.0 - beta1 ** t
    c2 = 1.0 - beta2 ** t
    m *= beta1
    m += (1.0 - beta1) * g
    v *= beta2
    v += (1.0 - beta2) * (g * g)
    mh = m / c1
    vh = v / c2
    p -= (lr * mh) / (np.sqrt(vh) + eps)
    return p


def calibrate(bytecode: bytes, params, obs, steps: int, lr: float, beta1: float = 0.9, beta2: float = 0.999,
              eps: float = 1e-8, threads: int = 0):
    """Adam on every lane's parameters for `steps` steps.  Returns (fitted
    params [L, P], loss of every lane before each step [steps, L])."""
    p = np.array(params, dtype=np.float64, copy=True)
    m = np.zeros_like(p)
    v = np.zeros_like(p)
    hist = np.empty((steps, p.shape[0]))
    for t in range(1, steps + 1):
        loss, g, _ = run(bytecode, p, obs, threads=threads)
        hist[t - 1] = loss
        adam_step(p, g, m, v, t, lr, beta1, beta2, eps)
    return p, hist
