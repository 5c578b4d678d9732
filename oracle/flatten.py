"""Flattened data axis -- TEST INFRASTRUCTURE ONLY (the oracle of
ndvm_grad_points; only the tests and the benchmark's CPU-baseline leg use it).

Section 3.5 batches over named axes (data, restart, cell, population) that
are flattened into one batch dimension.  Here the data axis is flattened
into the lane axis: a loss that is a scaled sum over N data points of a
per-point term, loss(theta) = scale * sum_i term(theta, point_i), is
evaluated with one lane per (parameter vector, data point) pair; each lane
runs the per-point term program on its own point's observation row, and a
reduction over the points of each parameter vector gives its loss and
gradient.  The reduction is defined here, and the GPU follows it:

    loss[l]    = scale * ((((0 + t_0) + t_1) + ...) + t_{N-1})
    grad[l, p] = scale * ((((0 + g_0p) + g_1p) + ...) + g_{N-1,p})

a left fold over the points in ascending order, one IEEE addition per term,
then one multiplication by scale; t_i and g_i are the term's value and
gradient (seed 1) along lane (l, i)'s realized trace, from the oracle's own
per-lane interpreter (oracle.run).  The fold is written out as a loop over
points (vectorised over parameter vectors only), never as a library sum
whose order is unspecified.
"""
from __future__ import annotations

import numpy as np

from . import run


def run_points(term_bytecode: bytes, params, points, scale: float, grad: bool = True, threads: int = 0):
    """Return (loss[L], grad[L, P] or None) of the flattened loss.

    params: [L, P]; points: [N, D], row i the observations of data point i
    (D = the term program's observation count)."""
    params = np.ascontiguousarray(params, dtype=np.float64)
    points = np.ascontiguousarray(points, dtype=np.float64)
    L, P = params.shape
    N = points.shape[0]
    acc_l = np.zeros(L)
    acc_g = np.zeros((L, P)) if grad else None
    for i in range(N):
        t, g, _ = run(term_bytecode, params, points[i], grad=grad, threads=threads)
        acc_l = acc_l + t
        if grad:
            acc_g = acc_g + g
    loss = acc_l * scale
    return loss, (acc_g * scale if grad else None)
