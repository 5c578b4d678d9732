"""PyTorch integration on top of the binding: an autograd function whose
forward is one ndvm_grad replay (loss and exact gradient of every lane in one
launch) and a calibration loop in which Adam (ndvm_adam_step) drives
ndvm_grad with the tape uploaded once, as in the paper's Kalman
maximum-likelihood fit (Section "From buckets to phases").  All arithmetic of
the replay and of the optimiser runs in the library's kernels; torch supplies
device memory and streams (and, for autograd, the chain rule of the caller's
own graph)."""
from __future__ import annotations

import torch

from . import Tape, _launch_stream, adam_step, grad


class ReplayLoss(torch.autograd.Function):
    """loss[L] = E(P, params[l]) per lane; backward scales each lane's exact
    gradient (computed in the forward replay) by the incoming loss gradient."""

    @staticmethod
    def forward(ctx, params, tape: Tape, obs, workspace=None):
        loss, g = grad(tape, params.detach(), obs, workspace=workspace)
        ctx.save_for_backward(g)
        return loss

    @staticmethod
    def backward(ctx, g_loss):
        (g,) = ctx.saved_tensors
        return g_loss.unsqueeze(1) * g, None, None, None


def replay_loss(tape: Tape, params, obs, workspace=None):
    """Per-lane loss with autograd support (see ReplayLoss)."""
    return ReplayLoss.apply(params, tape, obs, workspace)


def calibrate(tape: Tape, params, obs, steps: int, lr: float, beta1: float = 0.9, beta2: float = 0.999,
              eps: float = 1e-8, workspace=None, stream=None):
    """Fit every lane's parameters with `steps` Adam steps, in place.
    Returns the loss of every lane before each step, [steps, L]."""
    L, P = params.shape
    dev = params.device
    s = _launch_stream(stream, dev)
    # moments and buffers are allocated and zeroed on the stream the replay
    # and the optimiser steps run on, so the fills are ordered before them
    with torch.cuda.stream(s):
        m = torch.zeros((L, P), dtype=torch.float64, device=dev)
        v = torch.zeros((L, P), dtype=torch.float64, device=dev)
        g = torch.empty((L, P), dtype=torch.float64, device=dev)
        hist = torch.empty((steps, L), dtype=torch.float64, device=dev)
        for t in range(1, steps + 1):
            grad(tape, params, obs, loss=hist[t - 1], grad_out=g, workspace=workspace, stream=s)
            adam_step(params, g, m, v, t, lr, beta1, beta2, eps, stream=s)
    return hist
