"""autograd wrapper: the loss E^0 with the Lagrange-multiplier gradient.

Section 5 of the paper: the forward returns E^0(P) = sum P C at the
approximate minimiser of E^lambda, the backward returns the gradient of
E^lambda obtained from the multipliers (Section 2), not the gradient of E^0.
"""
from __future__ import annotations

import torch

from ._binding import (sinkhorn_backward, sinkhorn_backward_points, sinkhorn_backward_sharp, sinkhorn_forward,
                       sinkhorn_forward_points)


class SinkhornLoss(torch.autograd.Function):
    @staticmethod
    def forward(ctx, mu, nu, C, lam, n_iter, tol, sharp=False, alpha0=None):
        out = sinkhorn_forward(mu.contiguous(), nu.contiguous(), C.contiguous(), lam, n_iter, tol,
                               alpha0=None if alpha0 is None else alpha0.detach().contiguous())
        ctx.save_for_backward(mu, nu, C, out["alpha"], out["beta"])
        ctx.lam = lam
        ctx.sharp = sharp
        ctx.mark_non_differentiable(out["alpha"], out["beta"], out["marg_err"], out["iters"])
        return out["loss"], out["alpha"], out["beta"], out["marg_err"], out["iters"]

    @staticmethod
    def backward(ctx, grad_loss, *unused):
        mu, nu, C, alpha, beta = ctx.saved_tensors
        want_C = ctx.needs_input_grad[2]
        if ctx.sharp:
            if want_C:
                raise NotImplementedError("the sharp gradient is taken with respect to mu and nu only")
            g = sinkhorn_backward_sharp(grad_loss.contiguous(), mu.contiguous(), nu.contiguous(), C.contiguous(),
                                        ctx.lam, alpha, beta)
            return g["grad_mu"], g["grad_nu"], None, None, None, None, None, None
        g = sinkhorn_backward(grad_loss.contiguous(), mu.contiguous(), nu.contiguous(), C.contiguous(), ctx.lam,
                              alpha, beta, grad_C=want_C)
        gC = None
        if want_C:
            gC = g["grad_C"].reshape(C.shape) if C.dim() == 3 or g["grad_C"].shape[0] == 1 else g["grad_C"]
            gC = gC.reshape(C.shape)
        return g["grad_mu"], g["grad_nu"], gC, None, None, None, None, None


def sinkhorn_loss(mu, nu, C, lam, n_iter, tol=0.0, return_state=False, sharp=False, alpha0=None):
    """Per-sample loss E^0 [B]; differentiable w.r.t. mu, nu and C.  By default
    the backward is the multiplier gradient of E^lambda (Section 5's choice);
    sharp=True differentiates E^0 itself through the plan (mu and nu only).
    alpha0 [B, d1] (optional): warm start of the iteration, e.g. from the
    state of the previous step (return_state=True), treated as a constant."""
    loss, alpha, beta, merr, iters = SinkhornLoss.apply(mu, nu, C, lam, n_iter, tol, sharp, alpha0)
    if return_state:
        return loss, dict(alpha=alpha, beta=beta, marg_err=merr, iters=iters)
    return loss


class SinkhornPointsLoss(torch.autograd.Function):
    """The same loss with the cost given by point clouds, C_ij = |X_i - Y_j|^2;
    the gradient reaches the points through dW/dC = P (chain rule)."""

    @staticmethod
    def forward(ctx, mu, nu, X, Y, lam, n_iter, tol):
        out = sinkhorn_forward_points(mu.contiguous(), nu.contiguous(), X.contiguous(), Y.contiguous(), lam, n_iter,
                                      tol)
        ctx.save_for_backward(mu, nu, X, Y, out["alpha"], out["beta"])
        ctx.lam = lam
        ctx.mark_non_differentiable(out["alpha"], out["beta"], out["marg_err"], out["iters"])
        return out["loss"], out["alpha"], out["beta"], out["marg_err"], out["iters"]

    @staticmethod
    def backward(ctx, grad_loss, *unused):
        mu, nu, X, Y, alpha, beta = ctx.saved_tensors
        want = ctx.needs_input_grad[2] or ctx.needs_input_grad[3]
        g = sinkhorn_backward_points(grad_loss.contiguous(), mu.contiguous(), nu.contiguous(), X.contiguous(),
                                     Y.contiguous(), ctx.lam, alpha, beta, grad_points=want)
        gX = g["grad_X"].reshape(X.shape) if want and ctx.needs_input_grad[2] else None
        gY = g["grad_Y"].reshape(Y.shape) if want and ctx.needs_input_grad[3] else None
        return g["grad_mu"], g["grad_nu"], gX, gY, None, None, None


def sinkhorn_loss_points(mu, nu, X, Y, lam, n_iter, tol=0.0, return_state=False):
    """Per-sample loss E^0 [B] for point clouds; differentiable w.r.t. mu, nu, X and Y."""
    loss, alpha, beta, merr, iters = SinkhornPointsLoss.apply(mu, nu, X, Y, lam, n_iter, tol)
    if return_state:
        return loss, dict(alpha=alpha, beta=beta, marg_err=merr, iters=iters)
    return loss
