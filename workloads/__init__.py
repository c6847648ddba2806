"""Seeded synthetic inputs for batched Sinkhorn (shared by tests, smoke and bench).

This module only draws inputs -- histograms and cost matrices -- with numpy's
``default_rng``.  It holds none of the method's arithmetic, so both the GPU
library's callers and the fp64 oracle can consume the identical arrays.

Every generator draws in float64, renormalises probability vectors in float64,
then casts to float32; both sides consume the float32 arrays (the oracle
upcasts them).

The paper names no dataset.  The five workloads stand in for its use cases
(label-space losses over ~100 classes, image histograms, large grids at small
lambda, and point clouds with per-sample costs).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass
class Problem:
    name: str
    mu: np.ndarray        # [B, d1] float32
    nu: np.ndarray        # [B, d2] float32
    C: np.ndarray         # [1 or B, d1, d2] float32
    lam: float
    n_iter: int
    tol: float = 0.0
    grad_C: bool = False

    @property
    def B(self):
        return self.mu.shape[0]

    @property
    def d1(self):
        return self.mu.shape[1]

    @property
    def d2(self):
        return self.nu.shape[1]

    @property
    def c_batched(self):
        return self.C.shape[0] != 1


def _softmax_rows(z):
    z = z - z.max(axis=1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=1, keepdims=True)


def _normalise(p):
    return p / p.sum(axis=-1, keepdims=True)


def grid_points(side):
    """Pixel coordinates (r, c) of a side x side grid, flattened as side*r + c."""
    r, c = np.meshgrid(np.arange(side), np.arange(side), indexing="ij")
    return np.stack([r.ravel(), c.ravel()], axis=1).astype(np.float64)


def sq_dists(x, y):
    return ((x[:, None, :] - y[None, :, :]) ** 2).sum(-1)


def blob_histograms(rng, B, side, n_blobs=3, floor=1e-6):
    """B histograms on a side x side grid: equal-weight mixtures of n_blobs
    normalised isotropic 2-D Gaussian densities, centres U[0, side]^2,
    sigma U[1, 4]; then normalised, a floor added, renormalised."""
    pts = grid_points(side)
    out = np.empty((B, side * side))
    for b in range(B):
        centres = rng.uniform(0.0, side, size=(n_blobs, 2))
        sig = rng.uniform(1.0, 4.0, size=n_blobs)
        h = np.zeros(side * side)
        for k in range(n_blobs):
            d2 = ((pts - centres[k]) ** 2).sum(1)
            h += np.exp(-d2 / (2 * sig[k] ** 2)) / (2 * np.pi * sig[k] ** 2)
        p = h / h.sum() + floor
        out[b] = p / p.sum()
    return out


def tiny(seed=1001, B=4, d=10, n_iter=100):
    """Tiny: softmax(N(0,1)) histograms, C_ij = ((i-j)/(d-1))^2, lambda 0.1."""
    rng = np.random.default_rng(seed)
    mu = _softmax_rows(rng.standard_normal((B, d)))
    nu = _softmax_rows(rng.standard_normal((B, d)))
    i = np.arange(d, dtype=np.float64)
    C = ((i[:, None] - i[None, :]) / (d - 1)) ** 2
    return Problem("tiny", mu.astype(np.float32), nu.astype(np.float32),
                   C[None].astype(np.float32), 0.1, n_iter)


def label(seed=1002, B=1024, d=100, n_iter=200):
    """Label space: softmax(2 N(0,1)) histograms over d classes, C = squared
    distances between d class embeddings drawn U[0,1]^2, lambda 0.05."""
    rng = np.random.default_rng(seed)
    mu = _softmax_rows(2.0 * rng.standard_normal((B, d)))
    nu = _softmax_rows(2.0 * rng.standard_normal((B, d)))
    e = rng.uniform(0.0, 1.0, size=(d, 2))
    C = sq_dists(e, e)
    return Problem("label", mu.astype(np.float32), nu.astype(np.float32),
                   C[None].astype(np.float32), 0.05, n_iter)


def image(seed=1003, B=256, side=28, n_iter=300, lam=0.01):
    """Image histograms on a side x side grid (blob mixtures + 1e-6 floor),
    C = squared grid distance / (side-1)^2, lambda 0.01."""
    rng = np.random.default_rng(seed)
    mu = blob_histograms(rng, B, side)
    nu = blob_histograms(rng, B, side)
    pts = grid_points(side)
    C = sq_dists(pts, pts) / float(side - 1) ** 2
    return Problem(f"image{side}", mu.astype(np.float32), nu.astype(np.float32),
                   C[None].astype(np.float32), lam, n_iter)


def grid(seed=1004, B=64, side=64, n_iter=500, lam=1e-3, tol=1e-6):
    """Large grid at small lambda: the image generator on side x side,
    C = squared grid distance / (side-1)^2, lambda 1e-3, early stop tol."""
    p = image(seed=seed, B=B, side=side, n_iter=n_iter, lam=lam)
    p.name = f"grid{side}"
    p.tol = tol
    return p


def clouds(seed=1005, B=32, d1=1024, d2=2048, n_iter=100, lam=0.05):
    """Per-sample point clouds: x ~ N(0, I_3)^d1, y ~ N(0, I_3)^d2 + s_b with
    one shift s_b ~ N(0, I_3) per sample; C_b = squared Euclidean distances
    (per sample, [B, d1, d2]); uniform mu, nu; lambda 0.05; grad_C wanted."""
    rng = np.random.default_rng(seed)
    C = np.empty((B, d1, d2), dtype=np.float32)
    for b in range(B):
        x = rng.standard_normal((d1, 3))
        y = rng.standard_normal((d2, 3))
        s = rng.standard_normal(3)
        C[b] = sq_dists(x, y + s).astype(np.float32)
    mu = np.full((B, d1), 1.0 / d1)
    nu = np.full((B, d2), 1.0 / d2)
    return Problem("clouds", mu.astype(np.float32), nu.astype(np.float32), C, lam, n_iter,
                   grad_C=True)


@dataclass
class PointsProblem:
    """A batch whose cost is given by point clouds: C_ij = |X_i - Y_j|^2
    (X [1 or B, d1, D], Y [1 or B, d2, D]; the cost itself is not drawn)."""
    name: str
    mu: np.ndarray        # [B, d1] float32
    nu: np.ndarray        # [B, d2] float32
    X: np.ndarray         # [1 or B, d1, D] float32
    Y: np.ndarray         # [1 or B, d2, D] float32
    lam: float
    n_iter: int
    tol: float = 0.0
    grad_points: bool = False

    @property
    def B(self):
        return self.mu.shape[0]

    @property
    def d1(self):
        return self.mu.shape[1]

    @property
    def d2(self):
        return self.nu.shape[1]

    @property
    def D(self):
        return self.X.shape[2]

    @property
    def c_batched(self):
        return self.X.shape[0] != 1


def clouds_points(seed=1005, B=32, d1=1024, d2=2048, n_iter=100, lam=0.05):
    """The point-cloud workload with the cost left implicit: the same draws as
    clouds() (x ~ N(0, I_3)^d1, y ~ N(0, I_3)^d2 + s_b), stored as float32
    coordinates X[b] = x, Y[b] = y + s_b; uniform mu, nu; lambda 0.05."""
    rng = np.random.default_rng(seed)
    X = np.empty((B, d1, 3))
    Y = np.empty((B, d2, 3))
    for b in range(B):
        X[b] = rng.standard_normal((d1, 3))
        y = rng.standard_normal((d2, 3))
        Y[b] = y + rng.standard_normal(3)
    mu = np.full((B, d1), 1.0 / d1)
    nu = np.full((B, d2), 1.0 / d2)
    return PointsProblem("clouds_points", mu.astype(np.float32), nu.astype(np.float32), X.astype(np.float32),
                         Y.astype(np.float32), lam, n_iter, grad_points=True)


def random_points(seed, B, d1, d2, D, lam, n_iter, batched=True, zero_frac=0.0, tol=0.0, scale=1.0,
                  offset=0.0):
    """Generic point-cloud problem: positive histograms (optionally with a
    fraction of exact zeros, one non-zero kept per sample), X ~ scale*N(0,I_D)
    and Y ~ scale*N(0,I_D) + scale*N(0,I_D) shift per cloud, both moved by
    `offset` (tests translation robustness)."""
    rng = np.random.default_rng(seed)
    mu = rng.uniform(0.05, 1.0, size=(B, d1))
    nu = rng.uniform(0.05, 1.0, size=(B, d2))
    if zero_frac > 0:
        for h in (mu, nu):
            z = rng.random(h.shape) < zero_frac
            z[:, 0] = False
            h[z] = 0.0
    mu, nu = _normalise(mu), _normalise(nu)
    nc = B if batched else 1
    X = scale * rng.standard_normal((nc, d1, D)) + offset
    Y = scale * (rng.standard_normal((nc, d2, D)) + rng.standard_normal((nc, 1, D))) + offset
    return PointsProblem(f"points{seed}", mu.astype(np.float32), nu.astype(np.float32), X.astype(np.float32),
                         Y.astype(np.float32), lam, n_iter, tol=tol)


CONFIGS = {
    1: tiny,
    2: label,
    3: image,
    4: grid,
    5: clouds,
}


def make_config(k, **overrides):
    """Workload k (1..5) at full size, or with keyword overrides (B, d, ...)."""
    return CONFIGS[k](**overrides)


def random_problem(seed, B, d1, d2, lam, n_iter, c_batched=False, zero_frac=0.0,
                   cost="uniform", tol=0.0):
    """Generic random problem for edge cases: positive histograms (optionally
    with a fraction of exact zeros, at least one non-zero kept per sample) and
    a non-symmetric cost U[0,1) (or 'grid1d': |x_i - y_j| on [0,1]; or 'sym':
    (U + U^T) / 2 for d1 = d2, exactly symmetric)."""
    rng = np.random.default_rng(seed)
    mu = rng.uniform(0.05, 1.0, size=(B, d1))
    nu = rng.uniform(0.05, 1.0, size=(B, d2))
    if zero_frac > 0:
        for h in (mu, nu):
            z = rng.random(h.shape) < zero_frac
            z[:, 0] = False
            h[z] = 0.0
    mu, nu = _normalise(mu), _normalise(nu)
    nC = B if c_batched else 1
    if cost == "uniform":
        C = rng.uniform(0.0, 1.0, size=(nC, d1, d2))
    elif cost == "sym":
        assert d1 == d2, "a symmetric cost needs d1 == d2"
        U = rng.uniform(0.0, 1.0, size=(nC, d1, d2))
        C = 0.5 * (U + np.swapaxes(U, 1, 2))
    elif cost == "grid1d":
        x = np.linspace(0.0, 1.0, d1)
        y = np.linspace(0.0, 1.0, d2)
        C = np.broadcast_to(np.abs(x[:, None] - y[None, :]), (nC, d1, d2)).copy()
    else:
        raise ValueError(cost)
    return Problem(f"random{seed}", mu.astype(np.float32), nu.astype(np.float32),
                   C.astype(np.float32), lam, n_iter, tol=tol)
