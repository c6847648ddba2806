"""Comparison helpers for GPU-vs-oracle parity (tolerances of the build target:
loss relative error <= 1e-4, potentials absolute error <= 1e-3 after fixing the
additive gauge, gradients relative error <= 1e-3)."""
from __future__ import annotations

import numpy as np

LOSS_RTOL = 1e-4
POT_ATOL = 1e-3
GRAD_RTOL = 1e-3


def gauge_fixed_errors(mu, nu, a_gpu, b_gpu, a_ref, b_ref):
    """Max abs difference of (alpha, beta) after removing the gauge shift
    (alpha + c, beta - c give the same plan): c = mean over the support of mu
    of alpha_gpu - alpha_ref, per sample.  -inf entries must coincide."""
    ea = eb = 0.0
    for k in range(mu.shape[0]):
        sa = mu[k] > 0
        sb = nu[k] > 0
        assert np.all(np.isneginf(a_gpu[k][~sa])) and np.all(np.isneginf(a_ref[k][~sa]))
        assert np.all(np.isneginf(b_gpu[k][~sb])) and np.all(np.isneginf(b_ref[k][~sb]))
        assert np.all(np.isfinite(a_gpu[k][sa])) and np.all(np.isfinite(b_gpu[k][sb]))
        c = float(np.mean(a_gpu[k][sa].astype(np.float64) - a_ref[k][sa]))
        ea = max(ea, float(np.max(np.abs(a_gpu[k][sa] - c - a_ref[k][sa]))))
        eb = max(eb, float(np.max(np.abs(b_gpu[k][sb] + c - b_ref[k][sb]))))
    return ea, eb


def rel_err_rows(x, ref):
    """max over samples of ||x_b - ref_b||_2 / ||ref_b||_2 (flattened per sample)."""
    x = np.asarray(x, dtype=np.float64).reshape(ref.shape[0], -1)
    ref = np.asarray(ref, dtype=np.float64).reshape(ref.shape[0], -1)
    num = np.linalg.norm(x - ref, axis=1)
    den = np.linalg.norm(ref, axis=1)
    den = np.where(den > 0, den, 1.0)
    return float(np.max(num / den))


def loss_rel_err(loss, ref):
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(np.asarray(loss, dtype=np.float64) - ref) / np.maximum(np.abs(ref), 1e-30)))


def max_abs_rel_rows(x, ref):
    """max over samples of max|x_b - ref_b| / max|ref_b| (flattened per sample):
    the elementwise companion of rel_err_rows."""
    x = np.asarray(x, dtype=np.float64).reshape(ref.shape[0], -1)
    ref = np.asarray(ref, dtype=np.float64).reshape(ref.shape[0], -1)
    num = np.max(np.abs(x - ref), axis=1)
    den = np.max(np.abs(ref), axis=1)
    den = np.where(den > 0, den, 1.0)
    return float(np.max(num / den))
