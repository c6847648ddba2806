"""fp64 CPU oracle for batched log-domain Sinkhorn -- TEST INFRASTRUCTURE ONLY.

Loads ``libsinkhorn_oracle.so`` (plain C + OpenMP, built from
``sinkhorn_oracle.c`` by :func:`build`).  Only the test suite, the smoke check
and the benchmark's CPU-baseline leg may import this package; the GPU library
never does, and the two share no code.

Arrays are numpy; every input is upcast to float64 before the call, so the GPU
path and the oracle consume the identical (fp32) values.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sinkhorn_oracle.c")
_LIB = os.path.join(_HERE, "libsinkhorn_oracle.so")
_lib = None


def build(verbose: bool = False) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, IEEE semantics: no fast-math)."""
    tmp = _LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I = ctypes.c_int
        D = ctypes.c_double
        lib.oracle_forward.argtypes = [I, I, I, I, D, I, D, P, P, P, P, P, P, P, P, P, P, P]
        lib.oracle_forward.restype = I
        lib.oracle_backward.argtypes = [I, I, I, I, D, P, P, P, P, P, P, P, P, P]
        lib.oracle_backward.restype = I
        lib.oracle_objectives.argtypes = [I, I, D, P, P, P, P, P, P]
        lib.oracle_objectives.restype = I
        lib.oracle_plan.argtypes = [I, I, D, P, P, P, P]
        lib.oracle_plan.restype = I
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = I
        _lib = lib
    return _lib


def _f64(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _shapes(mu, nu, C):
    mu, nu, C = _f64(mu), _f64(nu), _f64(C)
    if mu.ndim == 1:
        mu = mu[None]
    if nu.ndim == 1:
        nu = nu[None]
    if C.ndim == 2:
        C = C[None]
    B, d1 = mu.shape
    B2, d2 = nu.shape
    if B2 != B or C.shape[1:] != (d1, d2) or C.shape[0] not in (1, B):
        raise ValueError(f"shape mismatch mu{mu.shape} nu{nu.shape} C{C.shape}")
    c_batched = int(C.shape[0] == B and B != 1)
    return mu, nu, C, B, d1, d2, c_batched


def num_threads() -> int:
    return _load().oracle_num_threads()


def forward(mu, nu, C, lam, n_iter, tol=0.0, n_iter_b=None, err_hist=False, alpha0=None):
    """Log-domain Sinkhorn forward in fp64.

    Returns a dict with alpha [B,d1], beta [B,d2] (log u, log v), loss [B]
    (E^0 = sum P C), marg_err [B] (||P1-mu||_1 + ||P^T1-nu||_1), iters [B]
    and, if requested, err_hist [B, n_iter].  alpha0 [B,d1] (optional): a
    warm start, log u^0 on the support of mu instead of 0 (the iteration's
    whole state, since each iteration begins with the v-update from log u).
    """
    mu, nu, C, B, d1, d2, cb = _shapes(mu, nu, C)
    a0 = None
    if alpha0 is not None:
        a0 = np.ascontiguousarray(np.asarray(alpha0, dtype=np.float64).reshape(B, d1))
    alpha = np.empty((B, d1))
    beta = np.empty((B, d2))
    loss = np.empty(B)
    merr = np.empty(B)
    iters = np.empty(B, dtype=np.int32)
    nb = None
    if n_iter_b is not None:
        nb = np.ascontiguousarray(np.asarray(n_iter_b, dtype=np.int32).reshape(B))
        n_iter = int(nb.max()) if B else 0
    hist = np.empty((B, max(n_iter, 1))) if err_hist else None
    rc = _load().oracle_forward(B, d1, d2, cb, float(lam), int(n_iter), float(tol), _ptr(nb),
                                _ptr(mu), _ptr(nu), _ptr(C), _ptr(alpha), _ptr(beta),
                                _ptr(loss), _ptr(merr), _ptr(iters), _ptr(hist), _ptr(a0))
    if rc != 0:
        raise ValueError("oracle_forward: invalid arguments")
    out = dict(alpha=alpha, beta=beta, loss=loss, marg_err=merr, iters=iters)
    if err_hist:
        out["err_hist"] = hist[:, :n_iter]
    return out


def backward(grad_loss, mu, nu, C, lam, alpha, beta, grad_C=False):
    """Multiplier gradient (Section 2) in fp64: grad_mu, grad_nu, optional grad_C."""
    mu, nu, C, B, d1, d2, cb = _shapes(mu, nu, C)
    g = _f64(grad_loss).reshape(B)
    alpha = _f64(alpha).reshape(B, d1)
    beta = _f64(beta).reshape(B, d2)
    gmu = np.empty((B, d1))
    gnu = np.empty((B, d2))
    gC = np.empty(C.shape) if grad_C else None
    rc = _load().oracle_backward(B, d1, d2, cb, float(lam), _ptr(g), _ptr(mu), _ptr(nu), _ptr(C),
                                 _ptr(alpha), _ptr(beta), _ptr(gmu), _ptr(gnu), _ptr(gC))
    if rc != 0:
        raise ValueError("oracle_backward: invalid arguments")
    out = dict(grad_mu=gmu, grad_nu=gnu)
    if grad_C:
        out["grad_C"] = gC
    return out


def objectives(mu, nu, C, lam, alpha, beta):
    """One sample: dict(dual, primal, e0, entropy) of the plan built from (alpha, beta)."""
    mu, nu, C = _f64(mu).ravel(), _f64(nu).ravel(), _f64(C).reshape(len(mu), -1)
    out = np.empty(4)
    rc = _load().oracle_objectives(len(mu), len(nu), float(lam), _ptr(mu), _ptr(nu), _ptr(C),
                                   _ptr(_f64(alpha).ravel()), _ptr(_f64(beta).ravel()), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_objectives: invalid arguments")
    return dict(dual=out[0], primal=out[1], e0=out[2], entropy=out[3])


def plan(C, lam, alpha, beta):
    """One sample: P = exp(alpha_i + beta_j - C_ij / lam) as a [d1, d2] array."""
    alpha, beta = _f64(alpha).ravel(), _f64(beta).ravel()
    C = _f64(C).reshape(len(alpha), len(beta))
    P = np.empty_like(C)
    rc = _load().oracle_plan(len(alpha), len(beta), float(lam), _ptr(C), _ptr(alpha), _ptr(beta), _ptr(P))
    if rc != 0:
        raise ValueError("oracle_plan: invalid arguments")
    return P


# ---- point clouds ----

def cost_from_points(X, Y):
    """Squared Euclidean cost by its definition, C_ij = sum_k (X_ik - Y_jk)^2,
    in fp64 (differences first, no expansion).  X [nb, d1, D] or [d1, D],
    Y [nb, d2, D] or [d2, D]  ->  C [nb, d1, d2]."""
    X, Y = _f64(X), _f64(Y)
    if X.ndim == 2:
        X = X[None]
    if Y.ndim == 2:
        Y = Y[None]
    C = np.empty((X.shape[0], X.shape[1], Y.shape[1]))
    for b in range(X.shape[0]):  # one cloud pair at a time: bounded memory
        diff = X[b][:, None, :] - Y[b][None, :, :]
        C[b] = (diff * diff).sum(-1)
    return C


def points_grads(G, X, Y):
    """Chain rule through C_ij = |X_i - Y_j|^2 for a cost gradient G = dW/dC
    [nb, d1, d2]: grad_X_i = sum_j G_ij 2 (X_i - Y_j), grad_Y_j = sum_i G_ij
    2 (Y_j - X_i), per cloud pair, in fp64."""
    X, Y, G = _f64(X), _f64(Y), _f64(G)
    if X.ndim == 2:
        X = X[None]
    if Y.ndim == 2:
        Y = Y[None]
    if G.ndim == 2:
        G = G[None]
    gX = np.empty_like(X)
    gY = np.empty_like(Y)
    for b in range(X.shape[0]):
        gX[b] = 2.0 * (G[b].sum(1)[:, None] * X[b] - G[b] @ Y[b])
        gY[b] = 2.0 * (G[b].sum(0)[:, None] * Y[b] - G[b].T @ X[b])
    return gX, gY


# ---- gradient of the sharp loss E^0 (implicit differentiation) ----

def sharp_gradient(grad_loss, mu, nu, C, lam, alpha, beta):
    """Gradient of E^0 = <P, C> with respect to (mu, nu), where P is the
    entropic plan, differentiated through its optimality conditions (the
    sharper gradient Section 5 points to), in fp64 with a dense solve.

    With P built from (alpha, beta), r = P 1, c = P^T 1, a = (P o C) 1 and
    b = (P o C)^T 1, a change (dmu, dnu) of the marginals moves the plan by
    dP_ij = P_ij (df_i + dg_j) / lambda with
        [diag(r)  P      ] [df]            [dmu]
        [P^T      diag(c)] [dg] = lambda * [dnu],
    and dE^0 = (1/lambda) (<a, df> + <b, dg>).  Hence dE^0 = <z, (dmu, dnu)>
    for the solution z of the same symmetric system with right-hand side
    (a, b).  The system is singular along (1, -1) (a constant moved from f to
    g); on the simplex the gradient is defined up to a constant per block, so
    z is taken by least squares and each block centred over its support (0
    off it), the convention of the multiplier gradient.  Scaled by
    grad_loss per problem.  Returns dict(grad_mu [B, d1], grad_nu [B, d2])."""
    mu, nu, C, B, d1, d2, cb = _shapes(mu, nu, C)
    g = _f64(grad_loss).reshape(B)
    alpha = _f64(alpha).reshape(B, d1)
    beta = _f64(beta).reshape(B, d2)
    gmu = np.zeros((B, d1))
    gnu = np.zeros((B, d2))
    for b in range(B):
        Cb = C[b if cb else 0]
        P = plan(Cb, lam, alpha[b], beta[b])
        si, sj = mu[b] > 0, nu[b] > 0
        Ps, Cs = P[np.ix_(si, sj)], Cb[np.ix_(si, sj)]
        n1, n2 = Ps.shape
        H = np.zeros((n1 + n2, n1 + n2))
        H[:n1, :n1] = np.diag(Ps.sum(1))
        H[n1:, n1:] = np.diag(Ps.sum(0))
        H[:n1, n1:] = Ps
        H[n1:, :n1] = Ps.T
        rhs = np.concatenate([(Ps * Cs).sum(1), (Ps * Cs).sum(0)])
        z = np.linalg.lstsq(H, rhs, rcond=None)[0]
        zf, zg = z[:n1], z[n1:]
        gmu[b, si] = g[b] * (zf - zf.mean())
        gnu[b, sj] = g[b] * (zg - zg.mean())
    return dict(grad_mu=gmu, grad_nu=gnu)
