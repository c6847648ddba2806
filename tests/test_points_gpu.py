"""GPU parity of the point-cloud entry points (cost C_ij = |X_i - Y_j|^2 given by
coordinates) through the C ABI, against the fp64 oracle run on the cost the
oracle builds from the same fp32 coordinates.  Tolerances as for a cost
matrix: loss relative error <= 1e-4, potentials absolute error <= 1e-3 after
fixing the gauge, gradients (mu, nu and the points) relative error <= 1e-3."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_1907_01729_amd as sk
import workloads
from parity_util import GRAD_RTOL, LOSS_RTOL, POT_ATOL, gauge_fixed_errors, loss_rel_err, rel_err_rows

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _gpu(prob):
    out = sk.sinkhorn_forward_points(_t(prob.mu), _t(prob.nu), _t(prob.X), _t(prob.Y), prob.lam, prob.n_iter,
                                     prob.tol)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def _clouds(prob, idx):
    if prob.c_batched:
        return prob.X[idx], prob.Y[idx]
    return prob.X, prob.Y


def check_points(prob, idx=None, merr_atol=2e-5, merr_rtol=5e-2, grads=True, seed=0):
    _say(f"[points] {prob.name} B={prob.B} d1={prob.d1} d2={prob.d2} D={prob.D} lam={prob.lam} "
         f"n_iter={prob.n_iter} tol={prob.tol} batched={prob.c_batched}")
    gpu = _gpu(prob)
    if idx is None:
        idx = np.arange(prob.B)
    X, Y = _clouds(prob, idx)
    C = oracle.cost_from_points(X, Y)
    mu, nu = prob.mu[idx], prob.nu[idx]
    iters = gpu["iters"][idx]
    if prob.tol > 0:
        free = oracle.forward(mu, nu, C, prob.lam, prob.n_iter, tol=prob.tol)
        assert np.all(np.abs(free["iters"] - iters) <= 1), (free["iters"], iters)
        ref = oracle.forward(mu, nu, C, prob.lam, prob.n_iter, n_iter_b=iters)
    else:
        assert np.all(iters == prob.n_iter), iters
        ref = oracle.forward(mu, nu, C, prob.lam, prob.n_iter)
    el = loss_rel_err(gpu["loss"][idx], ref["loss"])
    ea, eb = gauge_fixed_errors(mu, nu, gpu["alpha"][idx], gpu["beta"][idx], ref["alpha"], ref["beta"])
    dm = np.abs(gpu["marg_err"][idx] - ref["marg_err"])
    _say(f"   loss rel {el:.2e}  alpha {ea:.2e}  beta {eb:.2e}  marg_err |d| max {dm.max():.2e}")
    assert el <= LOSS_RTOL
    assert ea <= POT_ATOL and eb <= POT_ATOL
    assert np.all(dm <= merr_atol + merr_rtol * ref["marg_err"])
    if not grads:
        return gpu, ref
    rng = np.random.default_rng(seed)
    g = rng.uniform(0.5, 1.5, size=prob.B).astype(np.float32)
    out = sk.sinkhorn_backward_points(_t(g), _t(prob.mu), _t(prob.nu), _t(prob.X), _t(prob.Y), prob.lam,
                                      _t(gpu["alpha"]), _t(gpu["beta"]), grad_points=True)
    torch.cuda.synchronize()
    r = oracle.backward(g[idx], mu, nu, C, prob.lam, ref["alpha"], ref["beta"], grad_C=True)
    e1 = rel_err_rows(out["grad_mu"].cpu().numpy()[idx], r["grad_mu"])
    e2 = rel_err_rows(out["grad_nu"].cpu().numpy()[idx], r["grad_nu"])
    if prob.c_batched:
        gX, gY = oracle.points_grads(r["grad_C"], X, Y)
        e3 = rel_err_rows(out["grad_X"].cpu().numpy()[idx], gX)
        e4 = rel_err_rows(out["grad_Y"].cpu().numpy()[idx], gY)
    else:
        assert len(idx) == prob.B, "shared clouds: the point gradients sum the whole batch"
        gX, gY = oracle.points_grads(r["grad_C"], X, Y)
        e3 = rel_err_rows(out["grad_X"].cpu().numpy().reshape(gX.shape), gX)
        e4 = rel_err_rows(out["grad_Y"].cpu().numpy().reshape(gY.shape), gY)
    _say(f"   grad_mu {e1:.2e}  grad_nu {e2:.2e}  grad_X {e3:.2e}  grad_Y {e4:.2e}")
    assert max(e1, e2, e3, e4) <= GRAD_RTOL
    return gpu, ref


# ---------------------------------------------------------------- on-the-fly sweep (tiled, per-sample)

@pytest.mark.parametrize("d1,d2,D", [(256, 520, 3), (300, 129, 2), (129, 1000, 1), (200, 2048, 3), (1500, 70, 3),
                                     (131, 257, 2)])
def test_points_on_the_fly_shapes(d1, d2, D):
    prob = workloads.random_points(100 + d1 + d2 + D, B=3, d1=d1, d2=d2, D=D, lam=0.1, n_iter=30)
    assert sk.sinkhorn_regime(prob.B, d1, d2, 1) == 2
    check_points(prob)


def test_points_zero_masses():
    prob = workloads.random_points(51, B=4, d1=150, d2=300, D=3, lam=0.05, n_iter=50, zero_frac=0.2)
    assert (prob.mu == 0).any() and (prob.nu == 0).any()
    gpu, _ = check_points(prob)
    assert np.all(np.isneginf(gpu["alpha"][prob.mu == 0]))


def test_points_early_stop_per_sample():
    prob = workloads.random_points(52, B=5, d1=200, d2=260, D=2, lam=0.2, n_iter=400, tol=1e-4)
    gpu, _ = check_points(prob, grads=False)
    assert np.all(gpu["iters"] < 400) and len(set(gpu["iters"].tolist())) > 1


def test_points_small_lambda_exact_paths():
    """lambda small against the spread of the clouds (cost/lambda up to ~10^3):
    the sweep's exact logsumexp fallbacks recompute the cost from the points."""
    prob = workloads.random_points(53, B=2, d1=160, d2=384, D=3, lam=0.01, n_iter=60)
    check_points(prob, merr_atol=1e-4)


def test_points_translated_clouds():
    """Both clouds moved by 10 in every coordinate: the cost is translation
    invariant and computed from differences, so parity holds."""
    prob = workloads.random_points(54, B=2, d1=140, d2=300, D=3, lam=0.1, n_iter=40, offset=10.0)
    check_points(prob)


def test_points_clouds_full_size_sampled():
    """The point-cloud workload at full size (B=32, 1024 x 2048, D=3, 100
    iterations) with the cost never stored; oracle on two problems."""
    prob = workloads.clouds_points()
    check_points(prob, idx=np.array([0, 31]))


def test_points_matches_cost_matrix_path():
    """The on-the-fly sweep and the same problem with the cost written out
    (fp32 C from the same points) agree to the parity tolerances."""
    prob = workloads.random_points(55, B=3, d1=256, d2=512, D=3, lam=0.1, n_iter=50)
    a = _gpu(prob)
    C = oracle.cost_from_points(prob.X, prob.Y).astype(np.float32)
    b = sk.sinkhorn_forward(_t(prob.mu), _t(prob.nu), _t(C), prob.lam, prob.n_iter)
    b = {k: v.cpu().numpy() for k, v in b.items()}
    assert loss_rel_err(a["loss"], b["loss"].astype(np.float64)) <= LOSS_RTOL
    ea, eb = gauge_fixed_errors(prob.mu, prob.nu, a["alpha"], a["beta"], b["alpha"].astype(np.float64),
                                b["beta"].astype(np.float64))
    assert ea <= POT_ATOL and eb <= POT_ATOL


# ---------------------------------------------------------------- shapes that write the cost out first

@pytest.mark.parametrize("d1,d2,D,batched", [(50, 60, 3, True), (100, 100, 2, False), (300, 400, 3, False),
                                             (150, 2100, 2, True), (200, 300, 5, True), (7, 1, 3, True)])
def test_points_materialized_paths(d1, d2, D, batched):
    prob = workloads.random_points(200 + d1 + d2 + D, B=3, d1=d1, d2=d2, D=D, lam=0.1, n_iter=30,
                                   batched=batched)
    check_points(prob)


def test_points_autograd_wrapper():
    prob = workloads.random_points(56, B=3, d1=140, d2=200, D=3, lam=0.1, n_iter=60)
    mu = _t(prob.mu).requires_grad_()
    nu = _t(prob.nu).requires_grad_()
    X = _t(prob.X).requires_grad_()
    Y = _t(prob.Y).requires_grad_()
    loss = sk.sinkhorn_loss_points(mu, nu, X, Y, prob.lam, prob.n_iter)
    (loss * torch.arange(1, 4, device=DEV)).sum().backward()
    C = oracle.cost_from_points(prob.X, prob.Y)
    ref = oracle.forward(prob.mu, prob.nu, C, prob.lam, prob.n_iter)
    r = oracle.backward(np.arange(1, 4), prob.mu, prob.nu, C, prob.lam, ref["alpha"], ref["beta"], grad_C=True)
    gX, gY = oracle.points_grads(r["grad_C"], prob.X, prob.Y)
    assert rel_err_rows(mu.grad.cpu().numpy(), r["grad_mu"]) <= GRAD_RTOL
    assert rel_err_rows(nu.grad.cpu().numpy(), r["grad_nu"]) <= GRAD_RTOL
    assert rel_err_rows(X.grad.cpu().numpy(), gX) <= GRAD_RTOL
    assert rel_err_rows(Y.grad.cpu().numpy(), gY) <= GRAD_RTOL


def test_points_invalid_dimension():
    prob = workloads.random_points(57, B=2, d1=10, d2=12, D=17, lam=0.1, n_iter=5)
    with pytest.raises(sk.SinkhornError):
        _gpu(prob)


def test_points_batch_above_grid_limit():
    """65537 per-sample clouds of a tiled shape through the on-the-fly sweep,
    run as two chunks of the batch: problems on both sides of the boundary
    against the oracle, with the point gradients."""
    prob = workloads.random_points(seed=93, B=65537, d1=130, d2=8, D=3, lam=0.2, n_iter=30)
    check_points(prob, idx=np.array([0, 65534, 65535, 65536]))
