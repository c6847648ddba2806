"""GPU parity of the warm start (sinkhorn_forward_warm): the library started
from a given alpha0 against the oracle started from the same fp32 alpha0, in
both regimes, and the resume property on the GPU itself (K iterations, then n
more from their alpha, against K + n).  Tolerances as in test_parity_gpu."""
import ctypes
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_1907_01729_amd as sk
import workloads
from paper_1907_01729_amd import _binding
from parity_util import LOSS_RTOL, POT_ATOL, gauge_fixed_errors, loss_rel_err

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _subset(prob, idx):
    return prob.mu[idx], prob.nu[idx], (prob.C[idx] if prob.c_batched else prob.C)


def check_warm(prob, a0, n_iter, idx=None, tol=0.0):
    """GPU warm start from the fp32 alpha0 against the oracle's from the same
    values, on the samples idx (all by default)."""
    _say(f"[warm] {prob.name} B={prob.B} d1={prob.d1} d2={prob.d2} lam={prob.lam} n_iter={n_iter} tol={tol}")
    a0 = np.ascontiguousarray(a0, dtype=np.float32)
    out = sk.sinkhorn_forward(_t(prob.mu), _t(prob.nu), _t(prob.C), prob.lam, n_iter, tol, alpha0=_t(a0))
    torch.cuda.synchronize()
    gpu = {k: v.cpu().numpy() for k, v in out.items()}
    if idx is None:
        idx = np.arange(prob.B)
    mu, nu, C = _subset(prob, idx)
    iters = gpu["iters"][idx]
    if tol > 0:
        free = oracle.forward(mu, nu, C, prob.lam, n_iter, tol=tol, alpha0=a0[idx])
        assert np.all(np.abs(free["iters"] - iters) <= 1), (free["iters"], iters)
        ref = oracle.forward(mu, nu, C, prob.lam, n_iter, n_iter_b=iters, alpha0=a0[idx])
    else:
        assert np.all(iters == n_iter)
        ref = oracle.forward(mu, nu, C, prob.lam, n_iter, alpha0=a0[idx])
    el = loss_rel_err(gpu["loss"][idx], ref["loss"])
    ea, eb = gauge_fixed_errors(mu, nu, gpu["alpha"][idx], gpu["beta"][idx], ref["alpha"], ref["beta"])
    dm = np.abs(gpu["marg_err"][idx] - ref["marg_err"])
    _say(f"   loss rel {el:.2e}  alpha {ea:.2e}  beta {eb:.2e}  marg_err |d| max {dm.max():.2e}")
    assert el <= LOSS_RTOL
    assert ea <= POT_ATOL and eb <= POT_ATOL
    assert np.all(dm <= 2e-5 + 5e-2 * ref["marg_err"])
    # off the support of mu the returned alpha is -inf, whatever alpha0 held
    assert np.all(np.isneginf(gpu["alpha"][idx][mu == 0]))
    return gpu


def _cold_alpha(prob, n_iter):
    return oracle.forward(prob.mu, prob.nu, prob.C, prob.lam, n_iter)["alpha"].astype(np.float32)


def test_warm_resident_label():
    prob = workloads.make_config(2, B=48)
    check_warm(prob, _cold_alpha(prob, 60), 40)


def test_warm_resident_zero_masses_garbage_off_support():
    prob = workloads.random_problem(seed=61, B=5, d1=60, d2=45, lam=0.1, n_iter=50, zero_frac=0.2, c_batched=True)
    a0 = np.random.default_rng(1).normal(0.0, 1.0, (prob.B, prob.d1))
    a0[prob.mu == 0] = 77.0
    check_warm(prob, a0, 30)


def test_warm_resident_widest_bucket_and_early_stop():
    prob = workloads.random_problem(seed=62, B=6, d1=120, d2=128, lam=0.1, n_iter=100)
    check_warm(prob, _cold_alpha(prob, 20), 100, tol=2e-4)


def test_warm_tiled_shared_image():
    prob = workloads.make_config(3, B=16)
    cold = sk.sinkhorn_forward(_t(prob.mu), _t(prob.nu), _t(prob.C), prob.lam, 60)
    a0 = cold["alpha"].cpu().numpy()
    check_warm(prob, a0, 40, idx=np.array([0, 9, 15]))


def test_warm_tiled_per_sample_streamed():
    prob = workloads.random_problem(seed=63, B=4, d1=300, d2=512, lam=0.05, n_iter=60, c_batched=True,
                                    zero_frac=0.1)
    a0 = np.random.default_rng(2).normal(0.0, 3.0, (prob.B, prob.d1))
    check_warm(prob, a0, 30)


def test_warm_tiled_wide_rows_and_early_stop():
    prob = workloads.random_problem(seed=64, B=3, d1=140, d2=5000, lam=0.1, n_iter=60)
    check_warm(prob, _cold_alpha(prob, 10), 60, tol=1e-3)


@pytest.mark.parametrize("cfg", [2, 3])
def test_warm_resume_on_the_gpu(cfg):
    """K iterations on the GPU, then n more from their alpha, against K + n:
    equal up to rounding (the first v-update of the resumed run takes the
    exact logsumexp where the continuing run took the shifted sum)."""
    prob = workloads.make_config(cfg, B=32 if cfg == 2 else 8)
    mu, nu, C = _t(prob.mu), _t(prob.nu), _t(prob.C)
    first = sk.sinkhorn_forward(mu, nu, C, prob.lam, 70)
    resumed = sk.sinkhorn_forward(mu, nu, C, prob.lam, 50, alpha0=first["alpha"])
    # the warm start runs the log-domain kernels: compare with those (resident)
    whole = sk.sinkhorn_forward_select("log" if cfg == 2 else "default", mu, nu, C, prob.lam, 120)
    torch.cuda.synchronize()
    r = {k: v.cpu().numpy() for k, v in resumed.items()}
    w = {k: v.cpu().numpy() for k, v in whole.items()}
    el = loss_rel_err(r["loss"], w["loss"])
    ea, eb = gauge_fixed_errors(prob.mu, prob.nu, r["alpha"], r["beta"], w["alpha"], w["beta"])
    _say(f"[resume {cfg}] loss rel {el:.2e}  alpha {ea:.2e}  beta {eb:.2e}")
    assert el <= LOSS_RTOL and ea <= POT_ATOL and eb <= POT_ATOL


@pytest.mark.parametrize("cfg", [2, 3])
def test_warm_in_place(cfg):
    """alpha0 may be the alpha output buffer itself: the same bits as with a
    separate buffer."""
    prob = workloads.make_config(cfg, B=16)
    mu, nu, C = _t(prob.mu), _t(prob.nu), _t(prob.C)
    a0 = sk.sinkhorn_forward(mu, nu, C, prob.lam, 30)["alpha"]
    ref = sk.sinkhorn_forward(mu, nu, C, prob.lam, 20, alpha0=a0.clone())
    lib = sk.load_library()
    B, d1, d2 = prob.B, prob.d1, prob.d2
    p = _binding.problem(B, d1, d2, 0, prob.lam, 20)
    alpha = a0.clone()
    beta = torch.empty((B, d2), device=DEV)
    loss = torch.empty((B,), device=DEV)
    merr = torch.empty((B,), device=DEV)
    iters = torch.empty((B,), device=DEV, dtype=torch.int32)
    need = sk.sinkhorn_workspace_bytes(B, d1, d2, 0, prob.lam, 20)
    ws = torch.empty((max(need, 1),), device=DEV, dtype=torch.uint8)
    P = ctypes.c_void_p
    st = lib.sinkhorn_forward_warm(ctypes.byref(p), P(alpha.data_ptr()), P(mu.data_ptr()), P(nu.data_ptr()),
                                   P(C.data_ptr()), P(alpha.data_ptr()), P(beta.data_ptr()), P(loss.data_ptr()),
                                   P(merr.data_ptr()), P(iters.data_ptr()), P(ws.data_ptr()),
                                   ctypes.c_size_t(ws.numel()), P(torch.cuda.current_stream().cuda_stream))
    assert st == 0
    torch.cuda.synchronize()
    np.testing.assert_array_equal(alpha.cpu().numpy(), ref["alpha"].cpu().numpy())
    np.testing.assert_array_equal(loss.cpu().numpy(), ref["loss"].cpu().numpy())


def test_warm_loss_wrapper_takes_previous_state():
    """sinkhorn_loss with alpha0 from the previous call's state: the gradient
    formula is unchanged (it uses the returned potentials)."""
    prob = workloads.make_config(2, B=8)
    mu = _t(prob.mu).requires_grad_()
    nu = _t(prob.nu)
    C = _t(prob.C[0])
    _, st = sk.sinkhorn_loss(mu, nu, C, prob.lam, 50, return_state=True)
    loss, st2 = sk.sinkhorn_loss(mu, nu, C, prob.lam, 50, return_state=True, alpha0=st["alpha"])
    loss.sum().backward()
    a = st2["alpha"].detach().cpu().numpy()
    ref = oracle.backward(np.ones(prob.B), prob.mu, prob.nu, prob.C, prob.lam, a,
                          st2["beta"].detach().cpu().numpy())
    np.testing.assert_allclose(mu.grad.cpu().numpy(), ref["grad_mu"], atol=1e-4)
