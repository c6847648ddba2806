"""GPU parity: the HIP library (through the C ABI) against the fp64 oracle on
identical seeded fp32 inputs.  Tolerances (written here, per the build target):
loss relative error <= 1e-4, potentials absolute error <= 1e-3 after fixing the
additive gauge, gradients relative error <= 1e-3."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_1907_01729_amd as sk
import workloads
from parity_util import (GRAD_RTOL, LOSS_RTOL, POT_ATOL, gauge_fixed_errors, loss_rel_err, max_abs_rel_rows,
                         rel_err_rows)

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


# Kernel selector of the forwards run by _gpu (sinkhorn_forward_select):
# "default" is sinkhorn_forward itself; tests pin other kernels with set_form.
_FORM = {"select": "default"}


def set_form(select):
    _FORM["select"] = "default" if select == "auto" else select


@pytest.fixture(autouse=True)
def _default_form():
    set_form("default")
    yield
    set_form("default")


def _gpu(prob, sample=None):
    mu, nu, C = prob.mu, prob.nu, prob.C
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(DEV)
    out = sk.sinkhorn_forward_select(_FORM["select"], t(mu), t(nu), t(C), prob.lam, prob.n_iter, prob.tol)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def _subset(prob, idx):
    C = prob.C[idx] if prob.c_batched else prob.C
    return prob.mu[idx], prob.nu[idx], C


def check_forward(prob, gpu=None, idx=None, pot_atol=POT_ATOL, merr_atol=2e-5, merr_rtol=5e-2, free_k=True):
    """Compare a GPU forward with the oracle on samples idx (all by default),
    at the GPU's per-sample iteration counts."""
    _say(f"[parity] {prob.name} B={prob.B} d1={prob.d1} d2={prob.d2} lam={prob.lam} n_iter={prob.n_iter} "
         f"tol={prob.tol} c_batched={prob.c_batched}")
    if gpu is None:
        gpu = _gpu(prob)
    if idx is None:
        idx = np.arange(prob.B)
    mu, nu, C = _subset(prob, idx)
    iters = gpu["iters"][idx]
    if prob.tol > 0:
        if free_k:
            free = oracle.forward(mu, nu, C, prob.lam, prob.n_iter, tol=prob.tol)
            assert np.all(np.abs(free["iters"] - iters) <= 1), (free["iters"], iters)
        ref = oracle.forward(mu, nu, C, prob.lam, prob.n_iter, n_iter_b=iters)
    else:
        assert np.all(iters == prob.n_iter)
        ref = oracle.forward(mu, nu, C, prob.lam, prob.n_iter)
    el = loss_rel_err(gpu["loss"][idx], ref["loss"])
    ea, eb = gauge_fixed_errors(mu, nu, gpu["alpha"][idx], gpu["beta"][idx], ref["alpha"], ref["beta"])
    dm = np.abs(gpu["marg_err"][idx] - ref["marg_err"])
    _say(f"   loss rel {el:.2e}  alpha {ea:.2e}  beta {eb:.2e}  marg_err |d| max {dm.max():.2e} "
         f"(ref max {ref['marg_err'].max():.2e})")
    assert el <= LOSS_RTOL
    assert ea <= pot_atol and eb <= pot_atol
    assert np.all(dm <= merr_atol + merr_rtol * ref["marg_err"])
    return gpu, ref


def check_backward(prob, gpu, ref, idx=None, grad_C=False, seed=0):
    if idx is None:
        idx = np.arange(prob.B)
    rng = np.random.default_rng(seed)
    g = rng.uniform(0.5, 1.5, size=prob.B).astype(np.float32)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(DEV)
    out = sk.sinkhorn_backward(t(g), t(prob.mu), t(prob.nu), t(prob.C), prob.lam, t(gpu["alpha"]),
                               t(gpu["beta"]), grad_C=grad_C)
    torch.cuda.synchronize()
    mu, nu, C = _subset(prob, idx)
    r = oracle.backward(g[idx], mu, nu, C, prob.lam, ref["alpha"], ref["beta"], grad_C=grad_C and prob.c_batched)
    gm, gn = out["grad_mu"].cpu().numpy()[idx], out["grad_nu"].cpu().numpy()[idx]
    e1, e2 = rel_err_rows(gm, r["grad_mu"]), rel_err_rows(gn, r["grad_nu"])
    # elementwise: max |delta| within GRAD_RTOL of the sample's largest entry
    m1, m2 = max_abs_rel_rows(gm, r["grad_mu"]), max_abs_rel_rows(gn, r["grad_nu"])
    _say(f"   grad_mu rel {e1:.2e} (elementwise {m1:.2e})  grad_nu rel {e2:.2e} (elementwise {m2:.2e})")
    assert e1 <= GRAD_RTOL and e2 <= GRAD_RTOL
    assert m1 <= GRAD_RTOL and m2 <= GRAD_RTOL
    if grad_C:
        gC = out["grad_C"].cpu().numpy()
        if prob.c_batched:
            e3, m3 = rel_err_rows(gC[idx], r["grad_C"]), max_abs_rel_rows(gC[idx], r["grad_C"])
        else:
            assert len(idx) == prob.B, "shared grad_C sums the whole batch"
            rs = oracle.backward(g, prob.mu, prob.nu, prob.C, prob.lam, ref["alpha"], ref["beta"], grad_C=True)
            e3, m3 = rel_err_rows(gC, rs["grad_C"]), max_abs_rel_rows(gC, rs["grad_C"])
        _say(f"   grad_C rel {e3:.2e} (elementwise {m3:.2e})")
        assert e3 <= GRAD_RTOL and m3 <= GRAD_RTOL


@pytest.fixture(params=["auto", "nosym", "log"])
def form(request):
    """Resident regime: the plain-form kernels with their fallbacks (the
    default), the same without the symmetric-cost kernel (symmetric costs go
    to the general kernel), or the log-domain kernel alone."""
    set_form(request.param)
    return request.param


# ---------------------------------------------------------------- workloads

def test_tiny_full(form):
    prob = workloads.make_config(1)
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_label_subset_full_iterations(form):
    prob = workloads.make_config(2, B=48)
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_label_full_batch_shared_grad_C():
    """The label workload's full batch (B=1024) with the shared-cost grad_C,
    which sums g_b P_b over all 1024 problems: checked whole against the
    oracle's sum."""
    prob = workloads.make_config(2)
    gpu = _gpu(prob)
    ref = oracle.forward(prob.mu, prob.nu, prob.C, prob.lam, prob.n_iter)
    check_backward(prob, gpu, ref, grad_C=True)


def test_label_full_batch_sampled(form):
    """The benchmark's launch: B=1024, d=100, 200 iterations; the oracle checks
    a sample of the problems (each problem is independent)."""
    prob = workloads.make_config(2)
    gpu = _gpu(prob)
    idx = np.array([0, 1, 257, 511, 512, 777, 1022, 1023])
    gpu, ref = check_forward(prob, gpu=gpu, idx=idx)
    check_backward(prob, gpu, ref, idx=idx)
    assert np.all(np.isfinite(gpu["loss"])) and np.all(gpu["marg_err"] < 1e-2)


# ---------------------------------------------------------------- shapes and edge cases

@pytest.mark.parametrize("d1,d2", [(16, 16), (17, 9), (32, 31), (33, 64), (65, 100), (104, 37), (105, 128),
                                   (128, 128), (1, 7), (7, 1), (1, 1)])
def test_shapes_every_template(d1, d2, form):
    prob = workloads.random_problem(seed=d1 * 1000 + d2, B=5, d1=d1, d2=d2, lam=0.1, n_iter=40)
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_zero_masses(form):
    prob = workloads.random_problem(seed=7, B=6, d1=37, d2=100, lam=0.1, n_iter=60, zero_frac=0.25)
    assert (prob.mu == 0).any() and (prob.nu == 0).any()
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)
    gm = sk.sinkhorn_backward  # grads off the support are exactly 0
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(DEV)
    out = gm(t(np.ones(prob.B, np.float32)), t(prob.mu), t(prob.nu), t(prob.C), prob.lam, t(gpu["alpha"]),
             t(gpu["beta"]))
    assert np.all(out["grad_mu"].cpu().numpy()[prob.mu == 0] == 0)


def test_per_sample_cost_resident(form):
    prob = workloads.random_problem(seed=8, B=5, d1=20, d2=30, lam=0.05, n_iter=80, c_batched=True)
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


@pytest.mark.parametrize("n_iter", [0, 1, 2])
def test_few_iterations(n_iter, form):
    prob = workloads.random_problem(seed=9, B=3, d1=12, d2=9, lam=0.2, n_iter=n_iter)
    gpu, ref = check_forward(prob, merr_rtol=1e-3)
    assert np.all(gpu["iters"] == n_iter)


def test_single_sample_batch(form):
    prob = workloads.random_problem(seed=10, B=1, d1=50, d2=70, lam=0.05, n_iter=100)
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_early_stop_per_sample(form):
    prob = workloads.random_problem(seed=11, B=6, d1=30, d2=40, lam=0.1, n_iter=400, tol=1e-4)
    gpu, ref = check_forward(prob)
    assert np.all(gpu["iters"] < 400) and len(set(gpu["iters"].tolist())) > 1
    assert np.all(gpu["marg_err"] <= 1.5e-4)


def test_unreachable_tol_runs_all_iterations(form):
    prob = workloads.random_problem(seed=12, B=3, d1=20, d2=20, lam=0.01, n_iter=30, tol=1e-9)
    gpu, ref = check_forward(prob)
    assert np.all(gpu["iters"] == 30)


def test_large_lambda_independent_coupling(form):
    prob = workloads.random_problem(seed=13, B=4, d1=20, d2=25, lam=1e3, n_iter=5)
    gpu, ref = check_forward(prob)
    indep = np.einsum("bi,ij,bj->b", prob.mu.astype(np.float64), prob.C[0].astype(np.float64),
                      prob.nu.astype(np.float64))
    assert np.allclose(gpu["loss"], indep, rtol=1e-3)


def test_small_lambda_1d_grid_w1(form):
    """lambda = 1e-3 on a 1-D grid (C/lambda up to 1000): exercises the exact
    logsumexp fallbacks; E^0 approaches the closed-form W1."""
    prob = workloads.random_problem(seed=14, B=4, d1=100, d2=100, lam=1e-3, n_iter=300, cost="grid1d")
    gpu, ref = check_forward(prob, merr_atol=1e-4)
    x = np.linspace(0, 1, 100)
    for k in range(prob.B):
        w1 = np.abs(np.cumsum(prob.mu[k].astype(np.float64)) - np.cumsum(prob.nu[k].astype(np.float64)))[:-1].sum() * (x[1] - x[0])
        assert gpu["loss"][k] == pytest.approx(w1, abs=1e-2 + 5 * gpu["marg_err"][k])


def test_deterministic_bitwise(form):
    prob = workloads.make_config(2, B=64)
    a = _gpu(prob)
    b = _gpu(prob)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])


def test_autograd_wrapper(form):
    prob = workloads.random_problem(seed=15, B=4, d1=24, d2=24, lam=0.1, n_iter=50)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(DEV)
    mu = t(prob.mu).requires_grad_()
    nu = t(prob.nu).requires_grad_()
    C = t(prob.C[0]).requires_grad_()
    loss, st = sk.sinkhorn_loss(mu, nu, C, prob.lam, prob.n_iter, return_state=True)
    (loss * torch.arange(1, 5, device=DEV)).sum().backward()
    ref = oracle.forward(prob.mu, prob.nu, prob.C, prob.lam, prob.n_iter)
    g = oracle.backward(np.arange(1, 5), prob.mu, prob.nu, prob.C, prob.lam, ref["alpha"], ref["beta"], grad_C=True)
    assert rel_err_rows(mu.grad.cpu().numpy(), g["grad_mu"]) <= GRAD_RTOL
    assert rel_err_rows(nu.grad.cpu().numpy(), g["grad_nu"]) <= GRAD_RTOL
    assert rel_err_rows(C.grad.cpu().numpy()[None], g["grad_C"]) <= GRAD_RTOL


# ---------------------------------------------------------------- tiled regime (max(d1, d2) > 128)

# ---------------------------------------------------------------- plain form and its fallback

def test_plain_form_takes_in_range_problems():
    """The plain-form kernel alone (no fallback launch) solves every label
    problem (cost spread 54 bits) and leaves a lambda = 1e-3 grid problem
    (spread > 1000 bits) to the log-domain kernel: iters = -1."""
    set_form("plain")
    prob = workloads.make_config(2, B=32)
    gpu, ref = check_forward(prob)
    assert np.all(gpu["iters"] == prob.n_iter)
    check_backward(prob, gpu, ref, grad_C=True)
    far = workloads.random_problem(seed=16, B=3, d1=40, d2=40, lam=1e-3, n_iter=20, cost="grid1d")
    assert np.all(_gpu(far)["iters"] == -1)


def test_plain_fallback_mixed_batch():
    """Per-sample costs where every third problem's cost spread exceeds the
    plain form's range: with the fallback every problem matches the oracle;
    without it exactly those problems come back unsolved."""
    prob = workloads.random_problem(seed=17, B=9, d1=50, d2=60, lam=0.05, n_iter=80, c_batched=True)
    far = np.arange(prob.B) % 3 == 0
    prob.C[far] *= 3.0  # spread 3 * 28.9 bits > 64
    set_form("plain")
    alone = _gpu(prob)
    assert np.all((alone["iters"] == -1) == far)
    set_form("auto")
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)
    near = ~far
    for k in ("alpha", "beta", "loss", "marg_err", "iters"):
        np.testing.assert_array_equal(gpu[k][near], alone[k][near])


def test_plain_early_stop_agrees_with_log():
    prob = workloads.random_problem(seed=18, B=8, d1=64, d2=48, lam=0.1, n_iter=300, tol=1e-5)
    out = {}
    for f in ("plain", "log"):
        set_form(f)
        out[f] = check_forward(prob)[0]
    assert np.all(out["plain"]["iters"] >= 0)
    assert np.all(np.abs(out["plain"]["iters"] - out["log"]["iters"]) <= 1)


# ---------------------------------------------------------------- symmetric shared cost, one wavefront per problem

@pytest.mark.parametrize("d", [1, 2, 7, 8, 9, 16, 17, 32, 33, 64, 65, 96, 97, 100, 104])
def test_sym_kernel_shapes(d):
    """Every register-tile width of the symmetric-cost kernel, ragged tails
    included; alone (plain) it solves every problem."""
    prob = workloads.random_problem(seed=300 + d, B=5, d1=d, d2=d, lam=0.1, n_iter=60, cost="sym")
    set_form("plain")
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_sym_kernel_zero_masses():
    prob = workloads.random_problem(seed=31, B=7, d1=90, d2=90, lam=0.05, n_iter=120, cost="sym", zero_frac=0.3)
    set_form("plain")
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_sym_kernel_runs_general_iteration_on_asymmetric_cost():
    """An asymmetric cost (one pair differs): the symmetric kernel alone runs
    the general iteration in place, with the same bits as the general kernel
    launched by itself, and the result matches the oracle."""
    prob = workloads.random_problem(seed=32, B=6, d1=50, d2=50, lam=0.1, n_iter=50, cost="sym")
    prob.C[0, 3, 41] += 0.25
    set_form("nosym")
    ref_bits = _gpu(prob)
    assert np.all(ref_bits["iters"] == 50)
    for form in ("plain", "auto"):
        set_form(form)
        gpu, ref = check_forward(prob)
        for k in ("alpha", "beta", "loss", "marg_err", "iters"):
            np.testing.assert_array_equal(gpu[k], ref_bits[k])


def test_sym_kernel_hands_over_out_of_range():
    """lambda = 1e-3 on a symmetric 1-D grid cost (spread > 1000 bits): iters
    = -1 from the symmetric kernel alone; the log-domain kernel solves it."""
    prob = workloads.random_problem(seed=33, B=3, d1=60, d2=60, lam=1e-3, n_iter=100, cost="grid1d")
    set_form("plain")
    assert np.all(_gpu(prob)["iters"] == -1)
    set_form("auto")
    check_forward(prob, merr_atol=1e-4)


@pytest.mark.parametrize("tol,n_iter", [(0.0, 50), (1e-5, 300)])
def test_sym_kernel_guard_fails_in_loop(tol, n_iter):
    """A positive but tiny mass (1e-37) puts its row scaling below 2^-100 in
    the first u-update, a guard the symmetric kernel checks inside the
    iteration (the cost spread itself is in range): alone it returns that
    problem unsolved (iters = -1) and the rest solved; with the fallback the
    problem matches the oracle and the others keep their bits."""
    prob = workloads.random_problem(seed=35, B=6, d1=70, d2=70, lam=0.1, n_iter=n_iter, cost="sym", tol=tol)
    prob.mu[2, 5] = 1e-37
    set_form("plain")
    alone = _gpu(prob)
    rest = np.arange(prob.B) != 2
    assert alone["iters"][2] == -1
    assert np.all(alone["iters"][rest] >= 1)
    set_form("auto")
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref)
    for k in ("alpha", "beta", "loss", "marg_err", "iters"):
        np.testing.assert_array_equal(gpu[k][rest], alone[k][rest])


@pytest.mark.parametrize("tol,n_iter", [(0.0, 50), (1e-5, 300)])
def test_gen_kernel_guard_fails_in_loop(tol, n_iter):
    """Per-sample costs, d1 != d2: a tiny positive mass (1e-37) fails a guard
    of the general kernel inside the iteration; alone it returns that
    problem unsolved and the rest solved, with the fallback the problem
    matches the oracle and the others keep their bits."""
    prob = workloads.random_problem(seed=38, B=5, d1=60, d2=45, lam=0.1, n_iter=n_iter, c_batched=True, tol=tol)
    prob.mu[1, 9] = 1e-37
    set_form("plain")
    alone = _gpu(prob)
    rest = np.arange(prob.B) != 1
    assert alone["iters"][1] == -1
    assert np.all(alone["iters"][rest] >= 1)
    set_form("auto")
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)
    for k in ("alpha", "beta", "loss", "marg_err", "iters"):
        np.testing.assert_array_equal(gpu[k][rest], alone[k][rest])


def test_gen_kernel_full_batch_per_sample_sampled():
    """The general kernel at the label workload's launch size with one cost
    per problem (B=1024, d=100); the oracle checks a sample."""
    base = workloads.make_config(2)
    rng = np.random.default_rng(39)
    C = (base.C[0][None] * rng.uniform(0.75, 1.05, size=(base.B, 1, 1))).astype(np.float32)  # spread <= 57 bits
    C[:, 3, 5] += 0.05  # not symmetric
    prob = workloads.random_problem(seed=39, B=base.B, d1=100, d2=100, lam=base.lam, n_iter=base.n_iter,
                                    c_batched=True)
    prob.C = C
    gpu = _gpu(prob)
    assert np.all(gpu["iters"] == prob.n_iter)
    idx = np.array([0, 1, 300, 511, 512, 901, 1023])
    gpu, ref = check_forward(prob, gpu=gpu, idx=idx)
    check_backward(prob, gpu, ref, idx=idx, grad_C=True)


def test_sym_kernel_early_stop():
    prob = workloads.random_problem(seed=34, B=8, d1=80, d2=80, lam=0.1, n_iter=400, tol=1e-5, cost="sym")
    out = {}
    for f in ("plain", "log"):
        set_form(f)
        out[f] = check_forward(prob)[0]
    assert np.all(out["plain"]["iters"] >= 1) and np.all(out["plain"]["iters"] < 400)
    assert np.all(np.abs(out["plain"]["iters"] - out["log"]["iters"]) <= 1)


def test_image_reduced_batch():
    prob = workloads.make_config(3, B=4, n_iter=60)
    assert sk.sinkhorn_regime(prob.B, prob.d1, prob.d2, 0) == 2
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_image_full_batch_sampled():
    """The full image workload (B=256, d=784, 300 iterations); the oracle
    checks problems from four different 8-problem work-groups (0, 9, 16, 31)
    and both ends of the batch."""
    prob = workloads.make_config(3)
    gpu = _gpu(prob)
    idx = np.array([0, 77, 130, 255])
    gpu, ref = check_forward(prob, gpu=gpu, idx=idx)
    check_backward(prob, gpu, ref, idx=idx)


def test_grid_small_lambda_reduced():
    """lambda = 1e-3 on a 24x24 grid (C/lambda up to 2000): the stability regime."""
    prob = workloads.make_config(4, B=3, side=24, n_iter=120)
    gpu, ref = check_forward(prob, merr_atol=1e-4)
    check_backward(prob, gpu, ref)


@pytest.fixture(scope="module")
def grid_full():
    """One GPU forward of the full grid workload (B=64, d=4096, lambda=1e-3,
    500 iterations, tol=1e-6), shared by the sampled checks below."""
    prob = workloads.make_config(4)
    return prob, _gpu(prob)


@pytest.mark.parametrize("b", [0, 8, 63])
def test_grid_full_size_sampled(grid_full, b):
    """The full grid workload; the oracle (about 35 s per problem) checks
    problems from the first, second and last 8-problem work-group."""
    prob, gpu = grid_full
    # tol = 1e-6 is out of reach in 500 iterations at lambda = 1e-3 (the fp64
    # marginal error is ~6e-4 there), so every problem runs all iterations.
    assert np.all(gpu["iters"] == 500)
    idx = np.array([b])
    gpu, ref = check_forward(prob, gpu=gpu, idx=idx, merr_atol=1e-4, free_k=False)
    check_backward(prob, gpu, ref, idx=idx)


def test_clouds_reduced():
    prob = workloads.make_config(5, B=3, d1=256, d2=520, n_iter=40)
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_clouds_full_size_sampled():
    """Per-sample cost [32, 1024, 2048], 100 iterations, grad_C; oracle on 3 problems."""
    prob = workloads.make_config(5)
    gpu = _gpu(prob)
    idx = np.array([0, 15, 31])
    gpu, ref = check_forward(prob, gpu=gpu, idx=idx)
    check_backward(prob, gpu, ref, idx=idx, grad_C=True)


@pytest.mark.parametrize("d1,d2", [(300, 129), (129, 1000), (1500, 70), (200, 4096), (131, 257)])
def test_tiled_ragged_shapes(d1, d2):
    prob = workloads.random_problem(seed=d1 + 7 * d2, B=3, d1=d1, d2=d2, lam=0.1, n_iter=30)
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_tiled_per_sample_cost_and_zero_masses():
    prob = workloads.random_problem(seed=21, B=4, d1=150, d2=300, lam=0.05, n_iter=50, c_batched=True,
                                    zero_frac=0.2)
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_tiled_early_stop_per_sample():
    prob = workloads.random_problem(seed=22, B=5, d1=200, d2=160, lam=0.1, n_iter=400, tol=1e-4)
    gpu, ref = check_forward(prob)
    _say(f"   iters {gpu['iters'].tolist()}")
    assert np.all(gpu["iters"] < 400)
    assert np.all(gpu["marg_err"] <= 1.5e-4)


@pytest.mark.parametrize("n_iter", [0, 1, 2])
def test_tiled_few_iterations(n_iter):
    prob = workloads.random_problem(seed=23, B=2, d1=140, d2=200, lam=0.2, n_iter=n_iter)
    gpu, ref = check_forward(prob, merr_rtol=1e-3)
    assert np.all(gpu["iters"] == n_iter)


def test_tiled_small_lambda_1d_grid():
    prob = workloads.random_problem(seed=24, B=2, d1=300, d2=300, lam=1e-3, n_iter=300, cost="grid1d")
    gpu, ref = check_forward(prob, merr_atol=1e-4)


def test_tiled_deterministic_bitwise():
    prob = workloads.make_config(3, B=8, n_iter=20)
    a = _gpu(prob)
    b = _gpu(prob)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])


@pytest.mark.parametrize("B,d1,d2,c_batched", [
    (5, 200, 300, False),    # shared cost, 4 problems per work-group (+1 idle-padded group)
    (9, 150, 260, False),    # shared cost, 8 problems per work-group, 7 idle wavefronts in the last group
    (3, 160, 301, True),     # per-sample cost, d2 % 4 != 0: scalar per-problem sweep
    (3, 129, 516, True),     # per-sample cost, 128-bit streaming sweep with a ragged last vector
    (2, 300, 200, False),    # shared cost, batch too small for the shared sweep
])
def test_tiled_kernel_variants(B, d1, d2, c_batched):
    prob = workloads.random_problem(seed=B * 1000 + d2, B=B, d1=d1, d2=d2, lam=0.08, n_iter=35,
                                    c_batched=c_batched, zero_frac=0.1)
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_tiled_variants_early_stop_shared():
    """Early stop inside the shared-cost sweep (stopped problems keep staging)."""
    prob = workloads.random_problem(seed=31, B=10, d1=180, d2=200, lam=0.1, n_iter=300, tol=2e-4)
    gpu, ref = check_forward(prob)
    assert np.all(gpu["iters"] < 300)


@pytest.mark.parametrize("B,d1,d2,zero_frac", [
    (8, 300, 500, 0.0),     # 8 column registers per lane, rows reduced four at a time
    (12, 260, 1000, 0.1),   # 16 column registers, zero masses, a half-idle second group
    (8, 700, 1500, 0.0),    # 32 column registers, rows reduced two at a time
    (8, 520, 2100, 0.05),   # 64 column registers, one row at a time
    (9, 129, 801, 0.0),     # d2 % 4 != 0: 4-byte global->LDS copies
])
def test_shared_sweep_shapes(B, d1, d2, zero_frac):
    """The shared-cost sweep (W problems per work-group, cost rows staged in LDS)
    at every column-register width it is built for."""
    prob = workloads.random_problem(seed=B * 7 + d1 + d2, B=B, d1=d1, d2=d2, lam=0.06, n_iter=30,
                                    zero_frac=zero_frac)
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_shared_sweep_multi_segment_rows():
    """Row blocks of 150 rows (three 64-row segments of row potentials per
    wavefront) in the shared-cost sweep; oracle on 3 of 512 problems."""
    prob = workloads.random_problem(seed=77, B=512, d1=1200, d2=200, lam=0.1, n_iter=25)
    gpu = _gpu(prob)
    idx = np.array([0, 200, 511])
    gpu, ref = check_forward(prob, gpu=gpu, idx=idx)
    check_backward(prob, gpu, ref, idx=idx)


def test_shared_sweep_small_lambda_exact_rows():
    """lambda = 1e-3 on a 24x24 grid with a batch of 8 (shared-cost sweep):
    rows whose shifted sums leave [2^-64, 2^64] take the exact logsumexp."""
    prob = workloads.make_config(4, B=8, side=24, n_iter=120)
    gpu, ref = check_forward(prob, merr_atol=1e-4)
    check_backward(prob, gpu, ref)


def test_stream_early_stop_per_sample():
    """Per-sample costs streamed through LDS rings: the merge folded into the
    next sweep takes the same per-sample stop decision in every row block."""
    prob = workloads.random_problem(seed=41, B=5, d1=300, d2=400, lam=0.1, n_iter=400, c_batched=True, tol=1e-4)
    gpu, ref = check_forward(prob)
    _say(f"   iters {gpu['iters'].tolist()}")
    assert np.all(gpu["iters"] < 400)
    check_backward(prob, gpu, ref, grad_C=True)


@pytest.mark.parametrize("d1,d2", [(150, 4000), (100, 2400), (300, 512)])
def test_stream_widths(d1, d2):
    """Streaming sweep at 16 and 10 float4 groups per lane (two wavefronts per
    work-group) and at 2 groups with one-row blocks (B = 1: some wavefronts
    get no row)."""
    B = 1 if d2 == 512 else 2
    prob = workloads.random_problem(seed=d1 + d2, B=B, d1=d1, d2=d2, lam=0.07, n_iter=30, c_batched=True,
                                    zero_frac=0.05)
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_stream_small_lambda_exact_paths():
    """lambda = 1e-3 on a per-sample 1-D grid cost: rows and columns whose
    shifted sums leave [2^-64, 2^64] take the exact logsumexp in the ring
    sweep and in the folded merge (which reads the previous potentials plane)."""
    prob = workloads.random_problem(seed=43, B=2, d1=300, d2=304, lam=1e-3, n_iter=200, c_batched=True,
                                    cost="grid1d")
    gpu, ref = check_forward(prob, merr_atol=1e-4)
    check_backward(prob, gpu, ref)


# ---------------------------------------------------------------- early stop with batch compaction (shared sweep)

def test_shared_sweep_early_stop_compaction():
    """Image histograms with an early stop: problems stop at different
    iterations; the shared-cost sweep compacts the running problems into its
    8-problem work-groups.  Parity with the oracle at the GPU's iteration
    counts, and the same bits as without compaction."""
    prob = workloads.make_config(3, B=24, side=20, n_iter=400)
    prob.tol = 2e-4
    set_form("nocompact")
    plain = _gpu(prob)
    set_form("default")
    gpu, ref = check_forward(prob)
    its = gpu["iters"]
    assert (its < prob.n_iter).sum() >= prob.B - 2 and len(set(its.tolist())) > 3, its
    for k in plain:
        np.testing.assert_array_equal(gpu[k], plain[k])


def test_split_merge_early_stop():
    """Rows wider than 1024 columns: the merge after each sweep runs several
    work-groups per problem, and the last of them to finish takes the stop
    decision from their parts added in a fixed order.  Problems stop at
    different iterations; parity with the oracle at the GPU's counts, the same
    bits on a second run and without compaction."""
    prob = workloads.random_problem(seed=611, B=12, d1=200, d2=2300, lam=0.05, n_iter=300, tol=1e-3,
                                    zero_frac=0.1, cost="grid1d")
    set_form("nocompact")
    plain = _gpu(prob)
    set_form("default")
    gpu, ref = check_forward(prob)
    again = _gpu(prob)
    its = gpu["iters"]
    _say(f"   iterations {sorted(its.tolist())}")
    assert (its < prob.n_iter).sum() >= prob.B - 2 and len(set(its.tolist())) > 3, its
    for k in plain:
        np.testing.assert_array_equal(gpu[k], plain[k])
        np.testing.assert_array_equal(gpu[k], again[k])
    # A tolerance above every possible first error (at most 2 for unit masses):
    # parts are clamped at 2^p >= 2 tol, and every problem stops after one
    # iteration, as in the oracle.
    prob.tol = 5.0
    one = _gpu(prob)
    assert np.all(one["iters"] == 1), one["iters"]
    check_forward(prob, gpu=one)


# ---------------------------------------------------------------- randomized resident problems

def test_random_resident_problems():
    """Forty seeded random problems of the resident regime (d1, d2 <= 128,
    shared or per-sample, symmetric or not, zero masses, lambda over two
    decades so that some leave the plain form's range, fixed or early-stopped
    iterations), through whichever kernels take them, forward and backward
    against the oracle."""
    rng = np.random.default_rng(2024)
    for case in range(40):
        d1, d2 = int(rng.integers(1, 129)), int(rng.integers(1, 129))
        if rng.random() < 0.3:
            d2 = d1
        B = int(rng.integers(1, 10))
        lam = float(10 ** rng.uniform(-1.7, 0.3))
        n_iter = int(rng.integers(0, 120))
        tol = float(rng.choice([0.0, 0.0, 1e-4, 1e-5]))
        cb = bool(rng.random() < 0.4)
        zf = float(rng.choice([0.0, 0.0, 0.2]))
        cost = "sym" if (d1 == d2 and rng.random() < 0.6) else "uniform"
        set_form("nosym" if rng.random() < 0.25 else "auto")
        prob = workloads.random_problem(seed=int(rng.integers(1 << 30)), B=B, d1=d1, d2=d2, lam=lam,
                                        n_iter=n_iter, c_batched=cb, zero_frac=zf, cost=cost, tol=tol)
        _say(f"[random {case}]")
        gpu, ref = check_forward(prob)
        check_backward(prob, gpu, ref, grad_C=True)


def test_random_asymmetric_shared_costs():
    """Twelve seeded shared square costs, symmetric but for one pair, over the
    symmetric kernel's size buckets (d up to 104): each work-group finds the
    pair and runs the general iteration in place.  Same bits as the general
    kernel launched alone, and the oracle's results."""
    rng = np.random.default_rng(4242)
    for case, d in enumerate((2, 9, 16, 23, 40, 57, 64, 71, 90, 97, 100, 104)):
        B = int(rng.integers(1, 9))
        lam = float(10 ** rng.uniform(-1.3, 0.0))
        n_iter = int(rng.integers(1, 120))
        tol = float(rng.choice([0.0, 1e-5]))
        prob = workloads.random_problem(seed=int(rng.integers(1 << 30)), B=B, d1=d, d2=d, lam=lam, n_iter=n_iter,
                                        zero_frac=float(rng.choice([0.0, 0.2])), cost="sym", tol=tol)
        i = int(rng.integers(0, d))
        j = (i + 1 + int(rng.integers(0, d - 1))) % d  # j != i
        prob.C[0, i, j] += 0.01
        _say(f"[asym {case}] d={d} pair=({i},{j})")
        set_form("nosym")
        ref_bits = _gpu(prob)
        set_form("auto")
        gpu, ref = check_forward(prob)
        for k in ("alpha", "beta", "loss", "marg_err", "iters"):
            np.testing.assert_array_equal(gpu[k], ref_bits[k])
        check_backward(prob, gpu, ref, grad_C=True)


@pytest.mark.parametrize("form,c_batched", [("auto", False), ("nosym", False), ("log", False), ("auto", True)])
def test_large_batch_resident(form, c_batched):
    """B = 70000 small problems (more than 65535 work-groups for the plain
    kernels, problem indices past 16 bits) through each resident kernel; the
    oracle checks samples on both sides of 65536."""
    set_form(form)
    prob = workloads.random_problem(seed=77, B=70000, d1=8, d2=8, lam=0.1, n_iter=50, c_batched=c_batched,
                                    cost="uniform" if c_batched else "sym")
    gpu = _gpu(prob)
    assert np.all(gpu["iters"] == 50)
    idx = np.array([0, 1, 32767, 65535, 65536, 65537, 69998, 69999])
    gpu, ref = check_forward(prob, gpu=gpu, idx=idx)
    check_backward(prob, gpu, ref, idx=idx, grad_C=c_batched)


def test_tiled_on_side_stream():
    """The tiled regime on a caller's side stream while the current stream
    allocates and fills memory: the binding allocates the outputs and the
    temporary workspace on the library's stream, so the caching allocator
    never hands the freed workspace to other work before the kernels end."""
    prob = workloads.make_config(3, B=16, n_iter=60)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(DEV)
    mu, nu, C = t(prob.mu), t(prob.nu), t(prob.C)
    need = sk.sinkhorn_workspace_bytes(prob.B, prob.d1, prob.d2, 0, prob.lam, prob.n_iter)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    out = sk.sinkhorn_forward(mu, nu, C, prob.lam, prob.n_iter, stream=side)
    junk = [torch.full((need // 4 + 1,), float("nan"), device=DEV) for _ in range(8)]
    side.synchronize()
    torch.cuda.synchronize()
    del junk
    gpu = {k: v.cpu().numpy() for k, v in out.items()}
    check_forward(prob, gpu=gpu)


@pytest.mark.parametrize("c_batched,tol", [(False, 0.0), (True, 2e-4)])
def test_tiled_batch_above_grid_limit(c_batched, tol):
    """65537 problems of a tiled shape: more than one grid dimension holds,
    so the batch runs as two chunks (65535 + 2) that share one workspace.
    Problems on both sides of the boundary against the oracle, forward and
    backward, with a shared cost and with per-sample costs and early stop."""
    prob = workloads.random_problem(seed=91, B=65537, d1=130, d2=8, lam=0.1, n_iter=40, c_batched=c_batched,
                                    tol=tol)
    assert sk.sinkhorn_regime(prob.B, prob.d1, prob.d2, int(c_batched)) == 2
    idx = np.array([0, 1, 65533, 65534, 65535, 65536])
    gpu, ref = check_forward(prob, idx=idx)
    check_backward(prob, gpu, ref, idx=idx, grad_C=c_batched)


@pytest.mark.parametrize("B,d1,d2,c_batched,lam,n_iter,zero_frac,tol", [
    (5, 150, 5000, False, 0.1, 30, 0.0, 0.0),    # shared cost, rows just past one wavefront's registers
    (3, 9, 6000, True, 0.05, 40, 0.2, 1e-3),     # per-sample costs, zero masses, early stop, few rows
    (2, 300, 4097, False, 0.005, 40, 0.0, 0.0),  # ragged width, small lambda (exact fallbacks)
    (4, 130, 9000, True, 0.02, 25, 0.1, 0.0),
    (2, 3, 100000, True, 0.1, 20, 0.0, 0.0),     # 100000 columns, 3 rows
])
def test_wide_rows(B, d1, d2, c_batched, lam, n_iter, zero_frac, tol):
    """Rows wider than one wavefront's registers hold (d2 > 4096): two passes
    over the cost per iteration; forward and backward (with grad_C) against
    the oracle on every problem."""
    prob = workloads.random_problem(seed=d2 + d1, B=B, d1=d1, d2=d2, lam=lam, n_iter=n_iter, c_batched=c_batched,
                                    zero_frac=zero_frac, tol=tol)
    assert sk.sinkhorn_regime(B, d1, d2, int(c_batched)) == 2
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_wide_grid_image_sampled():
    """Image histograms on a 91x91 grid (d = 8281, shared squared grid cost of
    274 MB, lambda 0.01), B = 8: the first and last problems against the oracle."""
    prob = workloads.image(B=8, side=91, n_iter=100, lam=0.01)
    idx = np.array([0, 7])
    gpu, ref = check_forward(prob, idx=idx)
    check_backward(prob, gpu, ref, idx=idx)


@pytest.mark.parametrize("B,d1,d2", [(6, 40, 30), (5, 300, 260), (5, 200, 2000), (4, 150, 4100)])
def test_non_finite_cost_propagates(B, d1, d2):
    """A NaN in one problem's cost (per-sample costs): that problem's loss and
    error are not finite and it runs every iteration (its error is never
    <= tol); every other problem is bit-identical to a run without the NaN.
    A NaN in a shared cost makes every problem's loss non-finite.  Every call
    returns: the loops are bounded by the shapes and n_iter, never by the
    data."""
    prob = workloads.random_problem(seed=88, B=B, d1=d1, d2=d2, lam=0.1, n_iter=30, c_batched=True, tol=1e-5)
    clean = _gpu(prob)
    prob.C[2, d1 // 2, d2 // 3] = np.nan
    dirty = _gpu(prob)
    assert not np.isfinite(dirty["loss"][2]) and not np.isfinite(dirty["marg_err"][2])
    assert dirty["iters"][2] == prob.n_iter
    others = [b for b in range(B) if b != 2]
    for k in ("alpha", "beta", "loss", "marg_err", "iters"):
        np.testing.assert_array_equal(dirty[k][others], clean[k][others])
    shared = workloads.random_problem(seed=89, B=8, d1=d1, d2=d2, lam=0.1, n_iter=20, tol=1e-5)
    shared.C[0, 0, 0] = np.nan
    out = _gpu(shared)
    assert not np.any(np.isfinite(out["loss"])) and np.all(out["iters"] == shared.n_iter)


def test_shared_grad_C_many_rows():
    """A shared cost with d1 = 70000 rows (more than a grid's y dimension):
    the forward runs in the tiled regime and grad_C (rows grid-strided) covers
    every row; the oracle checks the whole gradient."""
    prob = workloads.random_problem(seed=79, B=2, d1=70000, d2=130, lam=0.2, n_iter=8)
    gpu, ref = check_forward(prob)
    check_backward(prob, gpu, ref, grad_C=True)


def test_tiled_max_batch():
    """The tiled regime's largest batch, B = 65535 (d = 130, shared cost):
    every grid dimension at its limit; the oracle checks samples."""
    prob = workloads.random_problem(seed=78, B=65535, d1=130, d2=130, lam=0.1, n_iter=20)
    gpu = _gpu(prob)
    assert np.all(gpu["iters"] == 20)
    idx = np.array([0, 1, 7, 8, 32767, 65527, 65528, 65534])
    gpu, ref = check_forward(prob, gpu=gpu, idx=idx)
    check_backward(prob, gpu, ref, idx=idx)
