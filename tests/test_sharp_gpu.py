"""GPU parity of the sharp-loss gradient (gradient of E^0 itself, implicit
differentiation of the plan, conjugate gradients on the GPU) through the C
ABI, against the oracle's dense fp64 solve on the same inputs (the forward's
alpha, beta).  Gradients relative error <= 1e-3."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_1907_01729_amd as sk
import workloads
from parity_util import GRAD_RTOL, rel_err_rows

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def check_sharp(prob, idx=None, seed=0, max_cg=300, cg_tol=1e-6):
    _say(f"[sharp] {prob.name} B={prob.B} d1={prob.d1} d2={prob.d2} lam={prob.lam} n_iter={prob.n_iter}")
    mu, nu, C = _t(prob.mu), _t(prob.nu), _t(prob.C)
    fw = sk.sinkhorn_forward(mu, nu, C, prob.lam, prob.n_iter, prob.tol)
    g = np.random.default_rng(seed).uniform(0.5, 1.5, size=prob.B).astype(np.float32)
    out = sk.sinkhorn_backward_sharp(_t(g), mu, nu, C, prob.lam, fw["alpha"], fw["beta"], max_cg=max_cg,
                                     cg_tol=cg_tol)
    torch.cuda.synchronize()
    if idx is None:
        idx = np.arange(prob.B)
    a, b = fw["alpha"].cpu().numpy()[idx], fw["beta"].cpu().numpy()[idx]
    Cs = prob.C[idx] if prob.c_batched else prob.C
    ref = oracle.sharp_gradient(g[idx], prob.mu[idx], prob.nu[idx], Cs, prob.lam, a, b)
    e1 = rel_err_rows(out["grad_mu"].cpu().numpy()[idx], ref["grad_mu"])
    e2 = rel_err_rows(out["grad_nu"].cpu().numpy()[idx], ref["grad_nu"])
    its = out["cg_iters"].cpu().numpy()[idx]
    _say(f"   grad_mu {e1:.2e}  grad_nu {e2:.2e}  cg iterations {its.min()}..{its.max()}")
    assert e1 <= GRAD_RTOL and e2 <= GRAD_RTOL
    assert np.all(its < max_cg) and np.all(its >= 1)
    return out, ref


def test_sharp_tiny():
    check_sharp(workloads.make_config(1))


def test_sharp_label_subset():
    check_sharp(workloads.make_config(2, B=32))


def test_sharp_label_full_batch_sampled():
    """The label workload's launch (B=1024, d=100); the dense solve on 8 problems."""
    check_sharp(workloads.make_config(2), idx=np.array([0, 1, 255, 511, 512, 700, 1022, 1023]))


@pytest.mark.parametrize("d1,d2", [(1, 7), (7, 1), (16, 16), (17, 9), (32, 5), (37, 100), (64, 64), (100, 37),
                                   (104, 104), (105, 10), (128, 128), (127, 33)])
def test_sharp_shapes(d1, d2):
    prob = workloads.random_problem(seed=400 + d1 + d2, B=4, d1=d1, d2=d2, lam=0.1, n_iter=200)
    check_sharp(prob)


def test_sharp_per_sample_cost_and_zero_masses():
    prob = workloads.random_problem(seed=41, B=5, d1=50, d2=70, lam=0.05, n_iter=300, c_batched=True,
                                    zero_frac=0.25)
    assert (prob.mu == 0).any() and (prob.nu == 0).any()
    out, _ = check_sharp(prob)
    assert np.all(out["grad_mu"].cpu().numpy()[prob.mu == 0] == 0)
    assert np.all(out["grad_nu"].cpu().numpy()[prob.nu == 0] == 0)


def test_sharp_against_converged_oracle():
    """Long enough that both forwards have converged: the GPU's sharp
    gradient matches the oracle's, each from its own forward."""
    prob = workloads.random_problem(seed=42, B=3, d1=30, d2=40, lam=0.1, n_iter=2000)
    mu, nu, C = _t(prob.mu), _t(prob.nu), _t(prob.C)
    fw = sk.sinkhorn_forward(mu, nu, C, prob.lam, prob.n_iter)
    g = torch.ones(prob.B, device=DEV)
    out = sk.sinkhorn_backward_sharp(g, mu, nu, C, prob.lam, fw["alpha"], fw["beta"])
    o = oracle.forward(prob.mu, prob.nu, prob.C, prob.lam, prob.n_iter)
    ref = oracle.sharp_gradient(np.ones(prob.B), prob.mu, prob.nu, prob.C, prob.lam, o["alpha"], o["beta"])
    assert rel_err_rows(out["grad_mu"].cpu().numpy(), ref["grad_mu"]) <= GRAD_RTOL
    assert rel_err_rows(out["grad_nu"].cpu().numpy(), ref["grad_nu"]) <= GRAD_RTOL


def test_sharp_iteration_cap_and_deterministic():
    prob = workloads.make_config(2, B=16)
    mu, nu, C = _t(prob.mu), _t(prob.nu), _t(prob.C)
    fw = sk.sinkhorn_forward(mu, nu, C, prob.lam, prob.n_iter)
    g = torch.ones(prob.B, device=DEV)
    one = sk.sinkhorn_backward_sharp(g, mu, nu, C, prob.lam, fw["alpha"], fw["beta"], max_cg=2, cg_tol=0.0)
    assert np.all(one["cg_iters"].cpu().numpy() == 2)
    a = sk.sinkhorn_backward_sharp(g, mu, nu, C, prob.lam, fw["alpha"], fw["beta"])
    b = sk.sinkhorn_backward_sharp(g, mu, nu, C, prob.lam, fw["alpha"], fw["beta"])
    for k in a:
        np.testing.assert_array_equal(a[k].cpu().numpy(), b[k].cpu().numpy())


def test_sharp_tiled_image_sampled():
    """Image histograms (28 x 28 grid, d = 784, lambda = 0.01, 300
    iterations; B = 16): larger than a work-group's registers, so every
    product rebuilds the plan in a sweep over the cost.  The dense solve on
    three problems."""
    prob = workloads.make_config(3, B=16)
    check_sharp(prob, idx=np.array([0, 7, 15]), max_cg=1000)


def test_sharp_tiled_per_sample_ragged_zero_masses():
    """Per-sample costs, 300 x 520 (a ragged last column block), zero masses:
    gradients exactly 0 off the supports."""
    prob = workloads.random_problem(seed=45, B=3, d1=300, d2=520, lam=0.1, n_iter=300, c_batched=True,
                                    zero_frac=0.1)
    assert (prob.mu == 0).any() and (prob.nu == 0).any()
    out, _ = check_sharp(prob, max_cg=1000)
    assert np.all(out["grad_mu"].cpu().numpy()[prob.mu == 0] == 0)
    assert np.all(out["grad_nu"].cpu().numpy()[prob.nu == 0] == 0)


@pytest.mark.parametrize("d1,d2", [(129, 7), (9, 600), (250, 4096)])
def test_sharp_tiled_shapes(d1, d2):
    prob = workloads.random_problem(seed=500 + d1 + d2, B=2, d1=d1, d2=d2, lam=0.2, n_iter=200)
    check_sharp(prob, max_cg=1000)


def test_sharp_tiled_against_converged_oracle():
    """Both forwards converged (3000 iterations, lambda = 0.2): the GPU's sharp
    gradient from its own forward matches the oracle's from its own."""
    prob = workloads.random_problem(seed=46, B=2, d1=150, d2=200, lam=0.2, n_iter=3000)
    mu, nu, C = _t(prob.mu), _t(prob.nu), _t(prob.C)
    fw = sk.sinkhorn_forward(mu, nu, C, prob.lam, prob.n_iter)
    g = torch.ones(prob.B, device=DEV)
    out = sk.sinkhorn_backward_sharp(g, mu, nu, C, prob.lam, fw["alpha"], fw["beta"], max_cg=1000)
    o = oracle.forward(prob.mu, prob.nu, prob.C, prob.lam, prob.n_iter)
    ref = oracle.sharp_gradient(np.ones(prob.B), prob.mu, prob.nu, prob.C, prob.lam, o["alpha"], o["beta"])
    e1 = rel_err_rows(out["grad_mu"].cpu().numpy(), ref["grad_mu"])
    e2 = rel_err_rows(out["grad_nu"].cpu().numpy(), ref["grad_nu"])
    _say(f"   converged tiled: grad_mu {e1:.2e} grad_nu {e2:.2e} cg {out['cg_iters'].cpu().numpy().tolist()}")
    assert e1 <= GRAD_RTOL and e2 <= GRAD_RTOL


def test_sharp_tiled_iteration_cap_and_deterministic():
    prob = workloads.random_problem(seed=47, B=3, d1=200, d2=150, lam=0.1, n_iter=100)
    mu, nu, C = _t(prob.mu), _t(prob.nu), _t(prob.C)
    fw = sk.sinkhorn_forward(mu, nu, C, prob.lam, prob.n_iter)
    g = torch.ones(prob.B, device=DEV)
    capped = sk.sinkhorn_backward_sharp(g, mu, nu, C, prob.lam, fw["alpha"], fw["beta"], max_cg=3, cg_tol=0.0)
    assert np.all(capped["cg_iters"].cpu().numpy() == 3)
    a = sk.sinkhorn_backward_sharp(g, mu, nu, C, prob.lam, fw["alpha"], fw["beta"], max_cg=500)
    b = sk.sinkhorn_backward_sharp(g, mu, nu, C, prob.lam, fw["alpha"], fw["beta"], max_cg=500)
    for k in a:
        np.testing.assert_array_equal(a[k].cpu().numpy(), b[k].cpu().numpy())


def test_sharp_tiled_batch_above_grid_limit():
    """The tiled sharp gradient on 65537 problems (two chunks of the batch):
    problems on both sides of the boundary against the dense solve."""
    prob = workloads.random_problem(seed=95, B=65537, d1=130, d2=8, lam=0.2, n_iter=200)
    check_sharp(prob, idx=np.array([0, 65534, 65535, 65536]), max_cg=400)


@pytest.mark.parametrize("d1,d2,c_batched,zero_frac", [(140, 4100, False, 0.0), (5, 4500, True, 0.2)])
def test_sharp_tiled_wide_rows(d1, d2, c_batched, zero_frac):
    """Rows wider than 4096 columns: every product in two passes over the
    cost (rows, then columns); against the dense solve."""
    prob = workloads.random_problem(seed=97 + d2, B=2, d1=d1, d2=d2, lam=0.3, n_iter=150, c_batched=c_batched,
                                    zero_frac=zero_frac)
    check_sharp(prob, max_cg=1000)


def test_sharp_autograd_wrapper():
    prob = workloads.random_problem(seed=44, B=4, d1=24, d2=30, lam=0.1, n_iter=300)
    mu = _t(prob.mu).requires_grad_()
    nu = _t(prob.nu).requires_grad_()
    C = _t(prob.C[0])
    loss, st = sk.sinkhorn_loss(mu, nu, C, prob.lam, prob.n_iter, return_state=True, sharp=True)
    (loss * torch.arange(1, 5, device=DEV)).sum().backward()
    a, b = st["alpha"].detach().cpu().numpy(), st["beta"].detach().cpu().numpy()
    ref = oracle.sharp_gradient(np.arange(1, 5), prob.mu, prob.nu, prob.C, prob.lam, a, b)
    assert rel_err_rows(mu.grad.cpu().numpy(), ref["grad_mu"]) <= GRAD_RTOL
    assert rel_err_rows(nu.grad.cpu().numpy(), ref["grad_nu"]) <= GRAD_RTOL


def test_sharp_random_problems():
    """Twenty seeded random problems (d1, d2 <= 128, shared or per-sample,
    symmetric or not, zero masses, lambda in [0.05, 1]) against the dense solve."""
    rng = np.random.default_rng(77)
    for case in range(20):
        d1, d2 = int(rng.integers(1, 129)), int(rng.integers(1, 129))
        if rng.random() < 0.3:
            d2 = d1
        cost = "sym" if (d1 == d2 and rng.random() < 0.5) else "uniform"
        prob = workloads.random_problem(seed=int(rng.integers(1 << 30)), B=int(rng.integers(1, 7)), d1=d1, d2=d2,
                                        lam=float(10 ** rng.uniform(-1.3, 0.0)), n_iter=int(rng.integers(100, 400)),
                                        c_batched=bool(rng.random() < 0.4), zero_frac=float(rng.choice([0.0, 0.0, 0.2])),
                                        cost=cost)
        _say(f"[random {case}]")
        check_sharp(prob, seed=case)
