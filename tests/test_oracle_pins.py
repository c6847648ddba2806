"""Pins of the fp64 oracle against facts that do not come from the oracle itself.

Each test names the passage of the paper (arXiv:1907.01729) or the piece of
mathematics it rests on.  Together they are chosen so that a plausible slip in
the oracle -- a dropped term, a flipped sign, a transposed C, the wrong update
order or initialisation, a wrong gradient factor -- fails at least one of them
(see test_planted_mistakes_are_caught, which plants such slips in a numpy copy
of the iteration and checks that the same pins reject them).
"""
import itertools
import json
import os

import numpy as np
import pytest
from scipy.optimize import minimize

import oracle
import workloads

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _entropy(p):
    p = np.asarray(p, dtype=np.float64).ravel()
    p = p[p > 0]
    return float(-(p * np.log(p)).sum())


def _rand_hist(rng, n, lo=0.05):
    h = rng.uniform(lo, 1.0, n)
    return h / h.sum()


def _converged(mu, nu, C, lam, max_iter=400000, tol=1e-13):
    o = oracle.forward(mu, nu, C, lam, max_iter, tol=tol)
    return o


# --------------------------------------------------------------------------
# Closed forms
# --------------------------------------------------------------------------

def test_separable_cost_gives_product_coupling():
    """C_ij = a_i + b_j makes K = exp(-C/lambda) rank one, so one v-update and
    one u-update give P = mu nu^T exactly and E^0 = <a,mu> + <b,nu>
    (Section 1: P = diag(u) K diag(v) with the marginal equations)."""
    rng = np.random.default_rng(0)
    d1, d2 = 7, 5
    mu, nu = _rand_hist(rng, d1), _rand_hist(rng, d2)
    a, b = rng.uniform(0, 3, d1), rng.uniform(0, 3, d2)
    C = a[:, None] + b[None, :]
    for lam in (0.05, 1.0):
        for n_iter in (1, 3):
            o = oracle.forward(mu, nu, C, lam, n_iter)
            P = oracle.plan(C, lam, o["alpha"][0], o["beta"][0])
            np.testing.assert_allclose(P, np.outer(mu, nu), rtol=1e-12, atol=1e-15)
            assert o["loss"][0] == pytest.approx(a @ mu + b @ nu, rel=1e-12)
            assert o["marg_err"][0] < 1e-13


@pytest.mark.parametrize("d1,d2", [(1, 6), (6, 1), (1, 1)])
def test_single_point_marginal_gives_product_coupling(d1, d2):
    """With one point on either side the coupling set U holds only mu nu^T
    (Section 1), whatever C and lambda."""
    rng = np.random.default_rng(1)
    mu, nu = _rand_hist(rng, d1), _rand_hist(rng, d2)
    C = rng.uniform(0, 2, (d1, d2))
    o = oracle.forward(mu, nu, C, 0.01, 2)
    P = oracle.plan(C, 0.01, o["alpha"][0], o["beta"][0])
    np.testing.assert_allclose(P, np.outer(mu, nu), rtol=1e-12, atol=1e-15)
    assert o["loss"][0] == pytest.approx(float(mu @ C @ nu), rel=1e-12)


def test_large_lambda_tends_to_independent_coupling():
    """As lambda -> infinity the entropy term dominates E^lambda (Section 1),
    the minimiser tends to mu nu^T and E^0 to mu^T C nu, with an O(1/lambda)
    gap."""
    rng = np.random.default_rng(2)
    d1, d2 = 6, 8
    mu, nu = _rand_hist(rng, d1), _rand_hist(rng, d2)
    C = rng.uniform(0, 1, (d1, d2))
    ref = float(mu @ C @ nu)
    gaps = []
    for lam in (1e2, 1e3, 1e4):
        o = _converged(mu, nu, C, lam)
        gaps.append(abs(o["loss"][0] - ref))
    assert gaps[0] < 1e-2
    assert gaps[1] < gaps[0] / 5 and gaps[2] < gaps[1] / 5


# --------------------------------------------------------------------------
# Small-lambda limit: exact OT by brute force and by the 1-D closed form
# --------------------------------------------------------------------------

def _small_lambda_bound_ok(e0, w0, lam, mu, nu, merr, cmax):
    """0 <= E^0(P_lam) - W0 <= lam * min(h(mu), h(nu)) for the exact minimiser
    (from the entropy-constrained argument of Section 1 with
    h(P_lam) <= h(mu)+h(nu) and h(P_0) >= max(h(mu), h(nu))); the finite-
    iteration plan misses U by its marginal error, worth at most cmax*merr."""
    slack = cmax * merr + 1e-12
    gap = e0 - w0
    return -slack <= gap <= lam * min(_entropy(mu), _entropy(nu)) + slack, gap


def test_golden_assignment_problem():
    g = json.load(open(os.path.join(GOLD, "hungarian3.json")))
    C = np.array(g["C"], dtype=np.float64)
    mu = np.full(3, 1.0 / 3)
    assert min(g["permutation_costs"].values()) / 3 == pytest.approx(g["W0"])
    prev = None
    for lam in (0.5, 0.1, 0.02):
        o = _converged(mu, mu, C, lam)
        ok, gap = _small_lambda_bound_ok(o["loss"][0], g["W0"], lam, mu, mu, o["marg_err"][0], C.max())
        assert ok, (lam, gap)
        if prev is not None:
            assert gap <= prev + 1e-12
        prev = gap


@pytest.mark.parametrize("n", [3, 4, 5, 6])
def test_bruteforce_permutations_small_lambda(n):
    """Uniform masses: by Birkhoff the exact OT value is the best permutation
    average; compare E^0 of the entropic plan against it."""
    rng = np.random.default_rng(10 + n)
    C = rng.uniform(0, 1, (n, n))
    mu = np.full(n, 1.0 / n)
    w0 = min(sum(C[i, s[i]] for i in range(n)) / n for s in itertools.permutations(range(n)))
    for lam in (0.1, 0.03):
        o = _converged(mu, mu, C, lam)
        ok, gap = _small_lambda_bound_ok(o["loss"][0], w0, lam, mu, mu, o["marg_err"][0], C.max())
        assert ok, (n, lam, gap)


def test_golden_w1_with_zero_masses():
    g = json.load(open(os.path.join(GOLD, "w1_halves.json")))
    x = np.array(g["x"], dtype=np.float64)
    mu, nu = np.array(g["mu"]), np.array(g["nu"])
    C = np.abs(x[:, None] - x[None, :])
    o = _converged(mu, nu, C, 0.05)
    # zero masses carry -inf potentials (Section 3)
    assert np.all(np.isneginf(o["alpha"][0][2:])) and np.all(np.isneginf(o["beta"][0][:2]))
    assert np.all(np.isfinite(o["alpha"][0][:2])) and np.all(np.isfinite(o["beta"][0][2:]))
    ok, gap = _small_lambda_bound_ok(o["loss"][0], g["W1"], 0.05, mu[mu > 0], nu[nu > 0],
                                     o["marg_err"][0], C.max())
    assert ok, gap


@pytest.mark.parametrize("lam", [0.02, 0.005])
def test_1d_w1_closed_form(lam):
    """On a line with cost |x_i - x_j|, W1 = sum_k |F_mu(k) - F_nu(k)| dx."""
    rng = np.random.default_rng(3)
    n = 24
    x = np.linspace(0.0, 1.0, n)
    C = np.abs(x[:, None] - x[None, :])
    mu, nu = _rand_hist(rng, n, 0.1), _rand_hist(rng, n, 0.1)
    w1 = float(np.abs(np.cumsum(mu) - np.cumsum(nu))[:-1].sum() * (x[1] - x[0]))
    o = _converged(mu, nu, C, lam)
    ok, gap = _small_lambda_bound_ok(o["loss"][0], w1, lam, mu, nu, o["marg_err"][0], 1.0)
    assert ok, gap


# --------------------------------------------------------------------------
# Independent solver: the entropic dual maximised by scipy
# --------------------------------------------------------------------------

def _scipy_dual(mu, nu, C, lam):
    """Maximise D(f,g) = <f,mu> + <g,nu> - lam sum exp((f_i+g_j-C_ij)/lam - 1),
    the Lagrangian dual of min_U sum PC + lam sum P log P (Section 1's
    augmented functional with the minimisation over P carried out)."""
    d1, d2 = C.shape

    def negD(z):
        f, g = z[:d1], z[d1:]
        E = np.exp((f[:, None] + g[None, :] - C) / lam - 1.0)
        val = f @ mu + g @ nu - lam * E.sum()
        grad = np.concatenate([mu - E.sum(1), nu - E.sum(0)])
        return -val, -grad

    r = minimize(negD, np.zeros(d1 + d2), jac=True, method="L-BFGS-B",
                 options=dict(maxiter=100000, ftol=1e-15, gtol=1e-12, maxcor=50))
    f, g = r.x[:d1], r.x[d1:]
    return -r.fun, f, g


@pytest.mark.parametrize("d1,d2,lam", [(4, 6, 0.5), (5, 3, 0.2), (6, 6, 0.1)])
def test_scipy_dual_matches(d1, d2, lam):
    """Non-symmetric C and d1 != d2, so a transposed C or swapped roles of
    alpha/beta fail.  Converged W_lambda, the plan and the gauge-fixed
    potentials must match the scipy optimum: P = exp((f+g-C)/lam - 1) so
    alpha = f/lam - 1/2 + c, beta = g/lam - 1/2 - c for some constant c."""
    rng = np.random.default_rng(100 + d1 * 10 + d2)
    mu, nu = _rand_hist(rng, d1), _rand_hist(rng, d2)
    C = rng.uniform(0, 1, (d1, d2))
    W, f, g = _scipy_dual(mu, nu, C, lam)
    o = _converged(mu, nu, C, lam)
    a, b = o["alpha"][0], o["beta"][0]
    obj = oracle.objectives(mu, nu, C, lam, a, b)
    assert obj["dual"] == pytest.approx(W, abs=1e-8)
    assert obj["primal"] == pytest.approx(W, abs=1e-8)
    P = oracle.plan(C, lam, a, b)
    Pref = np.exp((f[:, None] + g[None, :] - C) / lam - 1.0)
    np.testing.assert_allclose(P, Pref, atol=1e-7)
    af, bf = f / lam - 0.5, g / lam - 0.5
    s = (a - af).mean()
    np.testing.assert_allclose(a - s, af, atol=1e-5)
    np.testing.assert_allclose(b + s, bf, atol=1e-5)


# --------------------------------------------------------------------------
# Finite-iteration semantics: the plain-domain iteration of Section 1
# --------------------------------------------------------------------------

def _plain_sk(mu, nu, C, lam, n_iter):
    """eq. (sk_plain): v = nu / (K^T u), then u = mu / (K v), from u^0 = 1."""
    K = np.exp(-C / lam)
    u = np.ones(len(mu))
    v = np.ones(len(nu))
    for _ in range(n_iter):
        v = nu / (K.T @ u)
        u = mu / (K @ v)
    return u, v


@pytest.mark.parametrize("n_iter", [1, 2, 7])
def test_log_domain_matches_plain_iteration(n_iter):
    """At every finite k the log-domain iterate equals the plain one of
    eq. (sk_plain) (Section 3 rewrites it in log space): alpha = log u,
    beta = log v.  Fixes the update order (v first), the initialisation and
    both logsumexp signs.  lambda is large enough that K does not underflow."""
    rng = np.random.default_rng(5)
    d1, d2 = 9, 6
    mu, nu = _rand_hist(rng, d1), _rand_hist(rng, d2)
    C = rng.uniform(0, 1, (d1, d2))
    for lam in (0.05, 0.3):
        u, v = _plain_sk(mu, nu, C, lam, n_iter)
        o = oracle.forward(mu, nu, C, lam, n_iter)
        np.testing.assert_allclose(o["alpha"][0], np.log(u), rtol=1e-11, atol=1e-11)
        np.testing.assert_allclose(o["beta"][0], np.log(v), rtol=1e-11, atol=1e-11)
        P = u[:, None] * np.exp(-C / lam) * v[None, :]
        assert o["loss"][0] == pytest.approx((P * C).sum(), rel=1e-11)
        merr = np.abs(P.sum(1) - mu).sum() + np.abs(P.sum(0) - nu).sum()
        assert o["marg_err"][0] == pytest.approx(merr, rel=1e-6, abs=1e-14)


def test_row_marginal_exact_after_u_update():
    """The iteration alternately enforces each marginal (Section 1): after the
    u-update, P 1 = mu to rounding, while P^T 1 - nu is what is left."""
    rng = np.random.default_rng(6)
    mu, nu = _rand_hist(rng, 8), _rand_hist(rng, 11)
    C = rng.uniform(0, 1, (8, 11))
    o = oracle.forward(mu, nu, C, 0.05, 3)
    P = oracle.plan(C, 0.05, o["alpha"][0], o["beta"][0])
    np.testing.assert_allclose(P.sum(1), mu, rtol=1e-13)
    assert np.abs(P.sum(0) - nu).sum() > 1e-6


def test_gauge_invariance_of_plan_and_loss():
    """Multipliers are defined up to (c, -c) (Section 1): shifting alpha by c and
    beta by -c leaves P, E^0 and the gradients unchanged."""
    rng = np.random.default_rng(7)
    mu, nu = _rand_hist(rng, 5), _rand_hist(rng, 7)
    C = rng.uniform(0, 1, (5, 7))
    o = oracle.forward(mu, nu, C, 0.1, 20)
    a, b = o["alpha"][0], o["beta"][0]
    P0 = oracle.plan(C, 0.1, a, b)
    P1 = oracle.plan(C, 0.1, a + 3.7, b - 3.7)
    np.testing.assert_allclose(P0, P1, rtol=1e-13)
    g0 = oracle.backward([1.0], mu, nu, C, 0.1, a, b)
    g1 = oracle.backward([1.0], mu, nu, C, 0.1, a + 3.7, b - 3.7)
    np.testing.assert_allclose(g0["grad_mu"], g1["grad_mu"], atol=1e-13)
    np.testing.assert_allclose(g0["grad_nu"], g1["grad_nu"], atol=1e-13)


def test_transposition_at_convergence():
    """Swapping the roles (nu, mu, C^T) gives P^T at the fixed point."""
    rng = np.random.default_rng(8)
    mu, nu = _rand_hist(rng, 5), _rand_hist(rng, 7)
    C = rng.uniform(0, 1, (5, 7))
    o = _converged(mu, nu, C, 0.1)
    t = _converged(nu, mu, C.T.copy(), 0.1)
    P = oracle.plan(C, 0.1, o["alpha"][0], o["beta"][0])
    Pt = oracle.plan(C.T, 0.1, t["alpha"][0], t["beta"][0])
    np.testing.assert_allclose(P, Pt.T, atol=1e-12)
    assert o["loss"][0] == pytest.approx(t["loss"][0], rel=1e-11)


# --------------------------------------------------------------------------
# Gradients against finite differences (Section 2)
# --------------------------------------------------------------------------

def _W(mu, nu, C, lam):
    o = _converged(mu, nu, C, lam)
    return oracle.objectives(mu, nu, C, lam, o["alpha"][0], o["beta"][0])["dual"], o


@pytest.mark.parametrize("lam", [0.05, 0.5])
def test_fd_gradient_mu_nu(lam):
    """d W_lambda along e_i - e_k (a mean-zero move on the simplex) equals
    <grad, e_i - e_k> with grad = lambda (alpha - mean alpha) (Section 2, with
    the sign fixed by the Lagrangian of Section 1)."""
    rng = np.random.default_rng(9)
    d1, d2 = 6, 5
    mu, nu = _rand_hist(rng, d1), _rand_hist(rng, d2)
    C = rng.uniform(0, 1, (d1, d2))
    _, o = _W(mu, nu, C, lam)
    g = oracle.backward([1.0], mu, nu, C, lam, o["alpha"], o["beta"])
    assert abs(g["grad_mu"].sum()) < 1e-12 and abs(g["grad_nu"].sum()) < 1e-12
    h = 1e-6
    for (i, k) in [(0, 3), (2, 5), (4, 1)]:
        e = np.zeros(d1); e[i], e[k] = 1.0, -1.0
        fd = (_W(mu + h * e, nu, C, lam)[0] - _W(mu - h * e, nu, C, lam)[0]) / (2 * h)
        assert fd == pytest.approx(g["grad_mu"][0] @ e, abs=1e-7, rel=1e-6)
    for (j, k) in [(0, 4), (3, 1)]:
        e = np.zeros(d2); e[j], e[k] = 1.0, -1.0
        fd = (_W(mu, nu + h * e, C, lam)[0] - _W(mu, nu - h * e, C, lam)[0]) / (2 * h)
        assert fd == pytest.approx(g["grad_nu"][0] @ e, abs=1e-7, rel=1e-6)


def test_fd_gradient_C():
    """d W_lambda / d C_ij = P_ij (envelope theorem); scaled by g, and summed
    over the batch for a shared C.  Row and column sums of grad_C are g mu and
    g nu."""
    rng = np.random.default_rng(11)
    d1, d2, lam = 4, 5, 0.1
    mu, nu = _rand_hist(rng, d1), _rand_hist(rng, d2)
    C = rng.uniform(0, 1, (d1, d2))
    _, o = _W(mu, nu, C, lam)
    g = oracle.backward([2.5], mu, nu, C, lam, o["alpha"], o["beta"], grad_C=True)["grad_C"][0]
    h = 1e-6
    for (i, j) in [(0, 0), (1, 3), (3, 4)]:
        E = np.zeros_like(C); E[i, j] = 1.0
        fd = (_W(mu, nu, C + h * E, lam)[0] - _W(mu, nu, C - h * E, lam)[0]) / (2 * h)
        assert 2.5 * fd == pytest.approx(g[i, j], rel=1e-6, abs=1e-9)
    np.testing.assert_allclose(g.sum(1), 2.5 * mu, rtol=1e-9)
    np.testing.assert_allclose(g.sum(0), 2.5 * nu, rtol=1e-9)


def test_grad_C_shared_is_batch_sum():
    rng = np.random.default_rng(12)
    B, d1, d2, lam = 3, 4, 6, 0.2
    mu = np.stack([_rand_hist(rng, d1) for _ in range(B)])
    nu = np.stack([_rand_hist(rng, d2) for _ in range(B)])
    C = rng.uniform(0, 1, (d1, d2))
    o = oracle.forward(mu, nu, C, lam, 50)
    gl = np.array([0.5, -1.0, 2.0])
    shared = oracle.backward(gl, mu, nu, C, lam, o["alpha"], o["beta"], grad_C=True)["grad_C"][0]
    Cb = np.broadcast_to(C, (B, d1, d2)).copy()
    ob = oracle.forward(mu, nu, Cb, lam, 50)
    per = oracle.backward(gl, mu, nu, Cb, lam, ob["alpha"], ob["beta"], grad_C=True)["grad_C"]
    np.testing.assert_allclose(shared, per.sum(0), rtol=1e-12)
    for b in range(B):
        np.testing.assert_allclose(per[b], gl[b] * oracle.plan(C, lam, o["alpha"][b], o["beta"][b]),
                                   rtol=1e-12)


def test_zero_mass_gradient_is_zero_off_support():
    rng = np.random.default_rng(13)
    mu = _rand_hist(rng, 6); mu[2] = 0.0; mu /= mu.sum()
    nu = _rand_hist(rng, 5); nu[0] = 0.0; nu /= nu.sum()
    C = rng.uniform(0, 1, (6, 5))
    o = oracle.forward(mu, nu, C, 0.1, 30)
    g = oracle.backward([1.0], mu, nu, C, 0.1, o["alpha"], o["beta"])
    assert g["grad_mu"][0][2] == 0.0 and g["grad_nu"][0][0] == 0.0
    assert abs(g["grad_mu"][0].sum()) < 1e-12 and np.all(np.isfinite(g["grad_mu"]))


# --------------------------------------------------------------------------
# Early stopping and batching semantics
# --------------------------------------------------------------------------

def test_tol_stops_at_first_iterate_below_tol():
    rng = np.random.default_rng(14)
    B = 3
    mu = np.stack([_rand_hist(rng, 7) for _ in range(B)])
    nu = np.stack([_rand_hist(rng, 9) for _ in range(B)])
    C = rng.uniform(0, 1, (7, 9))
    tol = 1e-6
    o = oracle.forward(mu, nu, C, 0.1, 500, tol=tol, err_hist=True)
    for b in range(B):
        K = o["iters"][b]
        assert 1 <= K < 500
        h = o["err_hist"][b]
        assert h[K - 1] <= tol and np.all(h[: K - 1] > tol)
        r = oracle.forward(mu[b:b + 1], nu[b:b + 1], C, 0.1, int(K))
        np.testing.assert_array_equal(r["alpha"][0], o["alpha"][b])
        assert r["marg_err"][0] == pytest.approx(h[K - 1], rel=1e-12)
    # per-sample counts reproduce the same iterates in one batched call
    r = oracle.forward(mu, nu, C, 0.1, 0, n_iter_b=o["iters"])
    np.testing.assert_array_equal(r["alpha"], o["alpha"])


def test_batch_members_are_independent():
    """A sample's result does not depend on the rest of the batch."""
    rng = np.random.default_rng(15)
    B = 4
    mu = np.stack([_rand_hist(rng, 5) for _ in range(B)])
    nu = np.stack([_rand_hist(rng, 6) for _ in range(B)])
    C = rng.uniform(0, 1, (5, 6))
    o = oracle.forward(mu, nu, C, 0.07, 40)
    s = oracle.forward(mu[2:3], nu[2:3], C, 0.07, 40)
    np.testing.assert_array_equal(s["alpha"][0], o["alpha"][2])
    np.testing.assert_array_equal(s["beta"][0], o["beta"][2])


def test_zero_iterations():
    """n_iter = 0 returns the initial potentials (0 on the support)."""
    rng = np.random.default_rng(16)
    mu, nu = _rand_hist(rng, 3), _rand_hist(rng, 4)
    C = rng.uniform(0, 1, (3, 4))
    o = oracle.forward(mu, nu, C, 0.1, 0)
    assert np.all(o["alpha"] == 0) and np.all(o["beta"] == 0) and o["iters"][0] == 0


def test_invalid_arguments_raise():
    with pytest.raises(ValueError):
        oracle.forward(np.ones((1, 3)) / 3, np.ones((1, 3)) / 3, np.zeros((3, 3)), 0.0, 5)
    with pytest.raises(ValueError):
        oracle.forward(np.ones((1, 3)) / 3, np.ones((1, 3)) / 3, np.zeros((3, 3)), 0.1, -1)


# --------------------------------------------------------------------------
# The pins above reject plausible mistakes
# --------------------------------------------------------------------------

def _mutant_sk(mu, nu, C, lam, n_iter, mutation):
    """A numpy log-domain iteration with one planted mistake (CPU only)."""
    la, lb = np.log(mu), np.log(nu)
    a = np.zeros(len(mu))
    b = np.zeros(len(nu))

    def lse(x, axis):
        m = x.max(axis=axis, keepdims=True)
        return (m + np.log(np.exp(x - m).sum(axis=axis, keepdims=True))).squeeze(axis)

    Cs = C.T if mutation == "transposed" else C
    sgn = 1.0 if mutation == "cost_sign" else -1.0
    for _ in range(n_iter):
        if mutation == "u_first":
            a = la - lse(b[None, :] + sgn * Cs / lam, 1)
            b = lb - lse(a[:, None] + sgn * Cs / lam, 0)
        else:
            b = lb - lse(a[:, None] + sgn * Cs / lam, 0)
            a = la - lse(b[None, :] + sgn * Cs / lam, 1)
            if mutation == "dropped_potential":
                a = la - lse(sgn * Cs / lam + 0.0 * b[None, :], 1)
    return a, b


@pytest.mark.parametrize("mutation", ["transposed", "cost_sign", "u_first", "dropped_potential"])
def test_planted_mistakes_are_caught(mutation):
    """Each planted mistake breaks the plain-iteration pin or the scipy pin."""
    rng = np.random.default_rng(17)
    d = 6
    mu, nu = _rand_hist(rng, d), _rand_hist(rng, d)
    C = rng.uniform(0, 1, (d, d))
    lam = 0.3
    a, b = _mutant_sk(mu, nu, C, lam, 3, mutation)
    u, v = _plain_sk(mu, nu, C, lam, 3)
    finite_k_ok = np.allclose(a, np.log(u), atol=1e-9) and np.allclose(b, np.log(v), atol=1e-9)
    a2, b2 = _mutant_sk(mu, nu, C, lam, 3000, mutation)
    W, f, g = _scipy_dual(mu, nu, C, lam)
    dual_ok = abs(lam * (a2 @ mu + b2 @ nu) - W) < 1e-6
    assert not (finite_k_ok and dual_ok), mutation


# --------------------------------------------------------------------------
# Point clouds: the cost recreated from coordinates (Section 4's closing
# remark) and the gradient with respect to the points (chain rule through
# dW/dC = P)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("D", [1, 2, 3, 5])
def test_cost_from_points_matches_cdist(D):
    """The oracle's squared distances equal scipy's cdist('sqeuclidean') (an
    independent library routine), per cloud pair."""
    from scipy.spatial.distance import cdist
    p = workloads.random_points(40 + D, B=3, d1=7, d2=11, D=D, lam=0.1, n_iter=1, offset=3.0)
    C = oracle.cost_from_points(p.X, p.Y)
    for b in range(3):
        ref = cdist(p.X[b].astype(np.float64), p.Y[b].astype(np.float64), "sqeuclidean")
        np.testing.assert_allclose(C[b], ref, rtol=1e-12, atol=1e-12)


def _points_grads_fd_case(mutation=None):
    rng = np.random.default_rng(23)
    d1, d2, D, lam = 4, 5, 2, 0.3
    mu, nu = _rand_hist(rng, d1), _rand_hist(rng, d2)
    X = rng.standard_normal((d1, D))
    Y = rng.standard_normal((d2, D)) + 0.5
    C = oracle.cost_from_points(X, Y)[0]
    _, o = _W(mu, nu, C, lam)
    G = oracle.backward([1.0], mu, nu, C, lam, o["alpha"], o["beta"], grad_C=True)["grad_C"]
    gX, gY = oracle.points_grads(G, X, Y)
    if mutation == "sign":
        gX = -gX
    elif mutation == "factor":
        gX = 0.5 * gX
    h = 1e-6
    ok = True
    for (i, k) in [(0, 0), (2, 1), (3, 0)]:
        E = np.zeros_like(X); E[i, k] = 1.0
        fd = (_W(mu, nu, oracle.cost_from_points(X + h * E, Y)[0], lam)[0]
              - _W(mu, nu, oracle.cost_from_points(X - h * E, Y)[0], lam)[0]) / (2 * h)
        ok &= abs(fd - gX[0, i, k]) <= 1e-6 * max(1.0, abs(fd))
    for (j, k) in [(1, 1), (4, 0)]:
        E = np.zeros_like(Y); E[j, k] = 1.0
        fd = (_W(mu, nu, oracle.cost_from_points(X, Y + h * E)[0], lam)[0]
              - _W(mu, nu, oracle.cost_from_points(X, Y - h * E)[0], lam)[0]) / (2 * h)
        ok &= abs(fd - gY[0, j, k]) <= 1e-6 * max(1.0, abs(fd))
    return ok, gX, gY


def test_fd_gradient_points():
    """d W_lambda / d X and d Y by central differences of the converged dual
    match the chain rule through dW/dC = P; translating both clouds together
    leaves C unchanged, so the gradients sum to zero over all points."""
    ok, gX, gY = _points_grads_fd_case()
    assert ok
    np.testing.assert_allclose(gX.sum(axis=(0, 1)) + gY.sum(axis=(0, 1)), 0.0, atol=1e-12)


@pytest.mark.parametrize("mutation", ["sign", "factor"])
def test_points_grads_planted_mistakes_are_caught(mutation):
    ok, _, _ = _points_grads_fd_case(mutation)
    assert not ok


# --------------------------------------------------------------------------
# Gradient of the sharp loss E^0 (implicit differentiation of the plan)
# --------------------------------------------------------------------------

def _E0(mu, nu, C, lam):
    o = _converged(mu, nu, C, lam)
    return o["loss"][0], o


@pytest.mark.parametrize("lam", [0.05, 0.3])
def test_fd_sharp_gradient(lam):
    """d E^0 along mean-zero moves e_i - e_k of mu (and of nu), by central
    differences of the converged E^0 = <P, C>, matches <grad, e> from the
    implicit-differentiation solve; it differs from the multiplier gradient by
    O(lambda) (Section 5: the multiplier gradient is that of E^lambda)."""
    rng = np.random.default_rng(31)
    d1, d2 = 6, 5
    mu, nu = _rand_hist(rng, d1), _rand_hist(rng, d2)
    C = rng.uniform(0, 1, (d1, d2))
    _, o = _E0(mu, nu, C, lam)
    gs = oracle.sharp_gradient([1.0], mu, nu, C, lam, o["alpha"], o["beta"])
    gm = oracle.backward([1.0], mu, nu, C, lam, o["alpha"], o["beta"])
    h = 1e-6
    for (i, k) in [(0, 3), (2, 5), (4, 1)]:
        e = np.zeros(d1); e[i], e[k] = 1.0, -1.0
        fd = (_E0(mu + h * e, nu, C, lam)[0] - _E0(mu - h * e, nu, C, lam)[0]) / (2 * h)
        assert fd == pytest.approx(gs["grad_mu"][0] @ e, abs=1e-7, rel=1e-5)
    for (j, k) in [(0, 4), (3, 1)]:
        e = np.zeros(d2); e[j], e[k] = 1.0, -1.0
        fd = (_E0(mu, nu + h * e, C, lam)[0] - _E0(mu, nu - h * e, C, lam)[0]) / (2 * h)
        assert fd == pytest.approx(gs["grad_nu"][0] @ e, abs=1e-7, rel=1e-5)
    # the two gradients differ (the multiplier one is that of E^lambda, not E^0)
    assert np.abs(gs["grad_mu"] - gm["grad_mu"]).max() > 1e-4


def test_sharp_gradient_zero_mass_and_batch():
    """Zero masses get gradient 0 and leave the support's system unchanged;
    each problem of a batch is independent; grad_loss scales each problem."""
    rng = np.random.default_rng(33)
    d1, d2, lam = 6, 7, 0.1
    mu = np.stack([_rand_hist(rng, d1) for _ in range(2)])
    nu = np.stack([_rand_hist(rng, d2) for _ in range(2)])
    mu[1, 2] = 0.0; mu[1] /= mu[1].sum()
    C = rng.uniform(0, 1, (d1, d2))
    o = oracle.forward(mu, nu, C, lam, 3000)
    g = oracle.sharp_gradient([2.0, 0.5], mu, nu, C, lam, o["alpha"], o["beta"])
    assert g["grad_mu"][1, 2] == 0.0
    one = oracle.sharp_gradient([1.0], mu[1:], nu[1:], C, lam, o["alpha"][1:], o["beta"][1:])
    np.testing.assert_allclose(g["grad_mu"][1], 0.5 * one["grad_mu"][0], rtol=1e-10, atol=1e-14)
    np.testing.assert_allclose(g["grad_mu"][1, [0, 1, 3, 4, 5]].sum(), 0.0, atol=1e-12)


@pytest.mark.parametrize("mutation", ["no_coupling", "lambda_factor", "multiplier_rhs"])
def test_sharp_gradient_planted_mistakes_are_caught(mutation):
    """Plausible mistakes in the implicit-differentiation system (dropping the
    plan coupling, a stray lambda, the marginals instead of the cost-weighted
    sums on the right-hand side) disagree with the finite differences that
    pin the oracle."""
    rng = np.random.default_rng(34)
    d1, d2, lam = 5, 6, 0.1
    mu, nu = _rand_hist(rng, d1), _rand_hist(rng, d2)
    C = rng.uniform(0, 1, (d1, d2))
    _, o = _E0(mu, nu, C, lam)
    P = oracle.plan(C, lam, o["alpha"][0], o["beta"][0])
    H = np.block([[np.diag(P.sum(1)), P], [P.T, np.diag(P.sum(0))]])
    rhs = np.concatenate([(P * C).sum(1), (P * C).sum(0)])
    if mutation == "no_coupling":
        H = np.diag(np.diag(H))
    elif mutation == "lambda_factor":
        rhs = lam * rhs
    elif mutation == "multiplier_rhs":
        rhs = np.concatenate([P.sum(1), P.sum(0)])
    z = np.linalg.lstsq(H, rhs, rcond=None)[0][:d1]
    e = np.zeros(d1); e[1], e[3] = 1.0, -1.0
    h = 1e-6
    fd = (_E0(mu + h * e, nu, C, lam)[0] - _E0(mu - h * e, nu, C, lam)[0]) / (2 * h)
    good = oracle.sharp_gradient([1.0], mu, nu, C, lam, o["alpha"], o["beta"])["grad_mu"][0] @ e
    assert fd == pytest.approx(good, rel=1e-5, abs=1e-7)
    assert abs((z - z.mean()) @ e - fd) > 1e-4, mutation


# --------------------------------------------------------------------------
# Warm start: a given log u^0 instead of 0 (the resume of the iteration)
# --------------------------------------------------------------------------

def _plain_sk_from(mu, nu, C, lam, n_iter, u0):
    """eq. (sk_plain) from a given u^0: v = nu / (K^T u), then u = mu / (K v)."""
    K = np.exp(-C / lam)
    u = u0.copy()
    v = np.ones(len(nu))
    for _ in range(n_iter):
        v = nu / (K.T @ u)
        u = mu / (K @ v)
    return u, v


@pytest.mark.parametrize("n_iter", [1, 3, 8])
def test_warm_start_matches_plain_iteration_from_u0(n_iter):
    """A warm start is the plain iteration of eq. (sk_plain) started from
    u^0 = exp(alpha0) (an independent algorithm): it fixes that alpha0 is the
    start and that the first half-step is the v-update from it."""
    rng = np.random.default_rng(17)
    d1, d2, lam = 8, 5, 0.2
    mu, nu = _rand_hist(rng, d1), _rand_hist(rng, d2)
    C = rng.uniform(0, 1, (d1, d2))
    a0 = rng.normal(0.0, 2.0, d1)
    u, v = _plain_sk_from(mu, nu, C, lam, n_iter, np.exp(a0))
    o = oracle.forward(mu, nu, C, lam, n_iter, alpha0=a0[None])
    np.testing.assert_allclose(o["alpha"][0], np.log(u), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(o["beta"][0], np.log(v), rtol=1e-11, atol=1e-11)
    cold = oracle.forward(mu, nu, C, lam, n_iter)
    assert np.abs(cold["alpha"][0] - o["alpha"][0]).max() > 1e-6  # the start matters at finite n_iter


def test_warm_start_resumes_the_iteration():
    """K iterations, then n more from their alpha, are K + n iterations
    (alpha is the whole state): identical in every bit, per sample, with zero
    masses and a per-sample cost."""
    rng = np.random.default_rng(23)
    B, d1, d2, lam = 3, 9, 7, 0.1
    mu = np.stack([_rand_hist(rng, d1) for _ in range(B)])
    nu = np.stack([_rand_hist(rng, d2) for _ in range(B)])
    mu[1, 2] = 0.0
    mu[1] /= mu[1].sum()
    nu[2, 0] = 0.0
    nu[2] /= nu[2].sum()
    C = rng.uniform(0, 1, (B, d1, d2))
    first = oracle.forward(mu, nu, C, lam, 11)
    resumed = oracle.forward(mu, nu, C, lam, 6, alpha0=first["alpha"])
    whole = oracle.forward(mu, nu, C, lam, 17)
    for k in ("alpha", "beta", "loss", "marg_err"):
        np.testing.assert_array_equal(resumed[k], whole[k])


def test_warm_start_at_the_optimum_stays_there():
    """Started at the optimum of the entropic dual found by scipy (an
    independent solver), one iteration keeps the plan: the marginal error
    stays at the optimum's and the loss is the optimal plan's E^0."""
    rng = np.random.default_rng(29)
    d1, d2, lam = 6, 4, 0.3
    mu, nu = _rand_hist(rng, d1), _rand_hist(rng, d2)
    C = rng.uniform(0, 1, (d1, d2))
    _, f, g = _scipy_dual(mu, nu, C, lam)
    a_star = f / lam - 0.5  # log u of P = exp((f + g - C) / lam - 1), up to the gauge
    Pref = np.exp((f[:, None] + g[None, :] - C) / lam - 1.0)
    o = oracle.forward(mu, nu, C, lam, 1, alpha0=a_star[None])
    assert o["marg_err"][0] <= 1e-7
    assert o["loss"][0] == pytest.approx((Pref * C).sum(), rel=1e-7)
    np.testing.assert_allclose(oracle.plan(C, lam, o["alpha"][0], o["beta"][0]), Pref, atol=1e-7)


def test_warm_start_ignores_entries_off_the_support():
    """alpha0 is read on the support of mu only: -inf off it whatever alpha0
    holds there; a warm start from 0 on the support is the cold start."""
    rng = np.random.default_rng(31)
    d1, d2, lam = 7, 6, 0.2
    mu, nu = _rand_hist(rng, d1), _rand_hist(rng, d2)
    mu[3] = 0.0
    mu /= mu.sum()
    C = rng.uniform(0, 1, (d1, d2))
    a0 = np.zeros((1, d1))
    a0[0, 3] = 123.0
    warm = oracle.forward(mu, nu, C, lam, 5, alpha0=a0)
    cold = oracle.forward(mu, nu, C, lam, 5)
    for k in ("alpha", "beta", "loss"):
        np.testing.assert_array_equal(warm[k], cold[k])
    assert np.isneginf(warm["alpha"][0, 3])
