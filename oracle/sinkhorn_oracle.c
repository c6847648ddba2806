/*
 * sinkhorn_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 CPU implementation of batched log-domain Sinkhorn
 * (Viehmann, "Implementation of batched Sinkhorn iterations for
 * entropy-regularized Wasserstein loss", arXiv:1907.01729).  It exists to
 * check the GPU library against; it is not part of the product.  Only the
 * test suite, the smoke check and the benchmark's CPU-baseline leg may load
 * it.  It shares no code, header, table or helper with the HIP library.
 *
 * Everything is computed in double precision with the host libm exp/log,
 * in the order the paper states, without blocking, fusion or reordering
 * beyond loop interchange of independent sums.
 *
 * Notation (paper, Section 1, eq. (pij_form) and the definitions after it):
 *   P = diag(u) K diag(v),  K = exp(-C / lambda),
 *   alpha = log u, beta = log v   (dimensionless log-scalings; the paper's
 *   Lagrange multipliers in cost units are an affine function of these).
 *   So P_ij = exp(alpha_i + beta_j - C_ij / lambda).
 *
 * Readings taken where the paper is silent or garbled:
 *   - The log-domain update (Section 3, eq. (log_sk)) is printed with both
 *     logsumexp arguments sign-flipped; the batched form in Section 4 has the
 *     consistent sign, LSE_i(-C_ij/lambda + log u_i).  That form is used, and
 *     its row counterpart for the u-update.
 *   - Initialisation: log u^0 = 0 on the support of mu, -inf off it; or, for
 *     a warm start (a resume of the iteration; not in the paper), a given
 *     log u^0 on the support of mu, -inf off it.  Every iteration begins
 *     with the v-update from log u alone, so log u is the iteration's whole
 *     state: K iterations, then n more from their log u, are K + n.
 *   - One iteration = v-update then u-update (order of eq. (sk_plain)).
 *   - Zero mass: log u_i = -inf where mu_i = 0, log v_j = -inf where nu_j = 0
 *     (Section 3).
 *   - Early stop (the paper uses none, Section 5): per sample, after the
 *     u-update of iteration k < n_iter, if the marginal L1 error of the
 *     iterate k is <= tol the sample stops with K = k.  tol <= 0 disables it.
 *   - Loss = E^0(P) = sum_ij P_ij C_ij of the returned iterate (Section 5,
 *     the plain definition of E^0 from Section 1; the printed eq.
 *     (E0_calculation) is garbled, its plain left-hand side is used).
 *   - Gradient (Section 2) = lambda * (alpha - mean alpha) for mu, likewise
 *     for nu; this is the gradient of W_lambda(mu,nu) = min E^lambda.  The
 *     mean is over the support (the projection onto mean-zero variations of
 *     the face); zero-mass entries get 0.  grad_C = P (envelope theorem,
 *     consistent with Section 2's multiplier view; the paper does not state
 *     it).  Each is scaled by the incoming per-sample gradient g_b; a shared
 *     C gets sum_b g_b P_b.
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define NEG_INF (-INFINITY)

static int n_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Two-pass logsumexp of x[0..n) with stride: max first, then sum of
 * exp(x - max).  All -inf gives -inf.  (Section 3: "extracting the maximum
 * before exponentiation".) */
static double lse_strided(const double *x, long n, long stride)
{
    double m = NEG_INF;
    for (long k = 0; k < n; ++k) {
        double v = x[k * stride];
        if (v > m) m = v;
    }
    if (m == NEG_INF) return NEG_INF;
    double s = 0.0;
    for (long k = 0; k < n; ++k) s += exp(x[k * stride] - m);
    return m + log(s);
}

/* v-update (Section 4, batched form): for every column j,
 *   beta_j = log nu_j - LSE_i(alpha_i - C_ij / lambda).
 * x is scratch of size d1 (serial) -- the column is gathered into it so the
 * same logsumexp routine is used as for rows. */
static void v_update(int d1, int d2, double lam, const double *C,
                     const double *alpha, const double *nu, double *beta,
                     int par)
{
#pragma omp parallel for schedule(static) if (par)
    for (int j = 0; j < d2; ++j) {
        if (!(nu[j] > 0.0)) { beta[j] = NEG_INF; continue; }
        double *x = (double *)malloc(sizeof(double) * (size_t)d1);
        for (int i = 0; i < d1; ++i)
            x[i] = alpha[i] - C[(long)i * d2 + j] / lam;
        beta[j] = log(nu[j]) - lse_strided(x, d1, 1);
        free(x);
    }
}

/* u-update (Section 3, row form with the Section 4 sign): for every row i,
 *   alpha_i = log mu_i - LSE_j(beta_j - C_ij / lambda). */
static void u_update(int d1, int d2, double lam, const double *C,
                     const double *beta, const double *mu, double *alpha,
                     int par)
{
#pragma omp parallel for schedule(static) if (par)
    for (int i = 0; i < d1; ++i) {
        if (!(mu[i] > 0.0)) { alpha[i] = NEG_INF; continue; }
        double *x = (double *)malloc(sizeof(double) * (size_t)d2);
        for (int j = 0; j < d2; ++j)
            x[j] = beta[j] - C[(long)i * d2 + j] / lam;
        alpha[i] = log(mu[i]) - lse_strided(x, d2, 1);
        free(x);
    }
}

/* Entry of the plan, P_ij = exp(alpha_i + beta_j - C_ij / lambda)
 * (eq. (pij_form) written with u = exp(alpha), v = exp(beta)). */
static double plan_entry(double a, double b, double c, double lam)
{
    if (a == NEG_INF || b == NEG_INF) return 0.0;
    return exp(a + b - c / lam);
}

/* Marginal L1 error ||P 1 - mu||_1 + ||P^T 1 - nu||_1 and E^0 = sum P C,
 * straight from the definition of the coupling set U (Section 1). */
static void plan_stats(int d1, int d2, double lam, const double *C,
                       const double *alpha, const double *beta,
                       const double *mu, const double *nu,
                       double *err_out, double *loss_out, int par)
{
    double err_r = 0.0, loss = 0.0;
#pragma omp parallel for schedule(static) reduction(+ : err_r, loss) if (par)
    for (int i = 0; i < d1; ++i) {
        double r = 0.0, l = 0.0;
        for (int j = 0; j < d2; ++j) {
            double p = plan_entry(alpha[i], beta[j], C[(long)i * d2 + j], lam);
            r += p;
            l += p * C[(long)i * d2 + j];
        }
        err_r += fabs(r - mu[i]);
        loss += l;
    }
    double err_c = 0.0;
#pragma omp parallel for schedule(static) reduction(+ : err_c) if (par)
    for (int j = 0; j < d2; ++j) {
        double c = 0.0;
        for (int i = 0; i < d1; ++i)
            c += plan_entry(alpha[i], beta[j], C[(long)i * d2 + j], lam);
        err_c += fabs(c - nu[j]);
    }
    if (err_out) *err_out = err_r + err_c;
    if (loss_out) *loss_out = loss;
}

/* One sample.  Runs K <= n_iter iterations (early stop per the header).
 * err_hist (nullable, length n_iter) receives the marginal error of every
 * iterate that was evaluated (NaN for the others). */
static void sample_forward(int d1, int d2, double lam, int n_iter, double tol,
                           const double *mu, const double *nu, const double *C,
                           double *alpha, double *beta, double *loss,
                           double *marg_err, int *iters, double *err_hist,
                           int par, const double *alpha0)
{
    for (int i = 0; i < d1; ++i) alpha[i] = (mu[i] > 0.0) ? (alpha0 ? alpha0[i] : 0.0) : NEG_INF;
    for (int j = 0; j < d2; ++j) beta[j] = (nu[j] > 0.0) ? 0.0 : NEG_INF;
    if (err_hist)
        for (int k = 0; k < n_iter; ++k) err_hist[k] = NAN;

    int K = n_iter;
    for (int k = 1; k <= n_iter; ++k) {
        v_update(d1, d2, lam, C, alpha, nu, beta, par);
        u_update(d1, d2, lam, C, beta, mu, alpha, par);
        if (tol > 0.0 && k < n_iter) {
            double e;
            plan_stats(d1, d2, lam, C, alpha, beta, mu, nu, &e, NULL, par);
            if (err_hist) err_hist[k - 1] = e;
            if (e <= tol) { K = k; break; }
        }
    }
    double e, l;
    plan_stats(d1, d2, lam, C, alpha, beta, mu, nu, &e, &l, par);
    if (err_hist && K >= 1) err_hist[K - 1] = e;
    *loss = l;
    *marg_err = e;
    *iters = K;
}

/*
 * Batched forward.  All arrays are host, row-major, fp64.
 *   mu[B*d1], nu[B*d2], C[(c_batched ? B : 1) * d1 * d2]
 *   n_iter_b: nullable per-sample iteration counts (overrides n_iter).
 *   outputs alpha[B*d1], beta[B*d2], loss[B], marg_err[B], iters[B];
 *   err_hist: nullable [B*n_iter].
 *   alpha0: nullable [B*d1], the warm start's log u^0 (read on the support of
 *   mu only; it may be the alpha array itself).
 * Returns 0, or -1 on invalid arguments.
 */
int oracle_forward(int B, int d1, int d2, int c_batched, double lambda,
                   int n_iter, double tol, const int *n_iter_b,
                   const double *mu, const double *nu, const double *C,
                   double *alpha, double *beta, double *loss,
                   double *marg_err, int *iters, double *err_hist,
                   const double *alpha0)
{
    if (B < 0 || d1 < 1 || d2 < 1 || !(lambda > 0.0) || n_iter < 0) return -1;
    /* Parallelise across samples, or inside one sample's half-steps when
     * there are fewer samples than threads and the sample is large enough
     * for a parallel region to pay off. */
    int par_inner = B < n_threads() && (long)d1 * d2 >= 65536;
#pragma omp parallel for schedule(dynamic, 1) if (!par_inner)
    for (int b = 0; b < B; ++b) {
        const double *Cb = C + (c_batched ? (long)b * d1 * d2 : 0);
        int nb = n_iter_b ? n_iter_b[b] : n_iter;
        sample_forward(d1, d2, lambda, nb, n_iter_b ? 0.0 : tol,
                       mu + (long)b * d1, nu + (long)b * d2, Cb,
                       alpha + (long)b * d1, beta + (long)b * d2, loss + b,
                       marg_err + b, iters + b,
                       err_hist ? err_hist + (long)b * n_iter : NULL,
                       par_inner, alpha0 ? alpha0 + (long)b * d1 : NULL);
    }
    return 0;
}

/* Mean of x over the entries where w > 0 (the support). */
static double support_mean(const double *x, const double *w, int n)
{
    double s = 0.0;
    int m = 0;
    for (int k = 0; k < n; ++k)
        if (w[k] > 0.0) { s += x[k]; ++m; }
    return m ? s / m : 0.0;
}

/*
 * Batched backward (Section 2): with g = grad_loss[b],
 *   grad_mu_b = g * lambda * (alpha_b - mean_supp alpha_b), 0 off the support,
 *   grad_nu_b likewise with beta,
 *   grad_C (nullable): per-sample g * P_b, or sum_b g * P_b for shared C.
 */
int oracle_backward(int B, int d1, int d2, int c_batched, double lambda,
                    const double *grad_loss, const double *mu,
                    const double *nu, const double *C, const double *alpha,
                    const double *beta, double *grad_mu, double *grad_nu,
                    double *grad_C)
{
    if (B < 0 || d1 < 1 || d2 < 1 || !(lambda > 0.0)) return -1;
    for (int b = 0; b < B; ++b) {
        const double g = grad_loss[b];
        const double *a = alpha + (long)b * d1, *bt = beta + (long)b * d2;
        const double *m = mu + (long)b * d1, *n = nu + (long)b * d2;
        double ma = support_mean(a, m, d1), mb = support_mean(bt, n, d2);
        for (int i = 0; i < d1; ++i)
            grad_mu[(long)b * d1 + i] = (m[i] > 0.0) ? g * lambda * (a[i] - ma) : 0.0;
        for (int j = 0; j < d2; ++j)
            grad_nu[(long)b * d2 + j] = (n[j] > 0.0) ? g * lambda * (bt[j] - mb) : 0.0;
    }
    if (!grad_C) return 0;
    long cells = (long)d1 * d2;
    if (c_batched) {
#pragma omp parallel for schedule(static)
        for (int b = 0; b < B; ++b)
            for (int i = 0; i < d1; ++i)
                for (int j = 0; j < d2; ++j) {
                    long o = (long)b * cells + (long)i * d2 + j;
                    grad_C[o] = grad_loss[b] *
                        plan_entry(alpha[(long)b * d1 + i], beta[(long)b * d2 + j], C[o], lambda);
                }
    } else {
#pragma omp parallel for schedule(static)
        for (int i = 0; i < d1; ++i)
            for (int j = 0; j < d2; ++j) {
                double s = 0.0;
                for (int b = 0; b < B; ++b)
                    s += grad_loss[b] *
                        plan_entry(alpha[(long)b * d1 + i], beta[(long)b * d2 + j],
                                   C[(long)i * d2 + j], lambda);
                grad_C[(long)i * d2 + j] = s;
            }
    }
    return 0;
}

/*
 * Values used only by the pins: for one sample with potentials (alpha, beta)
 *   out[0] = dual value  lambda * (<alpha, mu> + <beta, nu>)   (support only)
 *   out[1] = primal E^lambda(P) = sum P C + lambda sum P log P (0 log 0 = 0)
 *   out[2] = E^0(P) = sum P C
 *   out[3] = h(P) = -sum P log P
 * At a fixed point of the iteration, out[0] == out[1] (no duality gap):
 * substituting eq. (pij_form) into the Lagrangian of Section 1.
 */
int oracle_objectives(int d1, int d2, double lambda, const double *mu,
                      const double *nu, const double *C, const double *alpha,
                      const double *beta, double *out)
{
    if (d1 < 1 || d2 < 1 || !(lambda > 0.0)) return -1;
    double dual = 0.0;
    for (int i = 0; i < d1; ++i) if (mu[i] > 0.0) dual += mu[i] * alpha[i];
    for (int j = 0; j < d2; ++j) if (nu[j] > 0.0) dual += nu[j] * beta[j];
    double e0 = 0.0, ent = 0.0;
    for (int i = 0; i < d1; ++i)
        for (int j = 0; j < d2; ++j) {
            double p = plan_entry(alpha[i], beta[j], C[(long)i * d2 + j], lambda);
            e0 += p * C[(long)i * d2 + j];
            if (p > 0.0) ent -= p * log(p);
        }
    out[0] = lambda * dual;
    out[1] = e0 - lambda * ent;
    out[2] = e0;
    out[3] = ent;
    return 0;
}

/* Plan of one sample, P[d1*d2] (for small pins only). */
int oracle_plan(int d1, int d2, double lambda, const double *C,
                const double *alpha, const double *beta, double *P)
{
    if (d1 < 1 || d2 < 1 || !(lambda > 0.0)) return -1;
    for (int i = 0; i < d1; ++i)
        for (int j = 0; j < d2; ++j)
            P[(long)i * d2 + j] = plan_entry(alpha[i], beta[j], C[(long)i * d2 + j], lambda);
    return 0;
}

int oracle_num_threads(void) { return n_threads(); }
