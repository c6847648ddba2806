/*
 * Host sanitizer run of the oracle (test infrastructure): built with
 * AddressSanitizer and UndefinedBehaviorSanitizer together with
 * oracle/sinkhorn_oracle.c and run on the CPU by tests/test_sanitize_host.py.
 *
 * Small problems go through every entry point of the oracle: zero masses,
 * ragged shapes, one row or one column, shared and per-sample costs, an
 * early stop, n_iter = 0, per-sample iteration counts and an empty batch.
 * The sanitizers abort on their own findings; besides, every case checks
 * properties the method fixes exactly, so a wrong index also shows here:
 *   - after a u-update the plan's row sums are mu (Section 3: the u-update
 *     makes the row marginal exact);
 *   - each gradient of mu (nu) sums to 0 over its support and is 0 off it
 *     (Section 2, the mean-centred multiplier);
 *   - a shared cost's grad_C sums to sum_b g_b (each plan has mass 1);
 *   - the loss equals sum_ij P_ij C_ij of the returned plan.
 * Exits 0 and prints "ok" when every check passes.
 */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_forward(int B, int d1, int d2, int c_batched, double lambda, int n_iter, double tol,
                   const int *n_iter_b, const double *mu, const double *nu, const double *C, double *alpha,
                   double *beta, double *loss, double *marg_err, int *iters, double *err_hist,
                   const double *alpha0);
int oracle_backward(int B, int d1, int d2, int c_batched, double lambda, const double *grad_loss,
                    const double *mu, const double *nu, const double *C, const double *alpha, const double *beta,
                    double *grad_mu, double *grad_nu, double *grad_C);
int oracle_objectives(int d1, int d2, double lambda, const double *mu, const double *nu, const double *C,
                      const double *alpha, const double *beta, double *out);
int oracle_plan(int d1, int d2, double lambda, const double *C, const double *alpha, const double *beta,
                double *P);

static unsigned long long state = 0x9E3779B97F4A7C15ull;

static double urand(void) /* xorshift64*, uniform in [0, 1) */
{
    state ^= state >> 12;
    state ^= state << 25;
    state ^= state >> 27;
    return (double)((state * 0x2545F4914F6CDD1Dull) >> 11) * (1.0 / 9007199254740992.0);
}

static void histograms(double *h, int B, int n, double zero_frac)
{
    for (int b = 0; b < B; ++b) {
        double s = 0.0;
        for (int i = 0; i < n; ++i) {
            double v = 0.05 + 0.95 * urand();
            if (i > 0 && urand() < zero_frac) v = 0.0;
            h[(long)b * n + i] = v;
            s += v;
        }
        for (int i = 0; i < n; ++i) h[(long)b * n + i] /= s;
    }
}

static int failures = 0;

static void check(int ok, const char *what, int line)
{
    if (!ok) {
        fprintf(stderr, "check failed (line %d): %s\n", line, what);
        ++failures;
    }
}
#define CHECK(x) check((x), #x, __LINE__)

static void run_case(int B, int d1, int d2, int cb, double lam, int n_iter, double tol, double zero_frac)
{
    const long nC = (long)(cb ? B : 1) * d1 * d2;
    double *mu = malloc(sizeof(double) * ((long)B * d1 + 1));
    double *nu = malloc(sizeof(double) * ((long)B * d2 + 1));
    double *C = malloc(sizeof(double) * (nC + 1));
    double *alpha = malloc(sizeof(double) * ((long)B * d1 + 1));
    double *beta = malloc(sizeof(double) * ((long)B * d2 + 1));
    double *loss = malloc(sizeof(double) * (B + 1));
    double *merr = malloc(sizeof(double) * (B + 1));
    int *iters = malloc(sizeof(int) * (B + 1));
    double *hist = malloc(sizeof(double) * ((long)B * (n_iter > 0 ? n_iter : 1) + 1));
    double *g = malloc(sizeof(double) * (B + 1));
    double *gmu = malloc(sizeof(double) * ((long)B * d1 + 1));
    double *gnu = malloc(sizeof(double) * ((long)B * d2 + 1));
    double *gC = malloc(sizeof(double) * (nC + 1));
    double *P = malloc(sizeof(double) * ((long)d1 * d2));
    histograms(mu, B, d1, zero_frac);
    histograms(nu, B, d2, zero_frac);
    for (long u = 0; u < nC; ++u) C[u] = urand();
    for (int b = 0; b < B; ++b) g[b] = 0.5 + urand();

    CHECK(oracle_forward(B, d1, d2, cb, lam, n_iter, tol, NULL, mu, nu, C, alpha, beta, loss, merr, iters,
                         n_iter > 0 ? hist : NULL, NULL) == 0);
    for (int b = 0; b < B; ++b) {
        const double *Cb = C + (cb ? (long)b * d1 * d2 : 0);
        const double *a = alpha + (long)b * d1, *bt = beta + (long)b * d2;
        CHECK(iters[b] >= 0 && iters[b] <= n_iter);
        CHECK(oracle_plan(d1, d2, lam, Cb, a, bt, P) == 0);
        double e0 = 0.0;
        for (int i = 0; i < d1; ++i) {
            double r = 0.0;
            for (int j = 0; j < d2; ++j) {
                r += P[(long)i * d2 + j];
                e0 += P[(long)i * d2 + j] * Cb[(long)i * d2 + j];
            }
            if (iters[b] > 0) CHECK(fabs(r - mu[(long)b * d1 + i]) <= 1e-12);
        }
        CHECK(fabs(e0 - loss[b]) <= 1e-12 * (1.0 + fabs(e0)));
        CHECK(isfinite(merr[b]) && merr[b] >= 0.0);
        double obj[4];
        CHECK(oracle_objectives(d1, d2, lam, mu + (long)b * d1, nu + (long)b * d2, Cb, a, bt, obj) == 0);
        CHECK(isfinite(obj[0]) && isfinite(obj[1]) && fabs(obj[2] - loss[b]) <= 1e-12 * (1.0 + fabs(e0)));
    }

    CHECK(oracle_backward(B, d1, d2, cb, lam, g, mu, nu, C, alpha, beta, gmu, gnu, gC) == 0);
    double gsum = 0.0, gCsum = 0.0;
    for (int b = 0; b < B; ++b) {
        double s1 = 0.0, s2 = 0.0;
        for (int i = 0; i < d1; ++i) {
            const double v = gmu[(long)b * d1 + i];
            if (mu[(long)b * d1 + i] > 0.0) s1 += v;
            else CHECK(v == 0.0);
        }
        for (int j = 0; j < d2; ++j) {
            const double v = gnu[(long)b * d2 + j];
            if (nu[(long)b * d2 + j] > 0.0) s2 += v;
            else CHECK(v == 0.0);
        }
        CHECK(fabs(s1) <= 1e-9 && fabs(s2) <= 1e-9);
        if (iters[b] > 0) gsum += g[b];
    }
    if (!cb && n_iter > 0) {
        for (long u = 0; u < nC; ++u) gCsum += gC[u];
        CHECK(fabs(gCsum - gsum) <= 1e-9 * (1.0 + gsum));
    }

    /* per-sample iteration counts: the same counts give the same iterates */
    if (n_iter > 0 && B > 0) {
        double *alpha2 = malloc(sizeof(double) * (long)B * d1), *beta2 = malloc(sizeof(double) * (long)B * d2);
        int *iters2 = malloc(sizeof(int) * B);
        CHECK(oracle_forward(B, d1, d2, cb, lam, n_iter, 0.0, iters, mu, nu, C, alpha2, beta2, loss, merr, iters2,
                             NULL, NULL) == 0);
        for (int b = 0; b < B; ++b) {
            CHECK(iters2[b] == iters[b]);
            for (int i = 0; i < d1; ++i)
                CHECK(alpha2[(long)b * d1 + i] == alpha[(long)b * d1 + i] ||
                      (isinf(alpha2[(long)b * d1 + i]) && isinf(alpha[(long)b * d1 + i])));
        }
        /* warm start, in place: 3 more iterations from the returned alpha
           equal a run of iters + 3 (the state is alpha alone) */
        int *more = malloc(sizeof(int) * B), *iters3 = malloc(sizeof(int) * B);
        double *alpha3 = malloc(sizeof(double) * (long)B * d1);
        for (int b = 0; b < B; ++b) more[b] = iters[b] + 3;
        CHECK(oracle_forward(B, d1, d2, cb, lam, n_iter + 3, 0.0, more, mu, nu, C, alpha3, beta2, loss, merr,
                             iters3, NULL, NULL) == 0);
        for (int b = 0; b < B; ++b) more[b] = 3;
        CHECK(oracle_forward(B, d1, d2, cb, lam, 3, 0.0, more, mu, nu, C, alpha2, beta2, loss, merr, iters2, NULL,
                             alpha2) == 0);
        for (long u = 0; u < (long)B * d1; ++u)
            CHECK(alpha2[u] == alpha3[u] || (isinf(alpha2[u]) && isinf(alpha3[u])));
        free(more);
        free(iters3);
        free(alpha3);
        free(alpha2);
        free(beta2);
        free(iters2);
    }
    free(mu); free(nu); free(C); free(alpha); free(beta); free(loss); free(merr); free(iters); free(hist);
    free(g); free(gmu); free(gnu); free(gC); free(P);
}

int main(void)
{
    run_case(3, 7, 5, 0, 0.2, 30, 0.0, 0.3);     /* shared cost, zero masses */
    run_case(2, 1, 9, 1, 0.05, 50, 1e-4, 0.2);   /* one row, per-sample cost, early stop */
    run_case(2, 9, 1, 0, 0.1, 20, 0.0, 0.0);     /* one column */
    run_case(4, 16, 16, 0, 0.5, 0, 0.0, 0.0);    /* n_iter = 0 */
    run_case(1, 33, 2, 1, 1.0, 10, 1e-3, 0.0);   /* ragged, early stop */
    run_case(2, 12, 40, 1, 0.01, 60, 0.0, 0.1);  /* small lambda, per-sample cost */
    run_case(0, 5, 5, 0, 0.1, 10, 0.0, 0.0);     /* empty batch */
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("ok\n");
    return 0;
}
