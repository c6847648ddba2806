/*
 * Host sanitizer run of the library's C ABI (test infrastructure): built
 * against a copy of libsinkhorn_hip.so whose host code carries
 * AddressSanitizer and UndefinedBehaviorSanitizer (device code unchanged),
 * run on the CPU by tests/test_sanitize_host.py.
 *
 * Only host-side paths are taken, and nothing is launched: every call either
 * is rejected on the host (invalid problem, NULL pointer, short workspace
 * with placeholder pointers that are never dereferenced, unknown selector)
 * or is a query (workspace sizes, regime, status strings, the dispatch
 * report), over ordinary, extreme and overflowing shapes.  Exits 0 and
 * prints "ok" when every status is the documented one.
 */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "sinkhorn.h"

static int failures = 0;

static void check(int ok, const char *what, int line)
{
    if (!ok) {
        fprintf(stderr, "check failed (line %d): %s\n", line, what);
        ++failures;
    }
}
#define CHECK(x) check((x), #x, __LINE__)

static sk_problem prob(int B, int d1, int d2, int cb, float lam, int n_iter, float tol)
{
    sk_problem p;
    p.B = B;
    p.d1 = d1;
    p.d2 = d2;
    p.c_batched = cb;
    p.lambda = lam;
    p.n_iter = n_iter;
    p.tol = tol;
    return p;
}

int main(void)
{
    /* a placeholder address: only ever passed where the call must stop at the
       workspace-size check, before anything is launched or dereferenced */
    float *fake = (float *)(uintptr_t)0x1000;
    int32_t *ifake = (int32_t *)(uintptr_t)0x1000;
    char line[512];

    /* status strings, including unknown codes */
    for (int s = -8; s <= 1; ++s) CHECK(sinkhorn_status_string((sk_status)s) != NULL);

    /* NULL problem */
    CHECK(sinkhorn_workspace_bytes(NULL) == 0);
    CHECK(sinkhorn_regime(NULL) == 0);
    CHECK(sinkhorn_forward(NULL, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, NULL) == SK_ERR_NULLPTR);
    CHECK(sinkhorn_describe(NULL, 0, line, sizeof line) == SK_ERR_NULLPTR);

    /* invalid problems, every entry point */
    const sk_problem bad[] = {
        prob(-1, 10, 10, 0, 0.1f, 10, 0.f), prob(4, 0, 10, 0, 0.1f, 10, 0.f), prob(4, 10, 0, 0, 0.1f, 10, 0.f),
        prob(4, 10, 10, 2, 0.1f, 10, 0.f), prob(4, 10, 10, 0, 0.f, 10, 0.f), prob(4, 10, 10, 0, -1.f, 10, 0.f),
        prob(4, 10, 10, 0, 0.1f, -1, 0.f), prob(4, 10, 10, 0, 0.1f, 10, 1.f / 0.f),
        prob(4, (1 << 24) + 1, 10, 0, 0.1f, 10, 0.f), prob(1 << 30, 1 << 20, 1 << 20, 1, 0.1f, 10, 0.f),
        prob(2, 1 << 22, 1 << 22, 0, 0.1f, 10, 0.f),
    };
    for (size_t k = 0; k < sizeof bad / sizeof bad[0]; ++k) {
        const sk_problem *p = &bad[k];
        CHECK(sinkhorn_workspace_bytes(p) == 0);
        CHECK(sinkhorn_sharp_workspace_bytes(p) == 0);
        CHECK(sinkhorn_points_workspace_bytes(p, 3) == 0);
        CHECK(sinkhorn_regime(p) == 0);
        CHECK(sinkhorn_forward(p, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, NULL) < 0);
        CHECK(sinkhorn_forward_noalloc(p, 0, 0, 0, 0, 0, 0, 0, 0, NULL) < 0);
        CHECK(sinkhorn_describe(p, 0, line, sizeof line) < 0);
    }

    /* valid shapes of every regime: queries, the report, rejections before launch */
    const sk_problem good[] = {
        prob(4, 10, 10, 0, 0.1f, 100, 0.f),      prob(1024, 100, 100, 0, 0.05f, 200, 0.f),
        prob(8, 120, 120, 1, 0.1f, 10, 0.f),     prob(256, 784, 784, 0, 0.01f, 300, 0.f),
        prob(64, 4096, 4096, 0, 1e-3f, 500, 1e-6f), prob(32, 1024, 2048, 1, 0.05f, 100, 0.f),
        prob(4, 200, 5000, 0, 0.1f, 10, 0.f),    prob(70000, 130, 8, 1, 0.1f, 10, 1e-4f),
        prob(3, 1, 100000, 1, 0.1f, 5, 0.f),     prob(1 << 20, 8, 8, 0, 0.1f, 10, 0.f),
    };
    for (size_t k = 0; k < sizeof good / sizeof good[0]; ++k) {
        const sk_problem *p = &good[k];
        const int regime = sinkhorn_regime(p);
        CHECK(regime == 1 || regime == 2);
        const size_t ws = sinkhorn_workspace_bytes(p);
        CHECK((regime == 1) == (ws == 0));
        (void)sinkhorn_sharp_workspace_bytes(p);
        (void)sinkhorn_points_workspace_bytes(p, 3);
        for (int sel = 0; sel <= 4; ++sel) {
            const int32_t n = sinkhorn_describe(p, sel, NULL, 0);
            CHECK(n > 0 && n < (int32_t)sizeof line);
            CHECK(sinkhorn_describe(p, sel, line, sizeof line) == n && (int32_t)strlen(line) == n);
            char small[8];
            memset(small, 'x', sizeof small);
            CHECK(sinkhorn_describe(p, sel, small, 5) == n && small[4] == 0 && small[5] == 'x');
        }
        CHECK(sinkhorn_describe(p, 7, line, sizeof line) == SK_ERR_ARG);
        CHECK(sinkhorn_forward_select(p, 9, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, NULL) == SK_ERR_ARG);
        /* NULL arrays */
        CHECK(sinkhorn_forward(p, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, NULL) == SK_ERR_NULLPTR);
        CHECK(sinkhorn_forward_warm(p, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, NULL) == SK_ERR_NULLPTR);
        CHECK(sinkhorn_backward(p, 0, 0, 0, 0, 0, 0, 0, 0, 0, NULL) == SK_ERR_NULLPTR);
        CHECK(sinkhorn_forward_points(p, 3, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, NULL) == SK_ERR_NULLPTR);
        /* a workspace one byte short, placeholder pointers: rejected before launch */
        if (ws > 0) {
            CHECK(sinkhorn_forward(p, fake, fake, fake, fake, fake, fake, fake, ifake, fake, ws - 1, NULL) ==
                  SK_ERR_WORKSPACE);
            CHECK(sinkhorn_forward_warm(p, fake, fake, fake, fake, fake, fake, fake, fake, ifake, fake, ws - 1,
                                        NULL) == SK_ERR_WORKSPACE);
        }
        const size_t sws = sinkhorn_sharp_workspace_bytes(p);
        if (sws > 0)
            CHECK(sinkhorn_backward_sharp(p, fake, fake, fake, fake, fake, fake, fake, fake, 10, 1e-6f, ifake,
                                          fake, sws - 1, NULL) == SK_ERR_WORKSPACE);
        const size_t pws = sinkhorn_points_workspace_bytes(p, 3);
        if (pws > 0)
            CHECK(sinkhorn_forward_points(p, 3, fake, fake, fake, fake, fake, fake, fake, fake, ifake, fake,
                                          pws - 1, NULL) == SK_ERR_WORKSPACE);
        /* points: coordinates per point outside 1..16 */
        CHECK(sinkhorn_points_workspace_bytes(p, 0) == 0 && sinkhorn_points_workspace_bytes(p, 17) == 0);
        /* sharp: iteration cap and tolerance */
        CHECK(sinkhorn_backward_sharp(p, 0, 0, 0, 0, 0, 0, 0, 0, 0, 1e-6f, 0, 0, 0, NULL) == SK_ERR_ITERS);
        CHECK(sinkhorn_backward_sharp(p, 0, 0, 0, 0, 0, 0, 0, 0, 5, -1.f, 0, 0, 0, NULL) == SK_ERR_ITERS);
    }

    /* an empty batch succeeds without touching any pointer */
    const sk_problem empty = prob(0, 10, 10, 0, 0.1f, 10, 0.f);
    CHECK(sinkhorn_forward(&empty, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, NULL) == SK_OK);
    CHECK(sinkhorn_forward_warm(&empty, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, NULL) == SK_OK);
    CHECK(sinkhorn_backward(&empty, 0, 0, 0, 0, 0, 0, 0, 0, 0, NULL) == SK_OK);
    CHECK(sinkhorn_forward_noalloc(&empty, 0, 0, 0, 0, 0, 0, 0, 0, NULL) == SK_OK);

    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("ok\n");
    return 0;
}
