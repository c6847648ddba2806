/*
 * sinkhorn.h -- C ABI of the MI355X (gfx950) batched Sinkhorn library.
 *
 * Method: Viehmann, "Implementation of batched Sinkhorn iterations for
 * entropy-regularized Wasserstein loss" (arXiv:1907.01729).  For a batch of
 * histogram pairs (mu_b, nu_b) and a cost C (shared, or one per sample) the
 * library runs the Sinkhorn iteration in the log domain (Section 3, eq. (log_sk),
 * with the sign of the batched form in Section 4) or, where fp32 range allows,
 * the same iterates in the plain form (eq. (sk_plain)), returns the log-scalings, the
 * loss E^0 (Section 5) and the marginal error, and computes the
 * Lagrange-multiplier gradient (Section 2).
 *
 * Conventions shared by every entry point
 *   - Every array argument is a DEVICE pointer to contiguous row-major data
 *     (fp32 unless stated).  The caller owns every buffer; the library never
 *     allocates, frees or synchronises, and keeps no state between calls.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Work is enqueued asynchronously; results are valid once the stream has
 *     been synchronised.  Calls that overlap on one workspace race.
 *   - Errors are detected on the host before anything is launched (launch
 *     failures map to SK_ERR_HIP).  On error, output contents are unspecified.
 *     No C++ exception or abort crosses this interface.
 *   - Preconditions NOT checked (they would need a device synchronisation):
 *     mu, nu >= 0 with sum mu = sum nu = 1 (Section 1: probability measures),
 *     finite C.  Zero masses are allowed: their log-scalings are -inf
 *     (Section 3) and their gradients 0.  Non-finite inputs propagate.
 *
 * Notation.  alpha = log u, beta = log v (natural log, dimensionless), so the
 * plan is P_ij = exp(alpha_i + beta_j - C_ij / lambda)   (Section 1,
 * eq. (pij_form) with P = diag(u) K diag(v), K = exp(-C/lambda)).
 * The dual potentials in cost units are lambda*alpha and lambda*beta.
 */
#ifndef SINKHORN_H_
#define SINKHORN_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__) || defined(__clang__)
#define SK_API __attribute__((visibility("default")))
#else
#define SK_API
#endif

typedef enum {
    SK_OK = 0,
    SK_ERR_NULLPTR = -1,   /* a required pointer is NULL                     */
    SK_ERR_SHAPE = -2,     /* B < 0, d1 < 1, d2 < 1, d1 or d2 > 2^24, or
                              sizes overflow (d1 d2 > 2^40, B d1 d2 > 2^46) */
    SK_ERR_LAMBDA = -3,    /* lambda not finite and > 0                       */
    SK_ERR_ITERS = -4,     /* n_iter < 0, or tol not finite                   */
    SK_ERR_WORKSPACE = -5, /* ws_bytes < sinkhorn_workspace_bytes(p)          */
    SK_ERR_HIP = -6,       /* a HIP launch failed (e.g. device is not gfx950) */
    SK_ERR_ARG = -7        /* an argument outside its documented set of values
                              (the selector of sinkhorn_forward_select)       */
} sk_status;

typedef struct {
    int32_t B;          /* batch size, >= 0 (0: nothing to do)                      */
    int32_t d1, d2;     /* support sizes of mu and nu, >= 1                         */
    int32_t c_batched;  /* 0: C is [d1, d2], shared by the batch (Section 4);
                           1: C is [B, d1, d2], one cost per sample               */
    float lambda;       /* entropic regularisation, > 0, in cost units (Section 1) */
    int32_t n_iter;     /* number of full iterations (v-update, then u-update)      */
    float tol;          /* <= 0: always run n_iter (the paper's choice, Section 5);
                           > 0: per sample, stop after the first iteration
                           k < n_iter whose iterate has marginal L1 error <= tol   */
} sk_problem;

/*
 * Bytes of device workspace sinkhorn_forward needs for problem *p (0 when the
 * problem runs entirely on-chip).  Returns 0 for an invalid problem.
 */
SK_API size_t sinkhorn_workspace_bytes(const sk_problem *p);

/*
 * Forward: log-domain Sinkhorn (Section 3 and 4) followed by the loss
 * (Section 5).  Iteration k (1-based) performs
 *     beta_j  <- log nu_j - LSE_i(alpha_i - C_ij/lambda)     (v-update)
 *     alpha_i <- log mu_i - LSE_j(beta_j  - C_ij/lambda)     (u-update)
 * from alpha^0 = 0 on the support of mu (-inf off it).  With n_iter = 0,
 * alpha = beta = 0 on the supports.
 *
 * For max(d1, d2) <= 128 the same iterates are first computed in the plain
 * form of eq. (sk_plain), u = mu / (K v), v = nu / (K^T u), with K scaled by
 * its largest entry, on the vector ALU with K in registers (a shared C with
 * d1 = d2 <= 104 that proves symmetric: K^T u = K u; any other C, shared or
 * per sample: both products); a problem whose scaled cost spans more than
 * 64 bits, or whose sums or scalings leave a guarded fp32 range at any
 * iteration, is re-solved from the start in the log domain by the same
 * work-group.  Every problem is solved: iters >= 0.
 *
 *   mu        [B, d1]              input histograms
 *   nu        [B, d2]
 *   C         [d1, d2] or [B, d1, d2] (see c_batched)
 *   alpha     [B, d1]   out        log u of the returned iterate
 *   beta      [B, d2]   out        log v of the returned iterate
 *   loss      [B]       out        E^0 = sum_ij P_ij C_ij (Section 5)
 *   marg_err  [B]       out        ||P 1 - mu||_1 + ||P^T 1 - nu||_1
 *   iters     [B] int32 out        iterations run per sample (n_iter unless
 *                                  the early stop fired)
 *   workspace, ws_bytes            device scratch of at least
 *                                  sinkhorn_workspace_bytes(p) bytes (may be
 *                                  NULL when that is 0); contents on entry are
 *                                  irrelevant, on exit unspecified
 */
SK_API sk_status sinkhorn_forward(const sk_problem *p, const float *mu, const float *nu,
                           const float *C, float *alpha, float *beta, float *loss,
                           float *marg_err, int32_t *iters, void *workspace,
                           size_t ws_bytes, void *stream);

/*
 * Diagnostic variant of sinkhorn_forward for tests and measurements: the
 * same arguments, plus a selector that pins which kernels run.
 *   SK_SELECT_DEFAULT        exactly sinkhorn_forward;
 *   SK_SELECT_LOG_ONLY       resident shapes: the log-domain kernel alone
 *                            (no plain-form attempt);
 *   SK_SELECT_PLAIN_ONLY     resident shapes: the first-choice plain-form
 *                            kernel alone, without its log-domain fallback:
 *                            a problem it cannot keep in range comes back
 *                            with iters = -1 and its other outputs
 *                            unspecified;
 *   SK_SELECT_NO_SYMMETRIC   resident shapes: the general plain-form kernel
 *                            even where the symmetric-cost kernel applies;
 *   SK_SELECT_NO_COMPACTION  tiled shapes with a shared cost and tol > 0:
 *                            stopped problems keep their sweep slots (the
 *                            running batch is not compacted).
 * Selectors that do not apply to the problem's regime change nothing.  Any
 * other value: SK_ERR_ARG.  Results of the selectors other than
 * SK_SELECT_PLAIN_ONLY equal those of sinkhorn_forward up to rounding (the
 * same iterates); SK_SELECT_NO_COMPACTION gives identical bits.
 */
typedef enum {
    SK_SELECT_DEFAULT = 0,
    SK_SELECT_LOG_ONLY = 1,
    SK_SELECT_PLAIN_ONLY = 2,
    SK_SELECT_NO_SYMMETRIC = 3,
    SK_SELECT_NO_COMPACTION = 4
} sk_select;

SK_API sk_status sinkhorn_forward_select(const sk_problem *p, int32_t select, const float *mu,
                                         const float *nu, const float *C, float *alpha, float *beta,
                                         float *loss, float *marg_err, int32_t *iters, void *workspace,
                                         size_t ws_bytes, void *stream);

/*
 * Warm start (checkpoint and resume; not in the paper): sinkhorn_forward
 * started from the caller's row log-scalings alpha0 [B, d1] (natural log,
 * as sinkhorn_forward returns them in alpha) on the support of mu instead of
 * alpha = 0 there; entries off the support are ignored (-inf).  Every
 * iteration begins with the v-update from alpha, so alpha is the iteration's
 * whole state: continuing a K-iteration forward from its alpha for n more
 * iterations gives the iterates of a (K + n)-iteration forward, up to
 * rounding.  alpha0 may be the alpha output buffer itself (read before it is
 * written).  Runs the log-domain kernels (the plain form starts from u = 1).
 * Arguments, workspace and errors as sinkhorn_forward; alpha0 NULL:
 * SK_ERR_NULLPTR.
 */
SK_API sk_status sinkhorn_forward_warm(const sk_problem *p, const float *alpha0, const float *mu,
                                       const float *nu, const float *C, float *alpha, float *beta, float *loss,
                                       float *marg_err, int32_t *iters, void *workspace, size_t ws_bytes,
                                       void *stream);

/*
 * Dispatch report, for logging and debugging (nothing is launched): writes
 * into buf a one-line, NUL-terminated description of the kernels and launch
 * shape that sinkhorn_forward_select(p, select, ...) takes for *p: the
 * regime, the kernel instantiations, row blocks, merges, hand-overs and the
 * workspace size.  snprintf semantics: at most len bytes are written (buf may
 * be NULL when len is 0) and the return value is the length of the whole
 * line without the NUL.  Invalid problem: its (negative) status; unknown
 * selector: SK_ERR_ARG.  The symmetry of a shared cost is only tested on the
 * device, so the report names the symmetric kernel with its in-place general
 * iteration.
 */
SK_API int32_t sinkhorn_describe(const sk_problem *p, int32_t select, char *buf, size_t len);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the forward
 * of sinkhorn_forward without a workspace argument.  Its scratch is a fixed
 * device array of SINKHORN_NOALLOC_SCRATCH_BYTES inside the library, one per
 * GPU, allocated when the library's code object is loaded and held until the
 * process ends; the call itself allocates and frees nothing.  The caller
 * still owns every input and output.  It runs on the current device (the
 * stream must belong to it).
 *   - Problems whose sinkhorn_workspace_bytes(p) exceeds the array are
 *     rejected with SK_ERR_WORKSPACE before anything is launched (problems
 *     that need no workspace always fit).
 *   - Every call on one GPU shares that GPU's array, which keeps the last
 *     call's contents (the kernels initialise what they read).  Calls that
 *     overlap on one GPU, on any streams or threads, race and give
 *     unspecified results: serialise them.
 *   - The first call on a device looks up the array's device address
 *     (SK_ERR_HIP if that fails).
 * Results are those of sinkhorn_forward on the same inputs.
 */
#define SINKHORN_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

SK_API sk_status sinkhorn_forward_noalloc(const sk_problem *p, const float *mu, const float *nu,
                                          const float *C, float *alpha, float *beta, float *loss,
                                          float *marg_err, int32_t *iters, void *stream);

/*
 * Backward (Section 2): the Lagrange-multiplier gradient of the entropic
 * objective W_lambda(mu, nu) = min_U E^lambda, taken at the iterate the
 * forward returned (Section 5 explains why this is used for the E^0 loss).
 * With g = grad_loss[b]:
 *   grad_mu[b,i] = g * lambda * (alpha[b,i] - mean over the support of mu_b of
 *                  alpha[b,.]),  0 where mu[b,i] == 0;
 *   grad_nu      likewise with beta and nu;
 *   grad_C (optional, may be NULL): d W_lambda / d C = P, i.e.
 *                  g * P_b           for c_batched (shape [B, d1, d2]),
 *                  sum_b g_b * P_b   for a shared C (shape [d1, d2]).
 * alpha and beta are the forward's outputs; n_iter and tol are ignored.
 * Needs no workspace.  Deterministic (fixed reduction order, no atomics).
 */
SK_API sk_status sinkhorn_backward(const sk_problem *p, const float *grad_loss,
                            const float *mu, const float *nu, const float *C,
                            const float *alpha, const float *beta,
                            float *grad_mu, float *grad_nu, float *grad_C,
                            void *stream);

/*
 * Gradient of the sharp loss E^0 = sum_ij P_ij C_ij itself with respect to
 * (mu, nu) (Section 5 points to this sharper gradient; sinkhorn_backward
 * returns the multiplier gradient of E^lambda).  The plan P of (alpha, beta)
 * is differentiated through its marginal constraints: with r = P 1,
 * c = P^T 1, a = (P o C) 1, b = (P o C)^T 1 the gradient is the solution z of
 *     [diag(r)  P      ] z = (a, b),
 *     [P^T      diag(c)]
 * each block centred over the support of mu (resp. nu) and 0 off it, times
 * grad_loss[b].  The matrix is singular along (1, -1); the right-hand side is
 * projected off that direction.  Solved per problem by conjugate gradients
 * preconditioned with (r, c): at most max_cg (>= 1) iterations, stopping when
 * the preconditioned residual norm falls below cg_tol (>= 0) times its start
 * value.  cg_iters [B] int32 (may be NULL) receives the iterations taken.
 * For max(d1, d2) <= 128 the plan of a problem sits in the registers of one
 * work-group and no workspace is needed (workspace may be NULL); larger
 * supports (the shapes sinkhorn_forward takes in its tiled regime) rebuild the
 * plan from (alpha, beta, C) in a sweep over the cost for every product and
 * keep the iteration's vectors in a workspace of at least
 * sinkhorn_sharp_workspace_bytes(p) bytes (SK_ERR_WORKSPACE if smaller); every
 * problem then runs max_cg launches of which those after its convergence do
 * nothing.  Deterministic.  Invalid max_cg or cg_tol: SK_ERR_ITERS.
 */
SK_API sk_status sinkhorn_backward_sharp(const sk_problem *p, const float *grad_loss,
                                  const float *mu, const float *nu, const float *C,
                                  const float *alpha, const float *beta, float *grad_mu,
                                  float *grad_nu, int32_t max_cg, float cg_tol,
                                  int32_t *cg_iters, void *workspace, size_t ws_bytes,
                                  void *stream);

/* Bytes of workspace sinkhorn_backward_sharp needs for *p (0 when the
 * problem needs none, and for an invalid problem). */
SK_API size_t sinkhorn_sharp_workspace_bytes(const sk_problem *p);

/*
 * Point clouds.  The cost is the squared Euclidean distance between points,
 *     C_ij = sum_k (X[i,k] - Y[j,k])^2,   k < D,   1 <= D <= 16,
 * with X [d1, D] and Y [d2, D] shared by the batch (c_batched = 0) or
 * X [B, d1, D] and Y [B, d2, D] per sample (c_batched = 1).  Everything else
 * is as in sinkhorn_forward / sinkhorn_backward with that C.  Section 4 notes
 * that cost entries can be recreated from the points rather than stored: for
 * per-sample clouds with max(d1, d2) > 128, d2 <= 2048 and D <= 3 the tiled
 * sweep does exactly that and no cost matrix exists (the cost is
 * -|r x_i - r y_j|^2 in the scaled base-2 units, r = sqrt(log2(e)/lambda),
 * evaluated in fp32); every other shape writes C into the workspace first and
 * runs the forward above on it.
 *
 * Bytes of workspace sinkhorn_forward_points needs (0 for an invalid problem
 * or D).
 */
SK_API size_t sinkhorn_points_workspace_bytes(const sk_problem *p, int32_t D);

SK_API sk_status sinkhorn_forward_points(const sk_problem *p, int32_t D, const float *mu,
                                  const float *nu, const float *X, const float *Y,
                                  float *alpha, float *beta, float *loss, float *marg_err,
                                  int32_t *iters, void *workspace, size_t ws_bytes,
                                  void *stream);

/*
 * Backward for point clouds: grad_mu and grad_nu as in sinkhorn_backward, and
 * (optional, either may be NULL) the gradient with respect to the points by
 * the chain rule through dW/dC = P:
 *   grad_X[b,i,:] = g_b * sum_j P_b,ij * 2 (X[b,i,:] - Y[b,j,:]),
 *   grad_Y[b,j,:] = g_b * sum_i P_b,ij * 2 (Y[b,j,:] - X[b,i,:]),
 * summed over the batch for shared clouds (shapes as X and Y).  P is rebuilt
 * from alpha, beta and the points; needs no workspace; deterministic.
 */
SK_API sk_status sinkhorn_backward_points(const sk_problem *p, int32_t D, const float *grad_loss,
                                   const float *mu, const float *nu, const float *X,
                                   const float *Y, const float *alpha, const float *beta,
                                   float *grad_mu, float *grad_nu, float *grad_X,
                                   float *grad_Y, void *stream);

/* Static description of a status code (never NULL). */
SK_API const char *sinkhorn_status_string(sk_status s);

/*
 * Which kernel family sinkhorn_forward uses for *p:
 *   1 = resident (max(d1, d2) <= 128: C and potentials on-chip for the whole
 *       iteration; plain form with the log-domain fallback described above),
 *   2 = tiled sweep (one pass over C per iteration, column partials merged
 *       across row blocks).
 * Returns 0 for an invalid problem.
 */
SK_API int32_t sinkhorn_regime(const sk_problem *p);

#ifdef __cplusplus
}
#endif

#endif /* SINKHORN_H_ */
