// sk_api.hip -- the C ABI declared in include/sinkhorn.h: argument checks,
// regime dispatch and launches.  No allocation, no synchronisation.
#include <math.h>
#include <stdint.h>
#include <stdio.h>

#include <mutex>

#include "sk_internal.h"

namespace {

constexpr int64_t kMaxDim = 1 << 24;

sk_status check_problem(const sk_problem *p) {
    if (!p) return SK_ERR_NULLPTR;
    if (p->B < 0 || p->d1 < 1 || p->d2 < 1 || p->d1 > kMaxDim || p->d2 > kMaxDim) return SK_ERR_SHAPE;
    if (p->c_batched != 0 && p->c_batched != 1) return SK_ERR_SHAPE;
    const int64_t cells = (int64_t)p->d1 * p->d2;  // <= 2^48: d1, d2 <= 2^24
    // B d1 d2 <= 2^46, tested without forming the product (it can overflow)
    if (cells > (int64_t(1) << 40) || (int64_t)p->B > (int64_t(1) << 46) / cells) return SK_ERR_SHAPE;
    if (!sk::resident_fits(p->d1, p->d2) && !sk::tiled_fits(p->B, p->d1, p->d2, p->c_batched)) return SK_ERR_SHAPE;
    if (!(p->lambda > 0.f) || !isfinite(p->lambda)) return SK_ERR_LAMBDA;
    if (p->n_iter < 0 || !isfinite(p->tol)) return SK_ERR_ITERS;
    return SK_OK;
}

sk::BwdArgs bwd_args(const sk_problem *p, const float *grad_loss, const float *mu, const float *nu, const float *C,
                     const float *alpha, const float *beta, float *grad_mu, float *grad_nu, float *grad_C) {
    sk::BwdArgs a;
    a.grad_loss = grad_loss;
    a.mu = mu;
    a.nu = nu;
    a.C = C;
    a.alpha = alpha;
    a.beta = beta;
    a.grad_mu = grad_mu;
    a.grad_nu = grad_nu;
    a.grad_C = grad_C;
    a.B = p->B;
    a.d1 = p->d1;
    a.d2 = p->d2;
    a.c_batched = p->c_batched;
    a.lambda = p->lambda;
    a.s = sk::kLog2eHost / p->lambda;
    return a;
}

// Resident regime.  First choice: the symmetric-cost kernel (shared cost,
// d1 = d2 <= 104; it runs the general iteration in place when the cost is
// not symmetric), else the general plain-form kernel (any cost).  Either
// solves the problems it cannot keep in range in the log domain, in place.
// The selector of sinkhorn_forward_select can pin one of these kernels.
hipError_t launch_resident_regime(const sk::FwdArgs &a, hipStream_t s) {
    if (a.select == SK_SELECT_LOG_ONLY) return sk::launch_resident(a, s);
    hipError_t e = hipSuccess;
    const bool ran = (a.select != SK_SELECT_NO_SYMMETRIC && sk::launch_resident_sym(a, s, &e)) ||
                     sk::launch_resident_gen(a, s, &e);
    if (!ran) return sk::launch_resident(a, s);
    // The widest bucket marks what it hands over; solve those problems next.
    if (e == hipSuccess && a.select != SK_SELECT_PLAIN_ONLY && (a.d1 > 104 || a.d2 > 104)) {
        sk::FwdArgs m = a;
        m.only_marked = 1;
        e = sk::launch_resident(m, s);
    }
    return e;
}

sk::FwdArgs fwd_args(const sk_problem *p, const float *mu, const float *nu, const float *C, float *alpha,
                     float *beta, float *loss, float *marg_err, int32_t *iters) {
    sk::FwdArgs a;
    a.mu = mu;
    a.nu = nu;
    a.C = C;
    a.alpha = alpha;
    a.beta = beta;
    a.loss = loss;
    a.marg_err = marg_err;
    a.iters = iters;
    a.B = p->B;
    a.d1 = p->d1;
    a.d2 = p->d2;
    a.n_iter = p->n_iter;
    a.c_batched = p->c_batched;
    a.lambda = p->lambda;
    a.tol = p->tol;
    a.s = sk::kLog2eHost / p->lambda;
    a.select = SK_SELECT_DEFAULT;
    a.only_marked = 0;
    a.alpha0 = nullptr;
    return a;
}

// The resident regime's choice (launch_resident_regime) in one line.
int resident_describe(const sk::FwdArgs &a, char *buf, size_t len) {
    const int nb = ((a.d1 > a.d2 ? a.d1 : a.d2) + 7) / 8;
    const int N = nb <= 2 ? 2 : nb <= 4 ? 4 : nb <= 8 ? 8 : nb <= 13 ? 13 : 16;
    if (a.select == SK_SELECT_LOG_ONLY || a.n_iter <= 0)
        return snprintf(buf, len,
                        "resident: sk_resident_log_kernel<%d> (log domain, two wavefronts per problem, the scaled "
                        "cost in registers, every iteration in one launch)",
                        N);
    const bool sym = a.select != SK_SELECT_NO_SYMMETRIC && !a.c_batched && a.d1 == a.d2 && N <= 13;
    const char *hand = a.select == SK_SELECT_PLAIN_ONLY
                           ? "a problem out of fp32 range is left unsolved (iters = -1)"
                           : (N <= 13 ? "a problem out of fp32 range is re-solved in the log domain in place"
                                      : "a problem out of fp32 range is re-solved by a second launch, "
                                        "sk_resident_log_kernel<16>");
    return snprintf(buf, len,
                    "resident: %s<%d> (plain form, K in registers, two wavefronts per problem%s); %s",
                    sym ? "sk_resident_sym_kernel" : "sk_resident_gen_kernel", N,
                    sym ? "; the general iteration in place if the cost is not symmetric" : "", hand);
}

// Regime dispatch of a forward over a cost matrix (tiled sweep, or the
// resident kernels with their hand-overs).
hipError_t run_forward(const sk::FwdArgs &a, void *workspace, hipStream_t s) {
    if (!sk::resident_fits(a.d1, a.d2)) return sk::launch_tiled(a, workspace, s);
    return launch_resident_regime(a, s);
}

// ---- point clouds ----

constexpr int64_t kMaxPointFloats = int64_t(1) << 40;

sk_status check_points(const sk_problem *p, int32_t D) {
    const sk_status st = check_problem(p);
    if (st != SK_OK) return st;
    if (D < 1 || D > sk::kPointsGradD) return SK_ERR_SHAPE;
    const int64_t nb = p->c_batched ? p->B : 1;
    if (nb * (int64_t)(p->d1 + (int64_t)p->d2) * D > kMaxPointFloats) return SK_ERR_SHAPE;
    return SK_OK;
}

// Per-sample clouds of the tiled regime go through the on-the-fly sweep when
// it takes the shape; everything else writes the cost out first.
bool points_on_the_fly(const sk_problem *p, int32_t D) {
    return p->c_batched && !sk::resident_fits(p->d1, p->d2) && sk::tiled_points_fits(p->B, p->d1, p->d2, D);
}

size_t cost_bytes(const sk_problem *p) {
    const size_t n = sizeof(float) * (size_t)(p->c_batched ? p->B : 1) * p->d1 * p->d2;
    return (n + 255) & ~size_t(255);
}

// ---- fixed scratch of sinkhorn_forward_noalloc ----
//
// One array per GPU, allocated when the code object is loaded and held until
// the process ends.  In host code `scratch` names a host-side stand-in, not
// device memory: its device address is taken once per device with
// hipGetSymbolAddress and only that address is handed to kernels.
__device__ __align__(256) unsigned char scratch[SINKHORN_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array (null on failure).
void *device_scratch() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
        g_scratch_ptr[dev] = ptr;
    }
    return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

const char *sinkhorn_status_string(sk_status s) {
    switch (s) {
        case SK_OK: return "ok";
        case SK_ERR_NULLPTR: return "a required pointer is NULL";
        case SK_ERR_SHAPE: return "invalid shape (B < 0, d1 < 1, d2 < 1, c_batched not 0/1, or size overflow)";
        case SK_ERR_LAMBDA: return "lambda must be finite and > 0";
        case SK_ERR_ITERS: return "n_iter must be >= 0 and tol finite";
        case SK_ERR_WORKSPACE: return "workspace smaller than sinkhorn_workspace_bytes()";
        case SK_ERR_HIP: return "HIP launch failed (is the device a gfx950?)";
        case SK_ERR_ARG: return "an argument is outside its documented set of values";
    }
    return "unknown status";
}

int32_t sinkhorn_regime(const sk_problem *p) {
    if (check_problem(p) != SK_OK) return 0;
    return sk::resident_fits(p->d1, p->d2) ? 1 : 2;
}

size_t sinkhorn_points_workspace_bytes(const sk_problem *p, int32_t D) {
    if (check_points(p, D) != SK_OK) return 0;
    if (points_on_the_fly(p, D)) return sk::tiled_points_workspace_bytes(p->B, p->d1, p->d2);
    return cost_bytes(p) + sinkhorn_workspace_bytes(p);
}

size_t sinkhorn_workspace_bytes(const sk_problem *p) {
    if (check_problem(p) != SK_OK) return 0;
    if (sk::resident_fits(p->d1, p->d2)) return 0;
    return sk::tiled_workspace_bytes(p->B, p->d1, p->d2, p->c_batched);
}

int32_t sinkhorn_describe(const sk_problem *p, int32_t select, char *buf, size_t len) {
    if (select < SK_SELECT_DEFAULT || select > SK_SELECT_NO_COMPACTION) return SK_ERR_ARG;
    const sk_status st = check_problem(p);
    if (st != SK_OK) return st;
    if (!buf && len) return SK_ERR_NULLPTR;
    sk::FwdArgs a = fwd_args(p, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr);
    a.select = select;
    if (p->B == 0) return snprintf(buf, len, "nothing to launch (B = 0)");
    if (!sk::resident_fits(p->d1, p->d2)) return sk::tiled_describe(a, buf, len);
    return resident_describe(a, buf, len);
}

sk_status sinkhorn_forward_select(const sk_problem *p, int32_t select, const float *mu, const float *nu,
                                  const float *C, float *alpha, float *beta, float *loss, float *marg_err,
                                  int32_t *iters, void *workspace, size_t ws_bytes, void *stream) {
    if (select < SK_SELECT_DEFAULT || select > SK_SELECT_NO_COMPACTION) return SK_ERR_ARG;
    sk_status st = check_problem(p);
    if (st != SK_OK) return st;
    if (p->B == 0) return SK_OK;
    if (!mu || !nu || !C || !alpha || !beta || !loss || !marg_err || !iters) return SK_ERR_NULLPTR;
    const size_t need = sinkhorn_workspace_bytes(p);
    if (ws_bytes < need) return SK_ERR_WORKSPACE;
    if (need > 0 && !workspace) return SK_ERR_NULLPTR;
    sk::FwdArgs a = fwd_args(p, mu, nu, C, alpha, beta, loss, marg_err, iters);
    a.select = select;
    return run_forward(a, workspace, static_cast<hipStream_t>(stream)) == hipSuccess ? SK_OK : SK_ERR_HIP;
}

sk_status sinkhorn_forward(const sk_problem *p, const float *mu, const float *nu, const float *C, float *alpha,
                           float *beta, float *loss, float *marg_err, int32_t *iters, void *workspace,
                           size_t ws_bytes, void *stream) {
    return sinkhorn_forward_select(p, SK_SELECT_DEFAULT, mu, nu, C, alpha, beta, loss, marg_err, iters, workspace,
                                   ws_bytes, stream);
}

sk_status sinkhorn_forward_warm(const sk_problem *p, const float *alpha0, const float *mu, const float *nu,
                                const float *C, float *alpha, float *beta, float *loss, float *marg_err,
                                int32_t *iters, void *workspace, size_t ws_bytes, void *stream) {
    sk_status st = check_problem(p);
    if (st != SK_OK) return st;
    if (p->B == 0) return SK_OK;
    if (!alpha0 || !mu || !nu || !C || !alpha || !beta || !loss || !marg_err || !iters) return SK_ERR_NULLPTR;
    const size_t need = sinkhorn_workspace_bytes(p);
    if (ws_bytes < need) return SK_ERR_WORKSPACE;
    if (need > 0 && !workspace) return SK_ERR_NULLPTR;
    sk::FwdArgs a = fwd_args(p, mu, nu, C, alpha, beta, loss, marg_err, iters);
    a.alpha0 = alpha0;
    a.select = SK_SELECT_LOG_ONLY;  // the plain form's start is fixed at u = 1
    return run_forward(a, workspace, static_cast<hipStream_t>(stream)) == hipSuccess ? SK_OK : SK_ERR_HIP;
}

sk_status sinkhorn_forward_noalloc(const sk_problem *p, const float *mu, const float *nu, const float *C,
                                   float *alpha, float *beta, float *loss, float *marg_err, int32_t *iters,
                                   void *stream) {
    sk_status st = check_problem(p);
    if (st != SK_OK) return st;
    if (p->B == 0) return SK_OK;
    if (!mu || !nu || !C || !alpha || !beta || !loss || !marg_err || !iters) return SK_ERR_NULLPTR;
    const size_t need = sinkhorn_workspace_bytes(p);
    if (need > SINKHORN_NOALLOC_SCRATCH_BYTES) return SK_ERR_WORKSPACE;
    void *ws = nullptr;
    if (need > 0 && !(ws = device_scratch())) return SK_ERR_HIP;
    const sk::FwdArgs a = fwd_args(p, mu, nu, C, alpha, beta, loss, marg_err, iters);
    return run_forward(a, ws, static_cast<hipStream_t>(stream)) == hipSuccess ? SK_OK : SK_ERR_HIP;
}

sk_status sinkhorn_backward(const sk_problem *p, const float *grad_loss, const float *mu, const float *nu,
                            const float *C, const float *alpha, const float *beta, float *grad_mu, float *grad_nu,
                            float *grad_C, void *stream) {
    sk_status st = check_problem(p);
    if (st != SK_OK) return st;
    if (p->B == 0) return SK_OK;
    if (!grad_loss || !mu || !nu || !alpha || !beta || !grad_mu || !grad_nu) return SK_ERR_NULLPTR;
    if (grad_C && !C) return SK_ERR_NULLPTR;

    const sk::BwdArgs a = bwd_args(p, grad_loss, mu, nu, C, alpha, beta, grad_mu, grad_nu, grad_C);
    hipError_t e = sk::launch_backward(a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SK_OK : SK_ERR_HIP;
}

size_t sinkhorn_sharp_workspace_bytes(const sk_problem *p) {
    if (check_problem(p) != SK_OK) return 0;
    if (p->d1 <= sk::kSharpMaxD && p->d2 <= sk::kSharpMaxD) return 0;
    if (!sk::sharp_tiled_fits(p->B, p->d1, p->d2)) return 0;
    return sk::sharp_tiled_workspace_bytes(p->B, p->d1, p->d2);
}

sk_status sinkhorn_backward_sharp(const sk_problem *p, const float *grad_loss, const float *mu, const float *nu,
                                  const float *C, const float *alpha, const float *beta, float *grad_mu,
                                  float *grad_nu, int32_t max_cg, float cg_tol, int32_t *cg_iters, void *workspace,
                                  size_t ws_bytes, void *stream) {
    sk_status st = check_problem(p);
    if (st != SK_OK) return st;
    const bool resident = p->d1 <= sk::kSharpMaxD && p->d2 <= sk::kSharpMaxD;
    if (!resident && !sk::sharp_tiled_fits(p->B, p->d1, p->d2)) return SK_ERR_SHAPE;
    if (max_cg < 1 || !(cg_tol >= 0.f) || !isfinite(cg_tol)) return SK_ERR_ITERS;
    if (p->B == 0) return SK_OK;
    if (!grad_loss || !mu || !nu || !C || !alpha || !beta || !grad_mu || !grad_nu) return SK_ERR_NULLPTR;
    const size_t need = sinkhorn_sharp_workspace_bytes(p);
    if (ws_bytes < need) return SK_ERR_WORKSPACE;
    if (need > 0 && !workspace) return SK_ERR_NULLPTR;
    sk::SharpArgs a;
    a.grad_loss = grad_loss;
    a.mu = mu;
    a.nu = nu;
    a.C = C;
    a.alpha = alpha;
    a.beta = beta;
    a.grad_mu = grad_mu;
    a.grad_nu = grad_nu;
    a.cg_iters = cg_iters;
    a.B = p->B;
    a.d1 = p->d1;
    a.d2 = p->d2;
    a.c_batched = p->c_batched;
    a.max_cg = max_cg;
    a.s = sk::kLog2eHost / p->lambda;
    a.cg_tol = cg_tol;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    const hipError_t e = resident ? sk::launch_sharp(a, s) : sk::launch_sharp_tiled(a, workspace, s);
    return e == hipSuccess ? SK_OK : SK_ERR_HIP;
}

sk_status sinkhorn_forward_points(const sk_problem *p, int32_t D, const float *mu, const float *nu, const float *X,
                                  const float *Y, float *alpha, float *beta, float *loss, float *marg_err,
                                  int32_t *iters, void *workspace, size_t ws_bytes, void *stream) {
    sk_status st = check_points(p, D);
    if (st != SK_OK) return st;
    if (p->B == 0) return SK_OK;
    if (!mu || !nu || !X || !Y || !alpha || !beta || !loss || !marg_err || !iters) return SK_ERR_NULLPTR;
    const size_t need = sinkhorn_points_workspace_bytes(p, D);
    if (ws_bytes < need) return SK_ERR_WORKSPACE;
    if (need > 0 && !workspace) return SK_ERR_NULLPTR;
    sk::FwdArgs a = fwd_args(p, mu, nu, nullptr, alpha, beta, loss, marg_err, iters);
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (points_on_the_fly(p, D)) {
        e = sk::launch_tiled_points(a, X, Y, D, sqrt((double)a.s), workspace, s);
    } else {
        float *C = static_cast<float *>(workspace);
        e = sk::launch_points_cost(X, Y, C, p->c_batched ? p->B : 1, p->d1, p->d2, D, s);
        if (e == hipSuccess) {
            a.C = C;
            e = run_forward(a, static_cast<char *>(workspace) + cost_bytes(p), s);
        }
    }
    return e == hipSuccess ? SK_OK : SK_ERR_HIP;
}

sk_status sinkhorn_backward_points(const sk_problem *p, int32_t D, const float *grad_loss, const float *mu,
                                   const float *nu, const float *X, const float *Y, const float *alpha,
                                   const float *beta, float *grad_mu, float *grad_nu, float *grad_X, float *grad_Y,
                                   void *stream) {
    sk_status st = check_points(p, D);
    if (st != SK_OK) return st;
    if (p->B == 0) return SK_OK;
    if (!grad_loss || !mu || !nu || !alpha || !beta || !grad_mu || !grad_nu) return SK_ERR_NULLPTR;
    if ((grad_X || grad_Y) && (!X || !Y)) return SK_ERR_NULLPTR;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = sk::launch_backward(bwd_args(p, grad_loss, mu, nu, nullptr, alpha, beta, grad_mu, grad_nu, nullptr), s);
    if (e == hipSuccess && (grad_X || grad_Y)) {
        sk::PointsBwdArgs g;
        g.grad_loss = grad_loss;
        g.alpha = alpha;
        g.beta = beta;
        g.X = X;
        g.Y = Y;
        g.grad_X = grad_X;
        g.grad_Y = grad_Y;
        g.B = p->B;
        g.d1 = p->d1;
        g.d2 = p->d2;
        g.D = D;
        g.batched = p->c_batched;
        g.rs = (float)sqrt((double)(sk::kLog2eHost / p->lambda));
        e = sk::launch_points_grads(g, s);
    }
    return e == hipSuccess ? SK_OK : SK_ERR_HIP;
}

}  // extern "C"
