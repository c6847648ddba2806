// sk_internal.h -- host-side launchers shared between the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/sinkhorn.h"

namespace sk {

constexpr float kLog2eHost = 1.44269504088896340736f;

struct FwdArgs {
    const float *mu, *nu, *C;
    float *alpha, *beta, *loss, *marg_err;
    int32_t *iters;
    int B, d1, d2, n_iter, c_batched;
    float lambda, tol;
    float s;  // log2(e) / lambda
    // Kernel selector of sinkhorn_forward_select (an sk_select value).
    int select;
    // Set (to 1) for the log-domain launch that follows a plain-form launch of
    // the widest bucket: it solves only the problems marked with iters = -1.
    int only_marked;
    // Warm start: alpha^0 [B, d1] (natural log) on the support of mu instead
    // of 0; null for the cold start.  Only the log-domain kernels take it.
    const float *alpha0;
};

struct BwdArgs {
    const float *grad_loss, *mu, *nu, *C, *alpha, *beta;
    float *grad_mu, *grad_nu, *grad_C;
    int B, d1, d2, c_batched;
    float lambda;
    float s;  // log2(e) / lambda
};

// Largest support size of the resident kernels (one work-group of two
// wavefronts per problem, the cost in VGPRs).
constexpr int kResidentMaxD = 128;

bool resident_fits(int d1, int d2);
// The log-domain kernel.
hipError_t launch_resident(const FwdArgs &a, hipStream_t st);
// Plain-form resident kernels: each returns false (and launches nothing) when
// it does not take the shape; otherwise *err is the launch status.  Problems
// it cannot keep in range are solved in the log domain by the same
// work-group (left with iters = -1 under SK_SELECT_PLAIN_ONLY).
// A shared cost with d1 = d2 <= 104, two wavefronts per problem
// on the vector ALU.  On a cost that is not symmetric each work-group runs
// the general kernel's iteration in place.
bool launch_resident_sym(const FwdArgs &a, hipStream_t st, hipError_t *err);
// Same contract; any cost (shared or per problem) with max(d1, d2) <= 128,
// two wavefronts per problem on the vector ALU.
bool launch_resident_gen(const FwdArgs &a, hipStream_t st, hipError_t *err);

// The tiled sweep keeps a whole cost row in one wavefront's registers.
constexpr int kTiledMaxD2 = 4096;
// The tiled kernels carry the batch on a grid dimension of at most 65535
// work-groups: a larger batch runs as consecutive chunks of at most that
// many problems (the problems are independent), each chunk reusing the
// workspace of the largest one in stream order.
constexpr int kTiledMaxBatch = 65535;
inline int tiled_chunk(int B) { return B < kTiledMaxBatch ? B : kTiledMaxBatch; }
// The arguments of problems [off, off + n) of a forward.
inline FwdArgs fwd_chunk(const FwdArgs &a, int off, int n) {
    FwdArgs c = a;
    const size_t o1 = (size_t)off * a.d1, o2 = (size_t)off * a.d2;
    c.mu += o1;
    c.alpha += o1;
    if (a.alpha0) c.alpha0 += o1;
    c.nu += o2;
    c.beta += o2;
    if (a.C && a.c_batched) c.C += o1 * a.d2;
    c.loss += off;
    c.marg_err += off;
    c.iters += off;
    c.B = n;
    return c;
}
// Runs launch(off, n) over the chunks of a batch of B problems, stopping at
// the first error.
template <class Launch>
hipError_t for_each_chunk(int B, Launch launch) {
    for (int off = 0; off < B; off += kTiledMaxBatch) {
        const hipError_t e = launch(off, B - off < kTiledMaxBatch ? B - off : kTiledMaxBatch);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}
bool tiled_fits(int B, int d1, int d2, int c_batched);
size_t tiled_workspace_bytes(int B, int d1, int d2, int c_batched);
hipError_t launch_tiled(const FwdArgs &a, void *ws, hipStream_t st);
// One line on the kernels and launch shape launch_tiled takes for a (snprintf
// semantics: the length of the whole line).
int tiled_describe(const FwdArgs &a, char *buf, size_t len);

hipError_t launch_backward(const BwdArgs &a, hipStream_t st);

// Gradient of the sharp loss E^0 (implicit differentiation of the plan,
// conjugate gradients per problem); the plan of one problem sits in the
// VGPRs of its two wavefronts.
constexpr int kSharpMaxD = 128;
struct SharpArgs {
    const float *grad_loss, *mu, *nu, *C, *alpha, *beta;
    float *grad_mu, *grad_nu;
    int32_t *cg_iters;  // may be null
    int B, d1, d2, c_batched, max_cg;
    float s;  // log2(e) / lambda
    float cg_tol;
};
hipError_t launch_sharp(const SharpArgs &a, hipStream_t st);
// Larger supports: the plan rebuilt in sweeps over the cost for every
// product, the conjugate-gradient vectors in a workspace.
bool sharp_tiled_fits(int B, int d1, int d2);
size_t sharp_tiled_workspace_bytes(int B, int d1, int d2);
hipError_t launch_sharp_tiled(const SharpArgs &a, void *ws, hipStream_t st);

// Point clouds (C_ij = sum_k (x_ik - y_jk)^2).  The tiled sweep computes the
// cost on the fly for per-sample clouds with up to kPointsMaxD coordinates
// and d2 <= kPointsMaxD2 (the columns' coordinates live in registers); other
// shapes write the cost out first.  Gradients take up to kPointsGradD
// coordinates.
constexpr int kPointsMaxD = 3;
constexpr int kPointsMaxD2 = 2048;
constexpr int kPointsGradD = 16;

struct PointsBwdArgs {
    const float *grad_loss, *alpha, *beta, *X, *Y;
    float *grad_X, *grad_Y;  // either may be null
    int B, d1, d2, D, batched;
    float rs;  // sqrt(log2(e) / lambda)
};

bool tiled_points_fits(int B, int d1, int d2, int D);
size_t tiled_points_workspace_bytes(int B, int d1, int d2);
hipError_t launch_tiled_points(const FwdArgs &a, const float *X, const float *Y, int D, double rs, void *ws,
                               hipStream_t st);
hipError_t launch_points_cost(const float *X, const float *Y, float *C, int nb, int d1, int d2, int D,
                              hipStream_t st);
hipError_t launch_points_grads(const PointsBwdArgs &a, hipStream_t st);

}  // namespace sk
