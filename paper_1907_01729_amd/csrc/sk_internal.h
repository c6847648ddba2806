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
    // Set when a plain-form launch ran first: solve only the problems it
    // marked with iters = -only_flagged (-1: out of the plain form's range;
    // -2: the cost is not symmetric) and leave the others untouched.
    int only_flagged;
};

struct BwdArgs {
    const float *grad_loss, *mu, *nu, *C, *alpha, *beta;
    float *grad_mu, *grad_nu, *grad_C;
    int B, d1, d2, c_batched;
    float lambda;
    float s;  // log2(e) / lambda
};

// Largest support size the resident (one wavefront per problem) kernel takes.
constexpr int kResidentMaxD = 128;

bool resident_fits(int d1, int d2);
hipError_t launch_resident(const FwdArgs &a, hipStream_t st);
// Plain-form resident kernel: returns false (and launches nothing) when it
// does not take the shape; otherwise *err is the launch status.  Problems it
// cannot keep in range come back with iters = -1.
bool launch_resident_plain(const FwdArgs &a, hipStream_t st, hipError_t *err);
// Same contract; a cost shared by the batch only, products on the matrix cores.
// With only_flagged = 2 it solves the problems marked iters = -2.
bool launch_resident_mfma(const FwdArgs &a, hipStream_t st, hipError_t *err);
// Same contract; a shared cost with d1 = d2 <= 104, one wavefront per problem
// on the vector ALU.  A cost that is not symmetric marks every problem with
// iters = -2 (for the matrix-core kernel).
bool launch_resident_sym(const FwdArgs &a, hipStream_t st, hipError_t *err);

// The tiled sweep keeps a whole cost row in one wavefront's registers.
constexpr int kTiledMaxD2 = 4096;
bool tiled_fits(int B, int d1, int d2, int c_batched);
size_t tiled_workspace_bytes(int B, int d1, int d2, int c_batched);
hipError_t launch_tiled(const FwdArgs &a, void *ws, hipStream_t st);

hipError_t launch_backward(const BwdArgs &a, hipStream_t st);

}  // namespace sk
