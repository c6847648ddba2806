// sk_points.hip -- costs given by point clouds: C_ij = sum_k (x_ik - y_jk)^2.
//
// Section 4 closes by noting that the cost entries can be recreated from the
// points instead of being stored.  The tiled sweep over per-sample clouds does
// exactly that (sk_tiled.hip, sk_tiled_sweep_points).  This file holds the
// rest of the point-cloud path:
//   * sk_points_cost: the cost matrix written out, for the shapes that keep
//     it on-chip anyway (max(d1, d2) <= 128), for shared clouds (one matrix
//     for the batch) and for shapes the on-the-fly sweep does not take;
//   * the gradient with respect to the points, by the chain rule through
//     dW/dC = P (the multiplier gradient of Section 2 extended to C):
//       grad_x[i] = g * sum_j P_ij * 2 (x_i - y_j),
//       grad_y[j] = g * sum_i P_ij * 2 (y_j - x_i),
//     with P_ij = exp(alpha_i + beta_j - C_ij / lambda) rebuilt on the fly and
//     (for shared clouds) the batch summed in order b = 0..B-1.
#include "sk_device.h"
#include "sk_internal.h"

namespace sk {
namespace {

constexpr int kPtThreads = 256;

// C[b, i, j] = sum_k (x_ik - y_jk)^2 in coordinate order; one thread per cell,
// grid-stride (clouds [nb, d, D], nb = B or 1).
__global__ __launch_bounds__(kPtThreads) void sk_points_cost(const float *X, const float *Y, float *C, int nb,
                                                             int d1, int d2, int D) {
    const size_t n = (size_t)nb * d1 * d2;
    for (size_t u = (size_t)blockIdx.x * kPtThreads + threadIdx.x; u < n; u += (size_t)gridDim.x * kPtThreads) {
        const size_t row = u / d2;  // = b * d1 + i
        const size_t j = u - row * d2;
        const size_t b = row / d1;
        const float *x = X + row * D;
        const float *y = Y + (b * d2 + j) * D;
        float acc = 0.f;
        for (int k = 0; k < D; ++k) {
            const float dd = x[k] - y[k];
            acc = __builtin_fmaf(dd, dd, acc);
        }
        C[u] = acc;
    }
}

// Scaled cost of a cell, the same expression as the tiled points sweep:
// -sum_k (rs x_k - rs y_k)^2 with rs = sqrt(log2(e) / lambda).
__device__ __forceinline__ float cl_cell(const float *x, const float *y, int D, float rs) {
    float acc = 0.f;
    for (int k = 0; k < D; ++k) {
        const float dd = rs * x[k] - rs * y[k];
        acc = __builtin_fmaf(dd, dd, acc);
    }
    return -acc;
}

// grad_x: one wavefront per row i (and problem b, or the whole batch for
// shared clouds); lanes stride over j; D <= kPointsGradD accumulators per lane.
__global__ __launch_bounds__(kPtThreads) void sk_points_grad_x(PointsBwdArgs A) {
    const int lane = threadIdx.x & 63;
    const size_t wid = (size_t)blockIdx.x * (kPtThreads / 64) + (threadIdx.x >> 6);
    const size_t nrows = (size_t)(A.batched ? A.B : 1) * A.d1;
    if (wid >= nrows) return;
    const int i = (int)(wid % A.d1);
    const int bx = (int)(wid / A.d1);  // clouds index (0 for shared clouds)
    const int D = A.D;
    const float *x = A.X + wid * D;
    float acc[kPointsGradD];
#pragma unroll
    for (int k = 0; k < kPointsGradD; ++k) acc[k] = 0.f;
    const int b0 = A.batched ? bx : 0, b1 = A.batched ? bx + 1 : A.B;
    for (int b = b0; b < b1; ++b) {
        const float g = 2.f * A.grad_loss[b];
        const float ai = A.alpha[(size_t)b * A.d1 + i] * kLog2e;
        const float *Yb = A.Y + (size_t)bx * A.d2 * D;
        float part[kPointsGradD];
#pragma unroll
        for (int k = 0; k < kPointsGradD; ++k) part[k] = 0.f;
        for (int j = lane; j < A.d2; j += 64) {
            const float *y = Yb + (size_t)j * D;
            const float p = ex2(__builtin_fmaf(A.beta[(size_t)b * A.d2 + j], kLog2e, ai) + cl_cell(x, y, D, A.rs));
#pragma unroll
            for (int k = 0; k < kPointsGradD; ++k)
                if (k < D) part[k] = __builtin_fmaf(p, x[k] - y[k], part[k]);
        }
#pragma unroll
        for (int k = 0; k < kPointsGradD; ++k) acc[k] = __builtin_fmaf(g, part[k], acc[k]);
    }
#pragma unroll
    for (int k = 0; k < kPointsGradD; ++k) {
        const float v = wave_sum(acc[k]);
        if (k < D && lane == 0) A.grad_X[wid * D + k] = v;
    }
}

// grad_y: lanes = 64 columns j (one wavefront per column block and problem,
// or the whole batch for shared clouds); rows summed in order.
__global__ __launch_bounds__(kPtThreads) void sk_points_grad_y(PointsBwdArgs A) {
    const int lane = threadIdx.x & 63;
    const int JB = (A.d2 + 63) / 64;
    const size_t wid = (size_t)blockIdx.x * (kPtThreads / 64) + (threadIdx.x >> 6);
    const size_t nw = (size_t)(A.batched ? A.B : 1) * JB;
    if (wid >= nw) return;
    const int bx = (int)(wid / JB);
    const int j = (int)(wid % JB) * 64 + lane;
    if (j >= A.d2) return;
    const int D = A.D;
    const float *y = A.Y + ((size_t)bx * A.d2 + j) * D;
    float acc[kPointsGradD];
#pragma unroll
    for (int k = 0; k < kPointsGradD; ++k) acc[k] = 0.f;
    const int b0 = A.batched ? bx : 0, b1 = A.batched ? bx + 1 : A.B;
    for (int b = b0; b < b1; ++b) {
        const float g = 2.f * A.grad_loss[b];
        const float bj = A.beta[(size_t)b * A.d2 + j] * kLog2e;
        const float *Xb = A.X + (size_t)bx * A.d1 * D;
        float part[kPointsGradD];
#pragma unroll
        for (int k = 0; k < kPointsGradD; ++k) part[k] = 0.f;
        for (int i = 0; i < A.d1; ++i) {
            const float *x = Xb + (size_t)i * D;
            const float p = ex2(__builtin_fmaf(A.alpha[(size_t)b * A.d1 + i], kLog2e, bj) + cl_cell(x, y, D, A.rs));
#pragma unroll
            for (int k = 0; k < kPointsGradD; ++k)
                if (k < D) part[k] = __builtin_fmaf(p, y[k] - x[k], part[k]);
        }
#pragma unroll
        for (int k = 0; k < kPointsGradD; ++k) acc[k] = __builtin_fmaf(g, part[k], acc[k]);
    }
#pragma unroll
    for (int k = 0; k < kPointsGradD; ++k)
        if (k < D) A.grad_Y[((size_t)bx * A.d2 + j) * D + k] = acc[k];
}

}  // namespace

hipError_t launch_points_cost(const float *X, const float *Y, float *C, int nb, int d1, int d2, int D,
                              hipStream_t st) {
    const size_t n = (size_t)nb * d1 * d2;
    size_t blocks = (n + kPtThreads - 1) / kPtThreads;
    if (blocks > 256 * 16) blocks = 256 * 16;
    hipLaunchKernelGGL(sk_points_cost, dim3(blocks), dim3(kPtThreads), 0, st, X, Y, C, nb, d1, d2, D);
    return hipGetLastError();
}

hipError_t launch_points_grads(const PointsBwdArgs &a, hipStream_t st) {
    const int wpb = kPtThreads / 64;
    const size_t nb = a.batched ? a.B : 1;
    if (a.grad_X) {
        const size_t waves = nb * a.d1;
        hipLaunchKernelGGL(sk_points_grad_x, dim3((waves + wpb - 1) / wpb), dim3(kPtThreads), 0, st, a);
    }
    if (a.grad_Y) {
        const size_t waves = nb * ((a.d2 + 63) / 64);
        hipLaunchKernelGGL(sk_points_grad_y, dim3((waves + wpb - 1) / wpb), dim3(kPtThreads), 0, st, a);
    }
    return hipGetLastError();
}

}  // namespace sk
