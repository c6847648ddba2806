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

// One side's point gradient for per-sample clouds, as a sweep over that
// side's points ("rows"; the other side's points are the "columns"):
//   out[b, i] = 2 g_b sum_j P_ij (r_i - c_j),
//   P_ij = 2^(a_i + b_j - |rs r_i - rs c_j|^2)   (a, b: base-2 potentials).
// Called once with (X, Y, alpha, beta) for grad_X and once with the roles
// swapped for grad_Y (P is the same in both roles).  Work-group (row block,
// problem), wavefront per row; lane l keeps the scaled coordinates and the
// potentials of its columns j = l + 64 c in registers; a row's coordinates
// and potential arrive one row ahead in vector registers.  Each row is
// finished by one wavefront (three wavefront sums), so no cross-work-group
// reduction and no workspace is needed.
struct GradSweepArgs {
    const float *rows, *cols;  // [B, nr, D], [B, nc, D]
    const float *pr, *pc;      // natural-log potentials [B, nr], [B, nc]
    const float *grad_loss;    // [B]
    float *out;                // [B, nr, D]
    int nr, nc, RBS;
    float rs;
};
constexpr float kFarCoord = 1.0e18f;  // padding columns: cl = -3e36, P = 0

template <int NCW, int D>
__global__ __launch_bounds__(kPtThreads) void sk_points_grad_sweep(GradSweepArgs A) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int b = blockIdx.y;
    const int nr = A.nr, nc = A.nc;
    const float rs = A.rs;
    const float *rb = A.rows + (size_t)b * nr * D;
    const float *cb = A.cols + (size_t)b * nc * D;
    const float *pr = A.pr + (size_t)b * nr;
    // Raw column values first (clamped index: all loads in flight together).
    float ys[NCW][D], bv[NCW];
#pragma unroll
    for (int c = 0; c < NCW; ++c) {
        const int jj = min(lane + 64 * c, nc - 1);
        bv[c] = A.pc[(size_t)b * nc + jj];
#pragma unroll
        for (int q = 0; q < D; ++q) ys[c][q] = cb[(size_t)jj * D + q];
    }
#pragma unroll
    for (int c = 0; c < NCW; ++c) {
        const bool in = lane + 64 * c < nc;
        bv[c] = in ? bv[c] * kLog2e : 0.f;
#pragma unroll
        for (int q = 0; q < D; ++q) ys[c][q] = in ? rs * ys[c][q] : kFarCoord;
    }
    const float g2 = 2.f * A.grad_loss[b] / rs;  // the sums below are in scaled coordinates
    int vz = 0;
    __asm__ volatile("" : "+v"(vz));  // a zero the compiler cannot see as uniform
    float xn[D], an = 0.f;
    const int i0 = blockIdx.x * A.RBS, i1 = min(nr, i0 + A.RBS);
    auto load_row = [&](int i) {  // raw values: the arithmetic waits for the next row
        const int ii = min(i, i1 - 1) + vz;  // clamped: the prefetch past the block re-reads its last row
#pragma unroll
        for (int q = 0; q < D; ++q) xn[q] = rb[(size_t)ii * D + q];
        an = pr[ii];
    };
    const int step = kPtThreads / 64;
    if (i0 + w < i1) load_row(i0 + w);
    for (int i = i0 + w; i < i1; i += step) {
        float xs[D];
#pragma unroll
        for (int q = 0; q < D; ++q) xs[q] = rs * xn[q];
        const float ai = an * kLog2e;
        load_row(i + step);
        float gq[D];
#pragma unroll
        for (int q = 0; q < D; ++q) gq[q] = 0.f;
#pragma unroll
        for (int c = 0; c < NCW; ++c) {
            float dd[D], acc = 0.f;
#pragma unroll
            for (int q = 0; q < D; ++q) {
                dd[q] = xs[q] - ys[c][q];
                acc = __builtin_fmaf(dd[q], dd[q], acc);
            }
            const float e = ex2((ai + bv[c]) - acc);
#pragma unroll
            for (int q = 0; q < D; ++q) gq[q] = __builtin_fmaf(e, dd[q], gq[q]);
        }
#pragma unroll
        for (int q = 0; q < D; ++q) {
            const float v = wave_sum(gq[q]);
            if (lane == 0) A.out[((size_t)b * nr + i) * D + q] = g2 * v;
        }
    }
}

template <int D>
void grad_sweep(const GradSweepArgs &g, int B, hipStream_t st) {
    const dim3 grid((g.nr + g.RBS - 1) / g.RBS, B), blk(kPtThreads);
    const int ncw = (g.nc + 63) / 64;
    if (ncw <= 4) hipLaunchKernelGGL((sk_points_grad_sweep<4, D>), grid, blk, 0, st, g);
    else if (ncw <= 8) hipLaunchKernelGGL((sk_points_grad_sweep<8, D>), grid, blk, 0, st, g);
    else if (ncw <= 16) hipLaunchKernelGGL((sk_points_grad_sweep<16, D>), grid, blk, 0, st, g);
    else hipLaunchKernelGGL((sk_points_grad_sweep<32, D>), grid, blk, 0, st, g);
}

void grad_sweep_side(const PointsBwdArgs &a, bool side_x, hipStream_t st) {
    GradSweepArgs g;
    g.rows = side_x ? a.X : a.Y;
    g.cols = side_x ? a.Y : a.X;
    g.pr = side_x ? a.alpha : a.beta;
    g.pc = side_x ? a.beta : a.alpha;
    g.grad_loss = a.grad_loss;
    g.out = side_x ? a.grad_X : a.grad_Y;
    g.nr = side_x ? a.d1 : a.d2;
    g.nc = side_x ? a.d2 : a.d1;
    g.RBS = 64;  // 16 rows per wavefront: the columns' registers are loaded once per 16 rows
    g.rs = a.rs;
    if (a.D == 1) grad_sweep<1>(g, a.B, st);
    else if (a.D == 2) grad_sweep<2>(g, a.B, st);
    else grad_sweep<3>(g, a.B, st);
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
    // Per-sample clouds with few coordinates: row sweeps with the other side
    // in registers (both sides at most 2048 points).
    if (a.batched && a.D <= kPointsMaxD && a.d1 <= kPointsMaxD2 && a.d2 <= kPointsMaxD2 && a.B <= 65535) {
        if (a.grad_X) grad_sweep_side(a, true, st);
        if (a.grad_Y) grad_sweep_side(a, false, st);
        return hipGetLastError();
    }
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
