// sk_backward.hip -- the Lagrange-multiplier gradient (Section 2) and d/dC.
//
//   grad_mu[b,i] = g_b * lambda * (alpha[b,i] - mean over supp(mu_b) of alpha[b,.])
//   grad_nu[b,j] = g_b * lambda * (beta[b,j]  - mean over supp(nu_b) of beta[b,.])
//   grad_C       = g_b * P_b (per-sample C) or sum_b g_b * P_b (shared C),
//                  P_ij = exp(alpha_i + beta_j - C_ij / lambda)
// The potential gradients are O(B (d1 + d2)); the only heavy part is grad_C,
// which for a per-sample C streams C in and grad_C out once (HBM bound).
#include "sk_device.h"
#include "sk_internal.h"

namespace sk {
namespace {

constexpr int kBwdThreads = 256;

// Block-wide sum in a fixed tree order (deterministic).
__device__ __forceinline__ float block_sum(float v, float *red) {
    v = wave_sum(v);
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    __syncthreads();
    if (lane == 0) red[w] = v;
    __syncthreads();
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < kBwdThreads / 64; ++k) s += red[k];
    return s;
}

// Mean of x over the entries with w > 0; writes g*lambda*(x - mean) there, 0 elsewhere.
__device__ __forceinline__ void centred(const float *x, const float *w, int n, float scale, float *out,
                                        float *red) {
    float s = 0.f, c = 0.f;
    for (int k = threadIdx.x; k < n; k += kBwdThreads) {
        if (w[k] > 0.f) {
            s += x[k];
            c += 1.f;
        }
    }
    s = block_sum(s, red);
    c = block_sum(c, red);
    const float mean = c > 0.f ? s / c : 0.f;
    for (int k = threadIdx.x; k < n; k += kBwdThreads) out[k] = (w[k] > 0.f) ? scale * (x[k] - mean) : 0.f;
}

__global__ __launch_bounds__(kBwdThreads) void sk_bwd_potentials(BwdArgs A) {
    __shared__ float red[kBwdThreads / 64];
    const int b = blockIdx.x;
    const float scale = A.grad_loss[b] * A.lambda;
    centred(A.alpha + (size_t)b * A.d1, A.mu + (size_t)b * A.d1, A.d1, scale, A.grad_mu + (size_t)b * A.d1,
            red);
    centred(A.beta + (size_t)b * A.d2, A.nu + (size_t)b * A.d2, A.d2, scale, A.grad_nu + (size_t)b * A.d2, red);
}

// Per-sample C: one thread per 4 consecutive cells of a row when d2 % 4 == 0
// (128-bit loads/stores), else one per cell.  Grid-stride over all B*d1*d2.
template <bool VEC4>
__global__ __launch_bounds__(kBwdThreads) void sk_bwd_gradC_batched(BwdArgs A) {
    const size_t d2 = A.d2;
    const size_t per = VEC4 ? 4 : 1;
    const size_t n = (size_t)A.B * A.d1 * d2 / per;
    for (size_t u = (size_t)blockIdx.x * kBwdThreads + threadIdx.x; u < n; u += (size_t)gridDim.x * kBwdThreads) {
        const size_t cell = u * per;
        const size_t row = cell / d2;  // = b * d1 + i
        const size_t j = cell - row * d2;
        const size_t b = row / A.d1;
        const float g = A.grad_loss[b];
        const float ai = A.alpha[row] * kLog2e;
        const float *be = A.beta + b * d2 + j;
        if (VEC4) {
            const float4 c = *reinterpret_cast<const float4 *>(A.C + cell);
            float4 o;
            o.x = g * ex2(__builtin_fmaf(be[0], kLog2e, ai) - A.s * c.x);
            o.y = g * ex2(__builtin_fmaf(be[1], kLog2e, ai) - A.s * c.y);
            o.z = g * ex2(__builtin_fmaf(be[2], kLog2e, ai) - A.s * c.z);
            o.w = g * ex2(__builtin_fmaf(be[3], kLog2e, ai) - A.s * c.w);
            __builtin_nontemporal_store(o.x, A.grad_C + cell + 0);
            __builtin_nontemporal_store(o.y, A.grad_C + cell + 1);
            __builtin_nontemporal_store(o.z, A.grad_C + cell + 2);
            __builtin_nontemporal_store(o.w, A.grad_C + cell + 3);
        } else {
            A.grad_C[cell] = g * ex2(__builtin_fmaf(be[0], kLog2e, ai) - A.s * A.C[cell]);
        }
    }
}

// Shared C: grad_C[i, j] = sum_b g_b P_b[i, j]; one thread per (i, j), the
// batch summed in order b = 0..B-1.  Rows are grid-strided over grid y, so any
// d1 fits the grid.
__global__ __launch_bounds__(kBwdThreads) void sk_bwd_gradC_shared(BwdArgs A) {
    const int j = blockIdx.x * kBwdThreads + threadIdx.x;
    if (j >= A.d2) return;
    for (int i = blockIdx.y; i < A.d1; i += gridDim.y) {
        const float c = -A.s * A.C[(size_t)i * A.d2 + j];
        float acc = 0.f;
        for (int b = 0; b < A.B; ++b) {
            const float ai = A.alpha[(size_t)b * A.d1 + i] * kLog2e;
            const float x = __builtin_fmaf(A.beta[(size_t)b * A.d2 + j], kLog2e, ai) + c;
            acc = __builtin_fmaf(A.grad_loss[b], ex2(x), acc);
        }
        A.grad_C[(size_t)i * A.d2 + j] = acc;
    }
}

}  // namespace

hipError_t launch_backward(const BwdArgs &a, hipStream_t st) {
    hipLaunchKernelGGL(sk_bwd_potentials, dim3(a.B), dim3(kBwdThreads), 0, st, a);
    if (a.grad_C) {
        if (a.c_batched) {
            const bool vec = (a.d2 % 4) == 0 && ((uintptr_t)a.C % 16) == 0 && ((uintptr_t)a.grad_C % 16) == 0;
            const size_t units = (size_t)a.B * a.d1 * a.d2 / (vec ? 4 : 1);
            size_t blocks = (units + kBwdThreads - 1) / kBwdThreads;
            if (blocks > 256 * 16) blocks = 256 * 16;
            if (vec)
                hipLaunchKernelGGL(sk_bwd_gradC_batched<true>, dim3(blocks), dim3(kBwdThreads), 0, st, a);
            else
                hipLaunchKernelGGL(sk_bwd_gradC_batched<false>, dim3(blocks), dim3(kBwdThreads), 0, st, a);
        } else {
            dim3 grid((a.d2 + kBwdThreads - 1) / kBwdThreads, a.d1 < 65535 ? a.d1 : 65535);
            hipLaunchKernelGGL(sk_bwd_gradC_shared, grid, dim3(kBwdThreads), 0, st, a);
        }
    }
    return hipGetLastError();
}

}  // namespace sk
