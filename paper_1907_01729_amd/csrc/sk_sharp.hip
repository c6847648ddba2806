// sk_sharp.hip -- gradient of the sharp loss E^0 = <P, C> with respect to
// (mu, nu) (Section 5 points to this sharper gradient; the multiplier
// gradient of sk_backward.hip is that of E^lambda).
//
// Implicit differentiation of the entropic plan through its marginal
// constraints: a change of the marginals moves the plan by
// dP_ij = P_ij (df_i + dg_j) / lambda with
//     [diag(r)  P      ] [df]            [dmu]
//     [P^T      diag(c)] [dg] = lambda * [dnu],       r = P 1, c = P^T 1,
// and dE^0 = (<a, df> + <b, dg>) / lambda with a = (P o C) 1, b = (P o C)^T 1,
// so the gradient is the solution z of H z = (a, b) for the same symmetric
// matrix H.  H is positive semi-definite and singular along (1, -1) (a
// constant moved from f to g); the right-hand side is projected off that
// direction and each block of z is centred over its support afterwards
// (the gradient on the simplex is defined up to a constant per block; 0 off
// the support).  Solved per problem by conjugate gradients preconditioned
// with diag(H) = (r, c).
//
// One work-group of 256 threads per problem, max(d1, d2) <= 128: P lives in
// LDS with an odd row stride (conflict-free both along rows and along
// columns); thread t < 128 owns row t, thread 128 + t owns column t, so one
// pass over P forms both halves of H p.  Reductions are fixed-order block
// sums (deterministic).
#include "sk_device.h"
#include "sk_internal.h"

namespace sk {
namespace {

constexpr int kShThreads = 256;
constexpr int kShHalf = kShThreads / 2;  // rows on threads [0, 128), columns on [128, 256)
static_assert(kShHalf >= kSharpMaxD, "one thread per row and per column");

__device__ __forceinline__ float block_sum(float v, float *red) {
    v = wave_sum(v);
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    __syncthreads();
    if (lane == 0) red[w] = v;
    __syncthreads();
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < kShThreads / 64; ++k) s += red[k];
    return s;
}

__host__ __device__ __forceinline__ int ld_of(int d2) { return d2 | 1; }  // odd row stride

// sum_m a[m * stride] * v[m], m < n, from LDS: eight loads in flight and four
// independent accumulators (a single chain would wait on every load).
__device__ __forceinline__ float dot_lds(const float *a, int stride, const float *v, int n) {
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
    int m = 0;
    for (; m + 8 <= n; m += 8) {
        float x[8], y[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            x[u] = a[(m + u) * stride];
            y[u] = v[m + u];
        }
        s0 = __builtin_fmaf(x[0], y[0], s0);
        s1 = __builtin_fmaf(x[1], y[1], s1);
        s2 = __builtin_fmaf(x[2], y[2], s2);
        s3 = __builtin_fmaf(x[3], y[3], s3);
        s0 = __builtin_fmaf(x[4], y[4], s0);
        s1 = __builtin_fmaf(x[5], y[5], s1);
        s2 = __builtin_fmaf(x[6], y[6], s2);
        s3 = __builtin_fmaf(x[7], y[7], s3);
    }
    for (; m < n; ++m) s0 = __builtin_fmaf(a[m * stride], v[m], s0);
    return (s0 + s1) + (s2 + s3);
}

__global__ __launch_bounds__(kShThreads) void sk_sharp_kernel(SharpArgs A) {
    extern __shared__ float P[];  // [d1][ld]: the cost first, then the plan
    __shared__ float pv[2 * kShHalf];
    __shared__ float av[kShHalf], bw[kShHalf];  // base-2 potentials
    __shared__ float red[kShThreads / 64];
    const int b = blockIdx.x, t = threadIdx.x;
    const int d1 = A.d1, d2 = A.d2, ld = ld_of(d2);
    const float *Cb = A.C + (A.c_batched ? (size_t)b * d1 * d2 : 0);
    const float *al = A.alpha + (size_t)b * d1;
    const float *be = A.beta + (size_t)b * d2;

    // Stage the cost (coalesced: thread t takes column t & 127 of every other
    // row, d2 <= 128) and the potentials in LDS.
    if (t < d1) av[t] = al[t] * kLog2e;
    if (t < d2) bw[t] = be[t] * kLog2e;
    // Eight loads in flight per thread before their stores: a load-store
    // pair per row would wait out the memory latency once per row.
    const int sj = t & (kShHalf - 1), si = t / kShHalf;
    constexpr int kRs = kShThreads / kShHalf;  // rows per pass
    if (sj < d2) {
        for (int i0 = si; i0 < d1; i0 += 8 * kRs) {
            float v[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int i = i0 + kRs * k;
                v[k] = i < d1 ? Cb[(size_t)i * d2 + sj] : 0.f;
            }
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int i = i0 + kRs * k;
                if (i < d1) P[i * ld + sj] = v[k];
            }
        }
    }
    __syncthreads();

    const bool isrow = t < kShHalf;
    const int k = isrow ? t : t - kShHalf;
    const bool own = isrow ? k < d1 : k < d2;
    // Diagonal of H (the plan's marginal) and the right-hand side (a or b),
    // with the plan entries P_ij = 2^(a_i + b_j - s C_ij) formed on the way.
    float dg = 0.f, rhs = 0.f;
    if (own) {
        if (isrow) {
            const float a = av[k];
#pragma unroll 4
            for (int j = 0; j < d2; ++j) {
                const float c = P[k * ld + j];
                const float p = ex2((a + bw[j]) - A.s * c);
                dg += p;
                rhs = __builtin_fmaf(p, c, rhs);
            }
        } else {
            const float bb = bw[k];
#pragma unroll 4
            for (int i = 0; i < d1; ++i) {
                const float c = P[i * ld + k];
                const float p = ex2((av[i] + bb) - A.s * c);
                dg += p;
                rhs = __builtin_fmaf(p, c, rhs);
            }
        }
    }
    __syncthreads();  // the cost has been read: the plan overwrites it
    if (sj < d2) {
        const float bj = bw[sj];
#pragma unroll 4
        for (int i = si; i < d1; i += kRs) P[i * ld + sj] = ex2((av[i] + bj) - A.s * P[i * ld + sj]);
    }
    __syncthreads();
    const float mass = own ? (isrow ? A.mu[(size_t)b * d1 + k] : A.nu[(size_t)b * d2 + k]) : 0.f;
    const bool sup = own && mass > 0.f && dg > 0.f;
    if (!sup) {
        dg = 0.f;
        rhs = 0.f;
    }
    // Project the right-hand side off (1, -1) over the supports.
    {
        const float sgn = isrow ? 1.f : -1.f;
        const float dot = block_sum(sup ? sgn * rhs : 0.f, red);
        const float n = block_sum(sup ? 1.f : 0.f, red);
        if (sup) rhs -= sgn * (dot / n);
    }

    // Jacobi-preconditioned conjugate gradients; every scalar below is a
    // block sum, so the control flow is uniform across the work-group.
    float x = 0.f, r = rhs;
    float z = sup ? r / dg : 0.f, p = z;
    float rz = block_sum(r * z, red);
    const float stop = A.cg_tol * A.cg_tol * rz;
    int it = 0;
    if (rz > 0.f) {
        while (it < A.max_cg) {
            if (own) pv[isrow ? k : kShHalf + k] = p;
            __syncthreads();
            float q = dg * p;
            if (sup) q += isrow ? dot_lds(P + k * ld, 1, pv + kShHalf, d2) : dot_lds(P + k, ld, pv, d1);
            const float pq = block_sum(p * q, red);  // its barriers also retire the reads of pv
            if (!(pq > 0.f)) break;
            const float step = rz / pq;
            x = __builtin_fmaf(step, p, x);
            r = __builtin_fmaf(-step, q, r);
            z = sup ? r / dg : 0.f;
            const float rzn = block_sum(r * z, red);
            ++it;
            if (!(rzn > stop)) break;
            p = __builtin_fmaf(rzn / rz, p, z);
            rz = rzn;
        }
    }

    // Centre each block over its support, scale by the upstream gradient.
    const float sx_r = block_sum(sup && isrow ? x : 0.f, red);
    const float n_r = block_sum(sup && isrow ? 1.f : 0.f, red);
    const float sx_c = block_sum(sup && !isrow ? x : 0.f, red);
    const float n_c = block_sum(sup && !isrow ? 1.f : 0.f, red);
    const float g = A.grad_loss[b];
    if (own) {
        const float mean = isrow ? (n_r > 0.f ? sx_r / n_r : 0.f) : (n_c > 0.f ? sx_c / n_c : 0.f);
        const float v = sup ? g * (x - mean) : 0.f;
        if (isrow)
            A.grad_mu[(size_t)b * d1 + k] = v;
        else
            A.grad_nu[(size_t)b * d2 + k] = v;
    }
    if (t == 0 && A.cg_iters) A.cg_iters[b] = it;
}

size_t sharp_lds_bytes(int d1, int d2) { return sizeof(float) * (size_t)d1 * ld_of(d2); }

}  // namespace

hipError_t launch_sharp(const SharpArgs &a, hipStream_t st) {
    const size_t lds = sharp_lds_bytes(a.d1, a.d2);
    static bool attr = false;  // above 64 KB of LDS (d near 128) needs the larger dynamic limit
    if (!attr) {
        (void)hipFuncSetAttribute(reinterpret_cast<const void *>(&sk_sharp_kernel),
                                  hipFuncAttributeMaxDynamicSharedMemorySize,
                                  (int)sharp_lds_bytes(kSharpMaxD, kSharpMaxD));
        attr = true;
    }
    hipLaunchKernelGGL(sk_sharp_kernel, dim3(a.B), dim3(kShThreads), lds, st, a);
    return hipGetLastError();
}

}  // namespace sk
