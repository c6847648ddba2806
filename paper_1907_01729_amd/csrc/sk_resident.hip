// sk_resident.hip -- one wavefront per problem, everything on-chip.
//
// For supports up to 128 points the whole problem lives on the CU for all
// iterations: the scaled cost cl = -C*log2(e)/lambda in LDS (one copy shared by
// the workgroup's wavefronts when C is shared by the batch, Section 4), the
// potentials in VGPRs.  HBM is touched only to load the inputs and to store the
// outputs; the convergence check runs in-kernel.
//
// Lane layout: the 64 lanes form an 8 x 8 grid, lane = 8p + q.  Lane (p, q)
// owns rows i = p + 8r (r < N) and columns j = q + 8t (t < N), i.e. an N x N
// block of cells.  Row sums are all-reduced over q (8 consecutive lanes, DPP),
// column sums over p (lanes with equal q).
//
// One iteration (v-update then u-update, Section 1 eq. (sk_plain), in the log
// form of Sections 3-4) is computed as ONE sweep over the cells with one
// exponential per cell:
//   e_ij = 2^(a_i + b_j + cl_ij)                (plan before the u-update)
//   rowsum_i = sum_j e_ij  ->  a_i' = a_i + log2 mu_i - log2 rowsum_i
//   f_i = 2^(a_i' - a_i),   P_ij = e_ij f_i     (plan after the u-update)
//   colsum_j = sum_i P_ij  ->  marginal error, and b_j' = b_j + log2 nu_j - log2 colsum_j
// This is exactly a_i' = log2 mu_i - LSE2_j(b_j + cl_ij) and
// b_j' = log2 nu_j - LSE2_i(a_i' + cl_ij): the logsumexp is shifted by the
// current potential instead of a running maximum.  The shift is a valid bound:
// after a v-update every column sum of the plan is nu_j <= 1, after a u-update
// every row sum is mu_i <= 1, so no term overflows.  When a sum underflows
// (< 2^-64) the exact max-then-sum logsumexp (Section 3) is used for that
// row or column.
#include "sk_device.h"
#include "sk_internal.h"

namespace sk {
namespace {

constexpr float kPadCost = -1.0e30f;

template <int N>
struct Cells {
    // cl for lane's (r, t) cell: base[(r * N + t) * 64]
    const float *base;
    __device__ __forceinline__ float operator()(int r, int t) const { return base[(r * N + t) * 64]; }
};

// Exact v-update for the columns selected by `sel`:
//   b_j = lb_j - LSE2_i(a_i + cl_ij)  (max first, then sum).
template <int N>
__device__ __forceinline__ void col_exact(const Cells<N> &cl, const float (&a)[N], float (&bv)[N],
                                          const float (&lb)[N], const bool (&sel)[N]) {
#pragma unroll
    for (int t = 0; t < N; ++t) {
        float m = neg_inf();
#pragma unroll
        for (int r = 0; r < N; ++r) m = fmaxf(m, a[r] + cl(r, t));
        m = max_p(m);
        const float ms = (m == neg_inf()) ? 0.f : m;
        float s = 0.f;
#pragma unroll
        for (int r = 0; r < N; ++r) s += ex2(a[r] + cl(r, t) - ms);
        s = sum_p(s);
        if (sel[t]) bv[t] = lb[t] - (ms + lg2(s));
    }
}

// Exact u-update of row r: returns a_r = la_r - LSE2_j(b_j + cl_rj).
template <int N>
__device__ __forceinline__ float row_exact(const Cells<N> &cl, int r, const float (&bv)[N], float la) {
    float m = neg_inf();
#pragma unroll
    for (int t = 0; t < N; ++t) m = fmaxf(m, bv[t] + cl(r, t));
    m = max_q(m);
    const float ms = (m == neg_inf()) ? 0.f : m;
    float s = 0.f;
#pragma unroll
    for (int t = 0; t < N; ++t) s += ex2(bv[t] + cl(r, t) - ms);
    s = sum_q(s);
    return la - (ms + lg2(s));
}

// One sweep = the u-update of the rows plus the column sums of the plan after
// it.  Column sums are left in cs (all-reduced, identical on every lane that
// shares the column); returns the marginal L1 error of that plan
// (wave-uniform).
template <int N, int RC>
__device__ __forceinline__ float sweep(const Cells<N> &cl, float (&a)[N], const float (&la)[N],
                                       const float (&mu)[N], const bool (&ract)[N], const float (&bv)[N],
                                       const float (&nu)[N], const bool (&cact)[N], float (&cs)[N], int p,
                                       int q) {
    float colpart[N];
#pragma unroll
    for (int t = 0; t < N; ++t) colpart[t] = 0.f;
    float rowerr = 0.f;

#pragma unroll
    for (int r0 = 0; r0 < N; r0 += RC) {
        // The cost tile in LDS never changes, so the compiler would otherwise
        // hoist all N*N reads out of the iteration loop into VGPRs.
        asm volatile("" ::: "memory");
        float e[RC][N];
        float rs[RC], f[RC];
#pragma unroll
        for (int rr = 0; rr < RC; ++rr) {
            const int r = r0 + rr;
            if (r < N) {
                float part = 0.f;
#pragma unroll
                for (int t = 0; t < N; ++t) {
                    const float v = ex2((a[r] + bv[t]) + cl(r, t));
                    e[rr][t] = v;
                    part += v;
                }
                rs[rr] = sum_q(part);
            }
        }
        bool bad_any = false;
#pragma unroll
        for (int rr = 0; rr < RC; ++rr) {
            const int r = r0 + rr;
            if (r < N) {
                const bool ok = rs[rr] >= kSumLo && rs[rr] <= kSumHi;
                if (ract[r] && ok) {
                    const float an = a[r] + la[r] - lg2(rs[rr]);
                    f[rr] = ex2(an - a[r]);
                    a[r] = an;
                } else {
                    f[rr] = 0.f;
                }
                bad_any |= ract[r] && !ok;
            }
        }
        if (__any(bad_any)) {
            // Exact u-update for the rows whose shifted sum left the trusted
            // range; their plan entries are recomputed from the new potential.
#pragma unroll
            for (int rr = 0; rr < RC; ++rr) {
                const int r = r0 + rr;
                if (r < N) {
                    const bool redo = ract[r] && !(rs[rr] >= kSumLo && rs[rr] <= kSumHi);
                    const float an = row_exact(cl, r, bv, la[r]);
                    if (redo) a[r] = an;
                    float part = 0.f;
#pragma unroll
                    for (int t = 0; t < N; ++t) {
                        const float v = ex2((a[r] + bv[t]) + cl(r, t));
                        if (redo) e[rr][t] = v;
                        part += v;
                    }
                    part = sum_q(part);
                    if (redo) {
                        rs[rr] = part;
                        f[rr] = 1.f;
                    }
                }
            }
        }
#pragma unroll
        for (int rr = 0; rr < RC; ++rr) {
            const int r = r0 + rr;
            if (r < N) {
                if (q == 0 && ract[r]) rowerr += fabsf(f[rr] * rs[rr] - mu[r]);
#pragma unroll
                for (int t = 0; t < N; ++t) colpart[t] = __builtin_fmaf(e[rr][t], f[rr], colpart[t]);
            }
        }
    }
    float colerr = 0.f;
#pragma unroll
    for (int t = 0; t < N; ++t) {
        cs[t] = sum_p(colpart[t]);
        if (p == 0 && cact[t]) colerr += fabsf(cs[t] - nu[t]);
    }
    return wave_sum(rowerr + colerr);
}

struct Stats {
    float err;   // ||P 1 - mu||_1 + ||P^T 1 - nu||_1
    float loss;  // sum_ij P_ij C_ij
};

// The plan of the current (a, b), built entry by entry and never stored
// (Section 4): its marginal error and E^0 = sum P C = -(1/s) sum P cl.
template <int N>
__device__ __forceinline__ Stats plan_stats(const Cells<N> &cl, const float (&a)[N], const float (&mu)[N],
                                            const bool (&ract)[N], const float (&bv)[N], const float (&nu)[N],
                                            const bool (&cact)[N], float s, int p, int q) {
    asm volatile("" ::: "memory");
    float colpart[N];
#pragma unroll
    for (int t = 0; t < N; ++t) colpart[t] = 0.f;
    float rowerr = 0.f, losspart = 0.f;
#pragma unroll
    for (int r = 0; r < N; ++r) {
        float part = 0.f;
#pragma unroll
        for (int t = 0; t < N; ++t) {
            const float c = cl(r, t);
            const float v = ex2((a[r] + bv[t]) + c);
            part += v;
            colpart[t] += v;
            losspart = __builtin_fmaf(v, c, losspart);
        }
        part = sum_q(part);
        if (q == 0 && ract[r]) rowerr += fabsf(part - mu[r]);
    }
    float colerr = 0.f;
#pragma unroll
    for (int t = 0; t < N; ++t) {
        const float c = sum_p(colpart[t]);
        if (p == 0 && cact[t]) colerr += fabsf(c - nu[t]);
    }
    Stats o;
    o.err = wave_sum(rowerr + colerr);
    o.loss = -wave_sum(losspart) / s;
    return o;
}

template <int N, int WPB, bool BATCHED>
__global__ __launch_bounds__(64 * WPB) void sk_resident_kernel(FwdArgs A) {
    extern __shared__ float lds[];
    constexpr int RC = N >= 4 ? 4 : N;
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int p = lane >> 3, q = lane & 7;
    const int b = blockIdx.x * WPB + w;
    const int d1 = A.d1, d2 = A.d2;

    // Stage cl = -C * log2(e) / lambda in the lane-blocked layout; cells
    // outside the d1 x d2 problem hold kPadCost so that their plan entry is 0
    // (finite, so that 0 * cl stays 0 in the loss).
    if (!BATCHED) {
        for (int idx = threadIdx.x; idx < N * N * 64; idx += 64 * WPB) {
            const int ln = idx & 63, rt = idx >> 6;
            const int r = rt / N, t = rt - r * N;
            const int i = (ln >> 3) + 8 * r, j = (ln & 7) + 8 * t;
            lds[idx] = (i < d1 && j < d2) ? -A.s * A.C[(size_t)i * d2 + j] : kPadCost;
        }
    } else if (b < A.B) {
        float *my = lds + w * N * N * 64;
        const float *Cb = A.C + (size_t)b * d1 * d2;
        for (int rt = 0; rt < N * N; ++rt) {
            const int r = rt / N, t = rt - r * N;
            const int i = p + 8 * r, j = q + 8 * t;
            my[rt * 64 + lane] = (i < d1 && j < d2) ? -A.s * Cb[(size_t)i * d2 + j] : kPadCost;
        }
    }
    __syncthreads();
    if (b >= A.B) return;

    Cells<N> cl{lds + (BATCHED ? w * N * N * 64 : 0) + lane};

    float a[N], la[N], mu[N];
    bool ract[N];
    float bv[N], lb[N], nu[N];
    bool cact[N];
    const float *mub = A.mu + (size_t)b * d1;
    const float *nub = A.nu + (size_t)b * d2;
#pragma unroll
    for (int r = 0; r < N; ++r) {
        const int i = p + 8 * r;
        const float m = (i < d1) ? mub[i] : 0.f;
        mu[r] = m;
        ract[r] = m > 0.f;
        la[r] = ract[r] ? log2f(m) : neg_inf();
        // log u^0 = 0 on the support, -inf off it; padding rows stay 0 (their
        // cells are -inf already).
        a[r] = (i < d1 && !ract[r]) ? neg_inf() : 0.f;
    }
#pragma unroll
    for (int t = 0; t < N; ++t) {
        const int j = q + 8 * t;
        const float m = (j < d2) ? nub[j] : 0.f;
        nu[t] = m;
        cact[t] = m > 0.f;
        lb[t] = cact[t] ? log2f(m) : neg_inf();
        bv[t] = (j < d2 && !cact[t]) ? neg_inf() : 0.f;
    }

    const int n_iter = A.n_iter;
    const float tol = A.tol;
    int K = n_iter;
    float cs[N];
    if (n_iter > 0) {
        col_exact<N>(cl, a, bv, lb, cact);  // v-update of iteration 1
        for (int k = 1; k < n_iter; ++k) {
            const float err = sweep<N, RC>(cl, a, la, mu, ract, bv, nu, cact, cs, p, q);
            if (tol > 0.f && err <= tol) {
                K = k;
                break;
            }
            // v-update of iteration k+1 from the column sums just measured.
            bool bad[N];
            bool bad_any = false;
#pragma unroll
            for (int t = 0; t < N; ++t) {
                const bool ok = cs[t] >= kSumLo && cs[t] <= kSumHi;
                bad[t] = cact[t] && !ok;
                bad_any |= bad[t];
                if (cact[t] && ok) bv[t] = bv[t] + lb[t] - lg2(cs[t]);
            }
            if (__any(bad_any)) col_exact<N>(cl, a, bv, lb, bad);
        }
        if (K == n_iter) sweep<N, RC>(cl, a, la, mu, ract, bv, nu, cact, cs, p, q);  // u-update of the last iteration
    }
    const Stats o = plan_stats<N>(cl, a, mu, ract, bv, nu, cact, A.s, p, q);

    if (q == 0) {
        float *al = A.alpha + (size_t)b * d1;
#pragma unroll
        for (int r = 0; r < N; ++r) {
            const int i = p + 8 * r;
            if (i < d1) al[i] = a[r] * kLn2;
        }
    }
    if (p == 0) {
        float *be = A.beta + (size_t)b * d2;
#pragma unroll
        for (int t = 0; t < N; ++t) {
            const int j = q + 8 * t;
            if (j < d2) be[j] = bv[t] * kLn2;
        }
    }
    if (lane == 0) {
        A.loss[b] = o.loss;
        A.marg_err[b] = o.err;
        A.iters[b] = K;
    }
}

template <int N>
hipError_t launch_n(const FwdArgs &a, hipStream_t st) {
    const size_t cells = (size_t)N * N * 64 * sizeof(float);
    if (!a.c_batched) {
        constexpr int WPB = 4;
        dim3 grid((a.B + WPB - 1) / WPB), block(64 * WPB);
        hipLaunchKernelGGL((sk_resident_kernel<N, WPB, false>), grid, block, cells, st, a);
    } else {
        constexpr int WPB = 1;
        dim3 grid(a.B), block(64 * WPB);
        hipLaunchKernelGGL((sk_resident_kernel<N, WPB, true>), grid, block, cells * WPB, st, a);
    }
    return hipGetLastError();
}

}  // namespace

bool resident_fits(int d1, int d2) { return d1 <= kResidentMaxD && d2 <= kResidentMaxD; }

hipError_t launch_resident(const FwdArgs &a, hipStream_t st) {
    const int dm = a.d1 > a.d2 ? a.d1 : a.d2;
    const int n = (dm + 7) / 8;
    if (n <= 2) return launch_n<2>(a, st);
    if (n <= 4) return launch_n<4>(a, st);
    if (n <= 8) return launch_n<8>(a, st);
    if (n <= 13) return launch_n<13>(a, st);
    return launch_n<16>(a, st);
}

}  // namespace sk
