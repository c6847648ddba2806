// sk_resident.hip -- small problems (max(d1, d2) <= 128) entirely on-chip.
//
// One wavefront runs one problem for all iterations: the scaled cost
// cl = -C*log2(e)/lambda sits in LDS (one copy per work-group when C is shared
// by the batch, Section 4), the potentials in VGPRs.  HBM is touched only to
// load the inputs and store the outputs; the convergence check runs in-kernel.
//
// Lane layout: the 64 lanes form an 8 x 8 grid, lane = 8p + q.  Lane (p, q)
// owns rows i = p + 8r (r < N) and columns j = q + 8t (t < N).  Row sums are
// all-reduced over q (8 consecutive lanes, DPP), column sums over p (DPP and
// permlane swaps).
//
// One iteration (v-update then u-update, eq. (sk_plain) order, in the log form
// of Sections 3-4) is ONE sweep with one exponential per cell:
//   e_ij = 2^(a_i + b_j + cl_ij)                (plan after the last v-update)
//   rowsum_i = sum_j e_ij  ->  a_i' = a_i + log2 mu_i - log2 rowsum_i
//   f_i = 2^(a_i' - a_i),   P_ij = e_ij f_i     (plan after the u-update)
//   colsum_j = sum_i P_ij  ->  marginal error, and b_j' = b_j + log2 nu_j - log2 colsum_j
// This is exactly a_i' = log2 mu_i - LSE2_j(b_j + cl_ij) and
// b_j' = log2 nu_j - LSE2_i(a_i' + cl_ij): the logsumexp is shifted by the
// current potential instead of a running maximum.  The shift is a valid bound:
// after a v-update every column sum of the plan is nu_j <= 1, after a u-update
// every row sum is mu_i <= 1, so no term overflows.  When a sum leaves
// [2^-64, 2^64] the exact max-then-sum logsumexp (Section 3) is used for that
// row or column.
#include "sk_device.h"
#include "sk_internal.h"

namespace sk {
namespace {

constexpr float kPadCost = -1.0e30f;              // cells outside the problem: plan entry 0, 0 * cl stays 0
constexpr float kTiny = 1.1754943508222875e-38f;  // 2^-126: floor before a log, keeps inactive sums finite

// The wavefront's cost cells in LDS: cl for (r, t) at base[(r * N + t) * 64].
template <int N>
struct Tile {
    const float *base;
    __device__ __forceinline__ float operator()(int r, int t) const { return base[(r * N + t) * 64]; }
};

// log2 of a shifted sum and whether the sum is trusted (|log2| <= 64).
__device__ __forceinline__ float log2_checked(float s, bool &ok) {
    const float l = lg2(fmaxf(s, kTiny));
    ok = fabsf(l) <= 64.f;
    return l;
}

// Exact v-update for the columns selected by `sel`:
//   b_j = lb_j - LSE2_i(a_i + cl_ij)  (max first, then sum).
template <int N>
__device__ __forceinline__ void col_exact(const Tile<N> &cl, const float (&a)[N], float (&bv)[N],
                                          const float (&lb)[N], const bool (&sel)[N]) {
#pragma unroll
    for (int t = 0; t < N; ++t) {
        asm volatile("" ::: "memory");
        float mx = neg_inf();
#pragma unroll
        for (int r = 0; r < N; ++r) mx = fmaxf(mx, a[r] + cl(r, t));
        mx = max_p(mx);
        const float ms = (mx == neg_inf()) ? 0.f : mx;
        float v[N];
#pragma unroll
        for (int r = 0; r < N; ++r) v[r] = ex2(a[r] + cl(r, t) - ms);
        const float s = sum_p(tree_sum<N>(v));
        if (sel[t]) bv[t] = lb[t] - (ms + lg2(s));
    }
}

// Exact u-update of row r: returns a_r = la_r - LSE2_j(b_j + cl_rj).
template <int N>
__device__ __forceinline__ float row_exact(const Tile<N> &cl, int r, const float (&bv)[N], float la) {
    float m = neg_inf();
#pragma unroll
    for (int t = 0; t < N; ++t) m = fmaxf(m, bv[t] + cl(r, t));
    m = max_q(m);
    const float ms = (m == neg_inf()) ? 0.f : m;
    float v[N];
#pragma unroll
    for (int t = 0; t < N; ++t) v[t] = ex2(bv[t] + cl(r, t) - ms);
    return la - (ms + lg2(sum_q(tree_sum<N>(v))));
}

// One sweep = the u-update of every row plus the column sums of the plan
// after it (left in cs, all-reduced over p).  Returns the marginal error of
// the rows (wavefront-uniform) when CHECK.
template <int N, int RC, bool CHECK>
__device__ __forceinline__ float sweep(const Tile<N> &cl, float (&a)[N], const float (&la)[N], const float *mub,
                                       const float (&bv)[N], float (&cs)[N], int p, int q) {
    float colpart[N];
#pragma unroll
    for (int t = 0; t < N; ++t) colpart[t] = 0.f;
    float rowerr = 0.f;

#pragma unroll
    for (int r0 = 0; r0 < N; r0 += RC) {
        // The cost tile never changes; without this the compiler hoists all
        // N*N LDS reads out of the iteration loop into VGPRs.
        asm volatile("" ::: "memory");
        float e[RC][N], rs[RC], f[RC];
#pragma unroll
        for (int rr = 0; rr < RC; ++rr) {
            const int r = r0 + rr;
            if (r < N) {
#pragma unroll
                for (int t = 0; t < N; ++t) e[rr][t] = ex2((a[r] + bv[t]) + cl(r, t));
                rs[rr] = sum_q(tree_sum<N>(e[rr]));
            }
        }
        bool bad_any = false;
        bool redo[RC];
#pragma unroll
        for (int rr = 0; rr < RC; ++rr) {
            const int r = r0 + rr;
            if (r < N) {
                const bool act = la[r] != neg_inf();
                bool ok;
                const float l = log2_checked(rs[rr], ok);
                const float an = (a[r] + la[r]) - l;
                f[rr] = (act && ok) ? ex2(an - a[r]) : 0.f;
                if (act && ok) a[r] = an;
                redo[rr] = act && !ok;
                bad_any |= redo[rr];
            }
        }
        if (__any(bad_any)) {
            // Exact u-update for the rows whose shifted sum left the trusted
            // range; their entries are rebuilt from the new potential in the
            // units the column accumulator uses.
#pragma unroll
            for (int rr = 0; rr < RC; ++rr) {
                const int r = r0 + rr;
                if (r < N) {
                    const float an = row_exact(cl, r, bv, la[r]);
                    float part = 0.f;
#pragma unroll
                    for (int t = 0; t < N; ++t) {
                        const float v = ex2((an + bv[t]) + cl(r, t));
                        if (redo[rr]) e[rr][t] = v;
                        part += v;
                    }
                    part = sum_q(part);
                    if (redo[rr]) {
                        a[r] = an;
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
                if (CHECK && q == 0 && la[r] != neg_inf()) rowerr += fabsf(f[rr] * rs[rr] - mub[p + 8 * r]);
#pragma unroll
                for (int t = 0; t < N; ++t) colpart[t] = __builtin_fmaf(e[rr][t], f[rr], colpart[t]);
            }
        }
    }
#pragma unroll
    for (int t = 0; t < N; ++t) cs[t] = sum_p(colpart[t]);
    return CHECK ? wave_sum(rowerr) : 0.f;
}

// The plan of the current (a, b), built entry by entry and never stored
// (Section 4): the marginal error and sum P*cl (wavefront-uniform).
template <int N>
__device__ __forceinline__ void plan_stats(const Tile<N> &cl, const float (&a)[N], const float (&la)[N],
                                           const float *mub, const float (&bv)[N], const float (&lb)[N],
                                           const float *nub, float &err, float &loss, int p, int q) {
    asm volatile("" ::: "memory");
    float colpart[N], lossp[N];
#pragma unroll
    for (int t = 0; t < N; ++t) colpart[t] = lossp[t] = 0.f;
    float rowerr = 0.f;
#pragma unroll
    for (int r = 0; r < N; ++r) {
        float v[N];
#pragma unroll
        for (int t = 0; t < N; ++t) {
            const float c = cl(r, t);
            v[t] = ex2((a[r] + bv[t]) + c);
            colpart[t] += v[t];
            lossp[t] = __builtin_fmaf(v[t], c, lossp[t]);
        }
        const float part = sum_q(tree_sum<N>(v));
        if (q == 0 && la[r] != neg_inf()) rowerr += fabsf(part - mub[p + 8 * r]);
    }
    float colerr = 0.f;
#pragma unroll
    for (int t = 0; t < N; ++t) {
        const float c = sum_p(colpart[t]);
        if (p == 0 && lb[t] != neg_inf()) colerr += fabsf(c - nub[q + 8 * t]);
    }
    err = wave_sum(rowerr + colerr);
    loss = wave_sum(tree_sum<N>(lossp));
}

// Column part of the marginal error, summed over the 8 lanes (p = 0) that hold
// distinct columns; wavefront-uniform.
template <int N>
__device__ __forceinline__ float col_error(const float (&cs)[N], const float (&lb)[N], const float *nub, int p,
                                           int q) {
    float e = 0.f;
    if (p == 0) {
#pragma unroll
        for (int t = 0; t < N; ++t)
            if (lb[t] != neg_inf()) e += fabsf(cs[t] - nub[q + 8 * t]);
    }
    return wave_sum(e);
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

    if (A.only_flagged) {
        // Skip the work-group unless one of its problems was left to this kernel.
        bool any = false;
#pragma unroll
        for (int v = 0; v < WPB; ++v) {
            const int bb = blockIdx.x * WPB + v;
            any |= bb < A.B && A.iters[bb] == -1;
        }
        if (!any) return;
    }
    // Stage cl in the lane-blocked layout; cells outside the problem hold kPadCost.
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
    if (A.only_flagged && A.iters[b] != -1) return;

    const Tile<N> cl{lds + (BATCHED ? w * N * N * 64 : 0) + lane};
    const float *mub = A.mu + (size_t)b * d1;
    const float *nub = A.nu + (size_t)b * d2;
    float a[N], la[N];  // row potentials, log2 mu (-inf: zero mass or padding)
    float bv[N], lb[N];  // column potentials, log2 nu
#pragma unroll
    for (int r = 0; r < N; ++r) {
        const int i = p + 8 * r;
        const float m = (i < d1) ? mub[i] : 0.f;
        la[r] = m > 0.f ? log2f(m) : neg_inf();
        // log u^0 = 0 on the support, -inf off it; padding rows stay 0 (their
        // cells are kPadCost already).
        a[r] = (i < d1 && !(m > 0.f)) ? neg_inf() : 0.f;
    }
#pragma unroll
    for (int t = 0; t < N; ++t) {
        const int j = q + 8 * t;
        const float m = (j < d2) ? nub[j] : 0.f;
        lb[t] = m > 0.f ? log2f(m) : neg_inf();
        bv[t] = (j < d2 && !(m > 0.f)) ? neg_inf() : 0.f;
    }

    const int n_iter = A.n_iter;
    const float tol = A.tol;
    int K = n_iter;
    float cs[N];
    if (n_iter > 0) {
        bool all[N];
#pragma unroll
        for (int t = 0; t < N; ++t) all[t] = lb[t] != neg_inf();
        col_exact<N>(cl, a, bv, lb, all);  // v-update of iteration 1
        for (int k = 1;; ++k) {
            if (k == n_iter) {
                sweep<N, RC, false>(cl, a, la, mub, bv, cs, p, q);  // u-update of the last iteration
                break;
            }
            if (tol > 0.f) {
                const float err = sweep<N, RC, true>(cl, a, la, mub, bv, cs, p, q);
                if (err + col_error<N>(cs, lb, nub, p, q) <= tol) {
                    K = k;
                    break;
                }
            } else {
                sweep<N, RC, false>(cl, a, la, mub, bv, cs, p, q);
            }
            // v-update of iteration k+1 from the column sums just measured.
            bool bad[N];
            bool bad_any = false;
#pragma unroll
            for (int t = 0; t < N; ++t) {
                const bool act = lb[t] != neg_inf();
                bool ok;
                const float l = log2_checked(cs[t], ok);
                if (act && ok) bv[t] = (bv[t] + lb[t]) - l;
                bad[t] = act && !ok;
                bad_any |= bad[t];
            }
            if (__any(bad_any)) col_exact<N>(cl, a, bv, lb, bad);
        }
    }
    float err, loss;
    plan_stats<N>(cl, a, la, mub, bv, lb, nub, err, loss, p, q);

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
        A.loss[b] = -loss / A.s;  // sum P*C = -(1/s) sum P*cl
        A.marg_err[b] = err;
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
