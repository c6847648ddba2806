// sk_resident_log.h -- the log-domain iteration (Section 3, eq. (log_sk) with
// the sign of the batched form of Section 4) of one problem with
// max(d1, d2) <= 128 by one work-group of two wavefronts, as a device
// function: the body of sk_resident_log_kernel, and what the plain-form
// kernels run in place for a problem they cannot keep in fp32 range.
//
// Lane layout of the plain-form kernels: lane (p, q) (p = lane & 7,
// q = lane >> 3) of wavefront w holds the scaled cost cl = -C log2(e)/lambda
// of cells [p + 8r][q + 8t] for its row blocks r (ceil(N / 2) of them from 0
// for wavefront 0, floor(N / 2) after them for wavefront 1) and every column
// block t < N, in VGPRs.  The row
// potential a_i (base 2) lives on lane (p, q < H) of the wavefront holding
// row i, the column potential b_j on thread j; each is published to LDS.
//
// One iteration (v-update then u-update) is one pass over the cells with one
// exponential per cell, as in the tiled sweep:
//   e_ij = 2^(a_i + b_j + cl_ij)                 (plan after the last v-update)
//   R_i = sum_j e_ij -> a_i' = a_i + log2 mu_i - log2 R_i,  f_i = 2^(a_i' - a_i)
//   S_j = sum_i e_ij f_i (plan after the u-update) -> b_j' = b_j + log2 nu_j - log2 S_j
// i.e. the logsumexp of each half-step shifted by the current potential
// (a valid bound: column sums of the plan after a v-update are nu_j <= 1, row
// sums after a u-update mu_i <= 1).  A row or column whose shifted sum leaves
// [2^-64, 2^64] takes the exact max-then-sum logsumexp instead; the first
// v-update always does.  Row sums meet through the per-wavefront LDS
// transpose, column sums through the work-group's column partials (two
// barriers per iteration: partials written, potentials published; a column
// that needs the exact update is flagged at the second and takes it after,
// with a third).  With
// N <= 13 the plan entries of a pass stay in VGPRs between the row sums and
// the column sums; wider problems (cost and entries would not fit together)
// rebuild them from the new row potentials: two exponentials per cell.
#ifndef SK_RESIDENT_LOG_H_
#define SK_RESIDENT_LOG_H_

#include "sk_resident_gen.h"

namespace sk {
namespace {

constexpr float kPadCl = -1.0e30f;  // scaled cost of cells off the problem: plan entry 0, finite (0 * cl = 0)

// LDS of the log-domain iteration: float offsets into its pool (16-byte
// aligned where 16-byte accesses are made).
constexpr int kLogColv = 0;                                // b by columns: [j & 7][j >> 3]
constexpr int kLogColm = kLogColv + 8 * kVS;               // column maxima of the exact v-update
constexpr int kLogRowa = kLogColm + 8 * kVS;               // a by rows: [p][r]
constexpr int kLogRowf = kLogRowa + 8 * kVS;               // f by rows (-1: the row took the exact update)
constexpr int kLogCp = kLogRowf + 8 * kVS;                 // column partials
constexpr int kLogTsum = kLogCp + kColumnPartialsFloats;   // per-wavefront row-total scratch
constexpr int kLogRed = kLogTsum + 2 * kRowTotalsFloats;   // stop-test and result reports
constexpr int kLogFlag = kLogRed + 8;                      // exact-update flags of the columns
constexpr int kLogLdsFloats = kLogFlag + 4;
static_assert(kLogColm % 4 == 0 && kLogRowa % 4 == 0 && kLogRowf % 4 == 0 && kLogCp % 4 == 0 &&
                  kLogTsum % 4 == 0 && kLogRed % 4 == 0,
              "16-byte offsets");

// Largest of column c's 16 partials (8 lanes p, 2 wavefronts).
__device__ __forceinline__ float column_max(const float *cp, int c) {
    const float4 *v0 = reinterpret_cast<const float4 *>(cp + c * 8);
    const float4 *v1 = reinterpret_cast<const float4 *>(cp + (128 + c) * 8);
    const float4 a = v0[0], b = v0[1], e = v1[0], f = v1[1];
    return fmaxf(fmaxf(fmaxf(fmaxf(a.x, a.y), fmaxf(a.z, a.w)), fmaxf(fmaxf(b.x, b.y), fmaxf(b.z, b.w))),
                 fmaxf(fmaxf(fmaxf(e.x, e.y), fmaxf(e.z, e.w)), fmaxf(fmaxf(f.x, f.y), fmaxf(f.z, f.w))));
}

// One problem (b = blockIdx.x) per work-group of 128 threads; every thread
// calls it from work-group-uniform control flow.  pool: kLogLdsFloats floats
// of LDS, 16-byte aligned, contents irrelevant.
// Wavefront W holds H row blocks from R0 on: ceil(N / 2) from 0 for W = 0,
// floor(N / 2) after them for W = 1 (no block past the problem); the two run
// separate instantiations of this body, which pass the same barriers.
template <int N, int W>
__device__ __forceinline__ void resident_log_wave(const FwdArgs &A, float *pool) {
    constexpr int H = W == 0 ? (N + 1) / 2 : N / 2;
    constexpr int R0 = W == 0 ? 0 : (N + 1) / 2;
    constexpr bool KEEP = N <= 13;  // plan entries of a pass held in VGPRs
    static_assert(8 * N <= 128 && H <= 8 && N <= kVS, "one thread per column, one lane per row");
    float(&colv)[8 * kVS] = lds_at<float[8 * kVS]>(pool, kLogColv);
    float(&colm)[8 * kVS] = lds_at<float[8 * kVS]>(pool, kLogColm);
    float(&rowa)[8 * kVS] = lds_at<float[8 * kVS]>(pool, kLogRowa);
    float(&rowf)[8 * kVS] = lds_at<float[8 * kVS]>(pool, kLogRowf);
    float(&cp)[kColumnPartialsFloats] = lds_at<float[kColumnPartialsFloats]>(pool, kLogCp);
    float(&tsum)[2][kRowTotalsFloats] = lds_at<float[2][kRowTotalsFloats]>(pool, kLogTsum);
    // [iteration parity][wavefront][row error, column error]
    float(&red)[2][2][2] = lds_at<float[2][2][2]>(pool, kLogRed);
    // [iteration parity][wavefront]: some column of the wavefront's threads
    // left the trusted range (the parity keeps a flag readable until both
    // wavefronts have passed the next iteration's barriers)
    float(&cflag)[2][2] = lds_at<float[2][2]>(pool, kLogFlag);

    const int b = blockIdx.x;
    const int lane = threadIdx.x & 63;
    constexpr int w = W;
    const int p = lane & 7, q = lane >> 3;
    const int d1 = A.d1, d2 = A.d2;
    const float s = A.s;
    const float *Cb = A.C + (A.c_batched ? (size_t)b * d1 * d2 : 0);
    const float *mub = A.mu + (size_t)b * d1;
    float *const tb = tsum[w];

    // Scaled cost of the lane's cells; cells off the problem hold kPadCl.
    const int voff = (p * d2 + q) * 4;
    const int rlim = (d1 - p + 7) >> 3, tlim = (d2 - q + 7) >> 3;
    float L[H][N];
#pragma unroll
    for (int ii = 0; ii < H; ++ii) {
        const __amdgpu_buffer_rsrc_t rs = rows_rsrc(Cb, d1, d2, 8 * (R0 + ii));
#pragma unroll
        for (int t = 0; t < N; ++t) L[ii][t] = load_cell(rs, voff + 32 * t);
    }
#pragma unroll
    for (int ii = 0; ii < H; ++ii)
#pragma unroll
        for (int t = 0; t < N; ++t) L[ii][t] = ((R0 + ii < rlim) && (t < tlim)) ? -s * L[ii][t] : kPadCl;

    // Owners: lane (p, q < H) owns row i = p + 8 (R0 + q); thread c owns
    // column c.  a^0 = 0 on the support of mu (a warm start's alpha^0 in
    // base 2 there), -inf off it (rows past d1 keep 0: their cells hold
    // kPadCl); b likewise before the first v-update.
    const bool rown = q < H;
    const int i_own = p + 8 * (R0 + q);
    const bool row_in = rown && i_own < d1;
    const int c = threadIdx.x;
    const bool col_in = c < d2;
    const float ms = row_in ? mub[i_own] : 0.f;
    const float ns = col_in ? A.nu[(size_t)b * d2 + c] : 0.f;
    const float la = ms > 0.f ? log2f(ms) : neg_inf();
    const float lb = ns > 0.f ? log2f(ns) : neg_inf();
    const int rslot = p * kVS + R0 + q;
    const int cslot = (c & 7) * kVS + (c >> 3);
    float a_own = row_in && !(ms > 0.f) ? neg_inf() : 0.f;
    if (row_in && ms > 0.f && A.alpha0) a_own = A.alpha0[(size_t)b * d1 + i_own] * kLog2e;
    float b_own = col_in && !(ns > 0.f) ? neg_inf() : 0.f;
    if (rown) rowa[rslot] = a_own;
    if (c < 8 * N) colv[cslot] = b_own;
    __syncthreads();

    auto read_rows = [&](const float(&src)[8 * kVS], float(&v)[H]) {
#pragma unroll
        for (int ii = 0; ii < H; ++ii) v[ii] = src[p * kVS + R0 + ii];
    };
    auto read_cols = [&](float(&v)[N]) {
#pragma unroll
        for (int t = 0; t < N; ++t) v[t] = colv[q * kVS + t];
    };

    // Exact v-update b_j = log2 nu_j - LSE2_i(a_i + cl_ij) (max, then sum) of
    // the columns whose thread passes sel; three barriers.
    auto exact_cols = [&](bool sel) {
        float ar[H];
        read_rows(rowa, ar);
#pragma unroll
        for (int t = 0; t < N; ++t) {
            float m = neg_inf();
#pragma unroll
            for (int ii = 0; ii < H; ++ii) m = fmaxf(m, ar[ii] + L[ii][t]);
            cp[partial_at(w, p, q, t)] = m;
        }
        __syncthreads();
        const float M = col_in ? column_max(cp, c) : neg_inf();
        if (c < 8 * N) colm[cslot] = M;
        __syncthreads();
#pragma unroll
        for (int t = 0; t < N; ++t) {
            const float mt = colm[q * kVS + t];
            const float sh = mt == neg_inf() ? 0.f : mt;
            float sum = 0.f;
#pragma unroll
            for (int ii = 0; ii < H; ++ii) sum += ex2(ar[ii] + L[ii][t] - sh);
            cp[partial_at(w, p, q, t)] = sum;
        }
        __syncthreads();
        if (sel) b_own = lb - ((M == neg_inf() ? 0.f : M) + lg2(column_total(cp, c)));
    };

    const int n_iter = A.n_iter;
    const float tol = A.tol;
    const bool check = tol > 0.f;
    int kstop = n_iter;
    if (n_iter > 0) {
        exact_cols(ns > 0.f);  // v-update of iteration 1
        if (c < 8 * N) colv[cslot] = b_own;
        __syncthreads();
        for (int k = 1;; ++k) {
            float(&rd)[2][2] = red[k & 1];
            const int pb = progress_priority(k, n_iter);
            // ---- u-update of iteration k: row sums of the plan e_ij
            float ar[H], bc[N], x[H];
            read_rows(rowa, ar);
            read_cols(bc);
            float e[KEEP ? H : 1][KEEP ? N : 1];
            set_issue_priority(pb);
#pragma unroll
            for (int ii = 0; ii < H; ++ii) {
                if constexpr (KEEP) {
#pragma unroll
                    for (int t = 0; t < N; ++t) e[ii][t] = ex2((ar[ii] + bc[t]) + L[ii][t]);
                    x[ii] = tree_sum<N>(e[ii]);
                } else {
                    float xs = 0.f;
#pragma unroll
                    for (int t = 0; t < N; ++t) xs += ex2((ar[ii] + bc[t]) + L[ii][t]);
                    x[ii] = xs;
                }
            }
            set_issue_priority(pb + 1);
            const float R = row_totals<H>(x, tb, p, q);
            float f = 0.f, rerr = 0.f;
            bool bad = false;
            if (ms > 0.f) {
                if (R >= kSumLo && R <= kSumHi) {
                    const float an = a_own + la - lg2(R);
                    f = ex2(an - a_own);
                    rerr = fabsf(f * R - ms);
                    a_own = an;
                } else {
                    bad = true;
                }
            }
            if (__any(bad)) {
                // Exact u-update (max, then sum) of this wavefront's rows;
                // the owners of the rows whose shifted sum left the trusted
                // range take it, and their plan entries are rebuilt from the
                // new potential below (f = -1 marks them).
                float my_lse = 0.f;
#pragma unroll
                for (int ii = 0; ii < H; ++ii) {
                    float m = neg_inf();
#pragma unroll
                    for (int t = 0; t < N; ++t) m = fmaxf(m, bc[t] + L[ii][t]);
                    m = max_p(m);
                    const float sh = m == neg_inf() ? 0.f : m;
                    float sum = 0.f;
#pragma unroll
                    for (int t = 0; t < N; ++t) sum += ex2(bc[t] + L[ii][t] - sh);
                    const float lse = sh + lg2(sum_p(sum));
                    my_lse = q == ii ? lse : my_lse;
                }
                if (bad) a_own = la - my_lse;
                // Row sums of the rebuilt entries (every lane: the new
                // potentials of the lane's rows come back through LDS, from
                // lanes of this wavefront).
                if (rown) rowa[rslot] = a_own;
                __builtin_amdgcn_wave_barrier();
                float my_rsum = 0.f;
#pragma unroll
                for (int ii = 0; ii < H; ++ii) {
                    const float an = rowa[p * kVS + R0 + ii];
                    float sum = 0.f;
#pragma unroll
                    for (int t = 0; t < N; ++t) sum += ex2((an + bc[t]) + L[ii][t]);
                    const float rs = sum_p(sum);
                    my_rsum = q == ii ? rs : my_rsum;
                }
                if (bad) {
                    f = -1.f;
                    rerr = fabsf(my_rsum - ms);
                }
            }
            if (rown) {
                rowa[rslot] = a_own;
                rowf[rslot] = f;
            }
            if (check) {
                const float re = wave_sum(rerr);
                if (lane == 0) rd[w][0] = re;
            }
            if (k == n_iter) break;

            // ---- column sums of the plan after the u-update
            __builtin_amdgcn_wave_barrier();  // this wavefront's rows published (its own rows only)
            float y[N];
            if constexpr (KEEP) {
                float fr[H];
                read_rows(rowf, fr);
                bool re_any = false;
#pragma unroll
                for (int ii = 0; ii < H; ++ii) re_any |= fr[ii] < 0.f;
                if (__any(re_any)) {
                    float an[H];
                    read_rows(rowa, an);
#pragma unroll
                    for (int ii = 0; ii < H; ++ii) {
                        const bool rb = fr[ii] < 0.f;
#pragma unroll
                        for (int t = 0; t < N; ++t) e[ii][t] = rb ? ex2((an[ii] + bc[t]) + L[ii][t]) : e[ii][t];
                        fr[ii] = rb ? 1.f : fr[ii];
                    }
                }
                set_issue_priority(pb);
#pragma unroll
                for (int t = 0; t < N; ++t) {
                    float acc = e[0][t] * fr[0];
#pragma unroll
                    for (int ii = 1; ii < H; ++ii) acc = __builtin_fmaf(e[ii][t], fr[ii], acc);
                    y[t] = acc;
                }
                set_issue_priority(pb + 1);
            } else {
                float an[H];
                read_rows(rowa, an);
                set_issue_priority(pb);
#pragma unroll
                for (int t = 0; t < N; ++t) y[t] = 0.f;
#pragma unroll
                for (int ii = 0; ii < H; ++ii)
#pragma unroll
                    for (int t = 0; t < N; ++t) y[t] += ex2((an[ii] + bc[t]) + L[ii][t]);
                set_issue_priority(pb + 1);
            }
#pragma unroll
            for (int t = 0; t < N; ++t) cp[partial_at(w, p, q, t)] = y[t];
            __syncthreads();
            // ---- v-update of iteration k + 1; column part of iterate k's error
            const float S = col_in ? column_total(cp, c) : 0.f;
            const float b_old = b_own;
            bool badc = false;
            if (ns > 0.f) {
                if (S >= kSumLo && S <= kSumHi)
                    b_own = b_own + lb - lg2(S);
                else
                    badc = true;
            }
            if (check) {
                const float ce = wave_sum(ns > 0.f ? fabsf(S - ns) : 0.f);
                if (lane == 0) rd[w][1] = ce;
            }
            {
                const float fl = __any(badc) ? 1.f : 0.f;
                if (lane == 0) cflag[k & 1][w] = fl;
            }
            if (c < 8 * N) colv[cslot] = b_own;
            __syncthreads();
            if (cflag[k & 1][0] + cflag[k & 1][1] != 0.f) {  // work-group-uniform, rare
                exact_cols(badc);
                if (c < 8 * N) colv[cslot] = b_own;
                __syncthreads();
            }
            if (check && (rd[0][0] + rd[0][1]) + (rd[1][0] + rd[1][1]) <= tol) {
                kstop = k;  // the returned plan is iterate k: its a and the b it was built with
                b_own = b_old;
                break;
            }
        }
    }

    // ---- the returned plan, measured (Section 4): marginal error and
    // sum_ij P_ij C_ij = -(1/s) sum_ij P_ij cl_ij, every entry rebuilt in
    // registers and never stored.
    if (c < 8 * N) colv[cslot] = b_own;
    if (rown) rowa[rslot] = a_own;
    __syncthreads();
    float err, lsum = 0.f;
    {
        float ar[H], bc[N], x[H], y[N];
        read_rows(rowa, ar);
        read_cols(bc);
#pragma unroll
        for (int t = 0; t < N; ++t) y[t] = 0.f;
#pragma unroll
        for (int ii = 0; ii < H; ++ii) {
            float xs = 0.f;
#pragma unroll
            for (int t = 0; t < N; ++t) {
                const float v = ex2((ar[ii] + bc[t]) + L[ii][t]);
                xs += v;
                y[t] += v;
                lsum = __builtin_fmaf(v, L[ii][t], lsum);
            }
            x[ii] = xs;
        }
        const float R = row_totals<H>(x, tb, p, q);
        err = ms > 0.f ? fabsf(R - ms) : 0.f;
#pragma unroll
        for (int t = 0; t < N; ++t) cp[partial_at(w, p, q, t)] = y[t];
    }
    __syncthreads();
    {
        const float S = col_in ? column_total(cp, c) : 0.f;
        err += ns > 0.f ? fabsf(S - ns) : 0.f;
    }
    err = wave_sum(err);
    lsum = wave_sum(lsum);
    if (lane == 0) {
        red[0][w][0] = err;
        red[0][w][1] = lsum;
    }
    if (row_in) A.alpha[(size_t)b * d1 + i_own] = a_own * kLn2;
    if (col_in) A.beta[(size_t)b * d2 + c] = b_own * kLn2;
    __syncthreads();
    if (threadIdx.x == 0) {
        A.loss[b] = -(red[0][0][1] + red[0][1][1]) / s;
        A.marg_err[b] = red[0][0][0] + red[0][1][0];
        A.iters[b] = kstop;
    }
}

template <int N>
__device__ __forceinline__ void resident_log_body(const FwdArgs &A, float *pool) {
    if (A.only_marked && A.iters[blockIdx.x] != -1) return;  // work-group-uniform
    if (__builtin_amdgcn_readfirstlane(threadIdx.x >> 6) == 0)
        resident_log_wave<N, 0>(A, pool);
    else
        resident_log_wave<N, 1>(A, pool);
}

// What a plain-form kernel does with a problem it cannot keep in range:
// solve it from the start in the log domain, in place (the LDS pool is free
// after the barrier), or leave it unsolved (iters = -1) when the caller pinned
// the plain-form kernel alone (SK_SELECT_PLAIN_ONLY).  Work-group-uniform.
// Problems of the widest bucket (N = 16: 128 cost registers per lane) are
// only marked (iters = -1) here, and a second launch of the log-domain kernel
// solves the marked ones: the log-domain body inlined would push the
// plain-form kernel past its registers.
template <int N>
__device__ __forceinline__ void hand_over_to_log(const FwdArgs &A, float *pool) {
    if (N > 13 || A.select == SK_SELECT_PLAIN_ONLY) {
        if (threadIdx.x == 0) A.iters[blockIdx.x] = -1;
        return;
    }
    if constexpr (N <= 13) {
        __syncthreads();
        resident_log_body<N>(A, pool);
    }
}

}  // namespace
}  // namespace sk

#endif  // SK_RESIDENT_LOG_H_
