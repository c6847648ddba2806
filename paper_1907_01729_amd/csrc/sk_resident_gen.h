// sk_resident_gen.h -- the general plain-form iteration of one problem by one
// work-group of two wavefronts, as a device function: the body of
// sk_resident_gen_kernel, and what the symmetric-cost kernel runs in place
// when it finds the shared cost not symmetric.
//
// Any cost (shared by the batch or one per problem)
// with max(d1, d2) <= 128: one work-group of two wavefronts per problem, the
// plain form of eq. (sk_plain) on the vector ALU, the kernel matrix in VGPRs.
//
// With K = 2^(cl - clmax) (cl = -C log2(e)/lambda, clmax = max cl over the
// problem) the iteration is R = K V, U = mu / R, S = K^T U, V = nu / S, from
// u^0 = 1 on the support of mu, with the range guards of the symmetric
// kernel: a cost spread over more than 64 bits, or a sum R_i, S_j outside
// [2^-64, 2^64] or a scaling outside [2^-100, 2^100] on the supports in any
// iteration, hands the problem to the log-domain iteration (the guard flags
// are kept per lane and exchanged once, after the loop).
// Outputs alpha = ln2 log2 U, beta = ln2 (log2 V - clmax): the potentials of
// the log-domain iterates up to rounding.
//
// Lane (p, q) of wavefront w holds K[p + 8r][q + 8t] for its row blocks r in
// [w H, w H + H) (H = ceil(N / 2)) and every column block t < N (8 N >=
// max(d1, d2)).  R = K V takes V by columns (lane (p, q) reads V[q + 8t]) and
// sums its row partials over the lanes q through the per-wavefront LDS
// transpose, so row i ends on one lane (p, q < H); S = K^T U takes U by rows
// and sums its column partials over the lanes p and the two wavefronts
// through LDS, so column j ends on thread j.  U lives on the row lanes, V on
// the column threads; each is published to LDS for the next product.  The
// U a lane needs comes only from its own wavefront (the rows it holds), so
// publishing U needs no barrier (a wavefront's LDS operations complete in
// order); two barriers per iteration: column partials written, V published.
#ifndef SK_RESIDENT_GEN_H_
#define SK_RESIDENT_GEN_H_

#include "sk_device.h"
#include "sk_internal.h"

namespace sk {
namespace {

constexpr float kLo = 5.42101086242752217e-20f;   // 2^-64
constexpr float kHi = 1.84467440737095516e19f;    // 2^64
constexpr float kSMin = 7.8886090522101181e-31f;  // 2^-100
constexpr float kSMax = 1.2676506002282294e30f;   // 2^100
constexpr float kRangeBits = 64.f;
constexpr int kVS = 20;  // LDS line stride of the published vectors (16-byte reads, 8 lines on distinct banks)

__device__ __forceinline__ bool sum_ok(float x) { return x >= kLo && x <= kHi; }
__device__ __forceinline__ bool scale_ok(float x) { return x >= kSMin && x <= kSMax; }

// Buffer descriptor over the d1 x d2 cost from row `row` on (reads past its
// end return 0), so that a lane's byte offset is one register for every row
// block and the column block an immediate.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const float *C, int d1, int d2, int row) {
    const int rest = (d1 - row) * d2;
    return __builtin_amdgcn_make_buffer_rsrc((void *)(C + (size_t)row * d2), (short)0, rest > 0 ? 4 * rest : 0,
                                             0x00020000);
}
__device__ __forceinline__ float load_cell(__amdgpu_buffer_rsrc_t rsrc, int byte_off) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rsrc, byte_off, 0, 0));
}

// A typed LDS array at a float offset into a work-group's pool, so that
// kernels whose phases never overlap can share one allocation.
template <class T>
__device__ __forceinline__ T &lds_at(float *pool, int off) {
    return *reinterpret_cast<T *>(pool + off);
}

// LDS of the general iteration: float offsets into its pool (16-byte
// aligned where 16-byte accesses are made).
constexpr int kGenColv = 0;
constexpr int kGenRowv = kGenColv + 8 * kVS;
constexpr int kGenCp = kGenRowv + 8 * kVS;
constexpr int kGenTsum = kGenCp + kColumnPartialsFloats;
constexpr int kGenRed = kGenTsum + 2 * kRowTotalsFloats;
constexpr int kGenIni = kGenRed + 8;
constexpr int kGenLdsFloats = kGenIni + 8;
static_assert(kGenRowv % 4 == 0 && kGenCp % 4 == 0 && kGenTsum % 4 == 0 && kGenRed % 4 == 0, "16-byte offsets");

// One problem (b = blockIdx.x) per work-group of 128 threads.  Every
// thread of the work-group calls it, from wavefront-uniform control flow;
// pool: kGenLdsFloats floats of LDS, 16-byte aligned, contents irrelevant.
// Returns true (on every thread, nothing written) when the problem leaves the
// plain form's range: the caller then solves it in the log domain.
template <int N>
__device__ __forceinline__ bool resident_gen_body(const FwdArgs &A, float *pool) {
    constexpr int H = (N + 1) / 2;
    static_assert(8 * N <= 128 && H <= 8, "one thread per column, one lane per row");
    // V[j] at colv[(j & 7) * kVS + (j >> 3)] (lane (p, q) reads line q);
    // U[p + 8 (w H + r)] at rowv[p * kVS + 8 w + r] (wavefront w's lanes p read line p from entry 8w).
    float(&colv)[8 * kVS] = lds_at<float[8 * kVS]>(pool, kGenColv);
    float(&rowv)[8 * kVS] = lds_at<float[8 * kVS]>(pool, kGenRowv);
    float(&cp)[kColumnPartialsFloats] = lds_at<float[kColumnPartialsFloats]>(pool, kGenCp);
    float(&tsum)[2][kRowTotalsFloats] = lds_at<float[2][kRowTotalsFloats]>(pool, kGenTsum);
    // Stop-test reports [iteration parity][wavefront][row error, column
    // error]: the parity keeps a report readable until both wavefronts have
    // passed the next iteration's barriers.
    float(&red)[2][2][2] = lds_at<float[2][2][2]>(pool, kGenRed);
    float(&ini)[2][4] = lds_at<float[2][4]>(pool, kGenIni);  // set-up exchanges, then the guard flags

    const int b = blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int p = lane & 7, q = lane >> 3;
    const int d1 = A.d1, d2 = A.d2;
    const float s = A.s;
    const float *Cb = A.C + (A.c_batched ? (size_t)b * d1 * d2 : 0);
    float *const tb = tsum[w];

    // Raw cost cells of the lane and their range.  Rows past d1 read 0,
    // columns past d2 the next row's cells; every such cell is masked (row
    // block r holds a row of the problem iff r < rlim, column block t a
    // column iff t < tlim).
    const int voff = (p * d2 + q) * 4;
    const int rlim = (d1 - p + 7) >> 3, tlim = (d2 - q + 7) >> 3;
    float K[H][N];
#pragma unroll
    for (int ii = 0; ii < H; ++ii) {
        const __amdgpu_buffer_rsrc_t rs = rows_rsrc(Cb, d1, d2, 8 * (w * H + ii));
#pragma unroll
        for (int t = 0; t < N; ++t) K[ii][t] = load_cell(rs, voff + 32 * t);
    }
    float mx = neg_inf(), mn = __builtin_inff();
    bool nan = false;
#pragma unroll
    for (int ii = 0; ii < H; ++ii) {
        float rmx = neg_inf(), rmn = __builtin_inff();
        bool rnan = false;
#pragma unroll
        for (int t = 0; t < N; ++t) {
            const bool in = t < tlim;
            rmx = fmaxf(rmx, in ? K[ii][t] : neg_inf());
            rmn = fminf(rmn, in ? K[ii][t] : __builtin_inff());
            rnan |= in & (K[ii][t] != K[ii][t]);
        }
        const bool in = w * H + ii < rlim;
        mx = fmaxf(mx, in ? rmx : neg_inf());
        mn = fminf(mn, in ? rmn : __builtin_inff());
        nan |= in & rnan;
    }
    mx = wave_max(mx);
    mn = -wave_max(-mn);
    const float fnan = __any(nan) ? 1.f : 0.f;
    if (lane == 0) {
        ini[w][0] = fnan;
        ini[w][1] = mn;
        ini[w][2] = mx;
    }
    __syncthreads();
    // Raw cost range -> cl range (cl = -s C with s > 0: the extremes swap).
    const float clmax = -s * fminf(ini[0][1], ini[1][1]);
    const float clmin = -s * fmaxf(ini[0][2], ini[1][2]);
    if (ini[0][0] + ini[1][0] != 0.f || !(clmax - clmin <= kRangeBits)) {  // a non-finite cost fails too
        return true;
    }
    // K on the cells of the problem, 0 elsewhere.
#pragma unroll
    for (int ii = 0; ii < H; ++ii)
#pragma unroll
        for (int t = 0; t < N; ++t)
            K[ii][t] = ((w * H + ii < rlim) && (t < tlim)) ? ex2(fminf(-s * K[ii][t] - clmax, 0.f)) : 0.f;

    // Owners: lane (p, q < H) owns row i = p + 8 (w H + q); thread c owns
    // column c.  Marginals are 0 off the problem.
    const bool rown = q < H;
    const int i_own = p + 8 * (w * H + q);
    const bool row_in = rown && i_own < d1;
    const int c = threadIdx.x;
    const bool col_in = c < d2;
    const float ms = row_in ? A.mu[(size_t)b * d1 + i_own] : 0.f;
    const float ns = col_in ? A.nu[(size_t)b * d2 + c] : 0.f;
    const int rslot = p * kVS + 8 * w + q;               // U of the lane's row in rowv
    const int cslot = (c & 7) * kVS + (c >> 3);          // V of the thread's column in colv
    {
        const float cm = wave_sum(ms > 0.f ? 1.f : 0.f), cn = wave_sum(ns > 0.f ? 1.f : 0.f);
        if (lane == 0) {
            ini[w][3] = cm;
            red[0][w][0] = cn;
        }
    }
    // Column operand of the first product: u^0 = 1 on the support of mu.
    if (rown) rowv[rslot] = ms > 0.f ? 1.f : 0.f;
    __syncthreads();
    if (ini[0][3] + ini[1][3] == 0.f || red[0][0][0] + red[0][1][0] == 0.f) {  // empty support
        return true;
    }

    // The FMAs of both products run at the lowest issue priority and the rest
    // of the iteration at the highest: the wavefronts sharing a SIMD belong
    // to different problems, and one problem's serial stretch (transposes,
    // updates, exchanges) should not queue behind another's FMAs.
    // (K w)_i of the lane's row, w published by columns.
    auto row_product = [&]() -> float {
        float wc[N];
#pragma unroll
        for (int t = 0; t < N; ++t) wc[t] = colv[q * kVS + t];
        __builtin_amdgcn_s_setprio(0);
        float x[H];
#pragma unroll
        for (int ii = 0; ii < H; ++ii) x[ii] = K[ii][0] * wc[0];
#pragma unroll
        for (int t = 1; t < N; ++t)
#pragma unroll
            for (int ii = 0; ii < H; ++ii) x[ii] = __builtin_fmaf(K[ii][t], wc[t], x[ii]);
        __builtin_amdgcn_s_setprio(3);
        return row_totals<H>(x, tb, p, q);
    };
    // Column partials of K^T u, u published by rows by this wavefront's own
    // lanes (column_total after a barrier).
    auto column_product = [&]() {
        __builtin_amdgcn_wave_barrier();
        float wr[H];
#pragma unroll
        for (int ii = 0; ii < H; ++ii) wr[ii] = rowv[p * kVS + 8 * w + ii];
        __builtin_amdgcn_s_setprio(0);
#pragma unroll
        for (int t = 0; t < N; ++t) {
            float y = K[0][t] * wr[0];
#pragma unroll
            for (int ii = 1; ii < H; ++ii) y = __builtin_fmaf(K[ii][t], wr[ii], y);
            cp[partial_at(w, p, q, t)] = y;
        }
        __builtin_amdgcn_s_setprio(3);
    };

    const int n_iter = A.n_iter;
    const float tol = A.tol;
    const bool check = tol > 0.f;
    int kstop = n_iter;
    float U = 0.f, V = 0.f, Vold = 0.f;
    bool bad_acc = false;

    // v-update of iteration 1.
    column_product();
    __syncthreads();
    {
        const float S = col_in ? column_total(cp, c) : 0.f;
        const float v = ns * __builtin_amdgcn_rcpf(S);
        bad_acc |= (ns > 0.f) & !(sum_ok(S) & scale_ok(v));
        V = ns > 0.f ? v : 0.f;
        if (c < 8 * N) colv[cslot] = V;
    }
    __syncthreads();

    // Iteration k: R = K V and the u-update; then (k < n_iter) S = K^T U,
    // the v-update of k+1 and the stop test of iterate k (its row error from
    // the u-update, its column error from S and the V it was built with).
    for (int k = 1; k <= n_iter; ++k) {
        float(&rd)[2][2] = red[k & 1];
        const float R = row_product();
        {
            const float u = ms * __builtin_amdgcn_rcpf(R);
            bad_acc |= (ms > 0.f) & !(sum_ok(R) & scale_ok(u));
            U = ms > 0.f ? u : 0.f;
            if (rown) rowv[rslot] = U;
            if (check) {
                const float e = wave_sum(ms > 0.f ? fabsf(u * R - ms) : 0.f);
                if (lane == 0) rd[w][0] = e;
            }
        }
        if (k == n_iter) break;

        column_product();
        __syncthreads();
        {
            const float S = col_in ? column_total(cp, c) : 0.f;
            const float v = ns * __builtin_amdgcn_rcpf(S);
            bad_acc |= (ns > 0.f) & !(sum_ok(S) & scale_ok(v));
            if (check) {
                const float e = wave_sum(ns > 0.f ? fabsf(V * S - ns) : 0.f);
                if (lane == 0) rd[w][1] = e;
            }
            Vold = V;
            V = ns > 0.f ? v : 0.f;
            if (c < 8 * N) colv[cslot] = V;
        }
        __syncthreads();
        if (check && (rd[0][0] + rd[0][1]) + (rd[1][0] + rd[1][1]) <= tol) {
            kstop = k;  // the returned plan is iterate k: U and the V it was built with
            V = Vold;
            break;
        }
    }
    {
        const float fb = __any(bad_acc) ? 1.f : 0.f;
        if (lane == 0) ini[w][0] = fb;
    }

    // ---- the returned plan P = U K V, measured (Section 4): its marginals
    // and sum_ij P_ij C_ij from the cost itself.  colv holds the returned V
    // unless the loop stopped early (then nothing has read it since the
    // loop's last barrier). ----
    if (kstop != n_iter && c < 8 * N) colv[cslot] = V;
    __syncthreads();
    if (ini[0][0] + ini[1][0] != 0.f) {
        return true;
    }
    float err, lsum;
    {
        float wc[N];
#pragma unroll
        for (int t = 0; t < N; ++t) wc[t] = colv[q * kVS + t];
        // L_i = sum_j K_ij V_j C_ij with the cost recovered from K itself:
        // on the cells of the problem log2 K = cl - clmax (the spread guard
        // keeps K >= 2^-64), so L_i = -(sum_j K_ij V_j log2 K_ij + clmax R_i) / s
        // -- no second read of the cost.  K is 0 off the problem (the select
        // keeps 0 * log2 0 from becoming NaN).
        float x[H], l[H];
#pragma unroll
        for (int ii = 0; ii < H; ++ii) {
            float xs = 0.f, ls = 0.f;
#pragma unroll
            for (int t = 0; t < N; ++t) {
                const float kv = K[ii][t] * wc[t];
                xs += kv;
                ls = __builtin_fmaf(kv, kv > 0.f ? lg2(K[ii][t]) : 0.f, ls);
            }
            x[ii] = xs;
            l[ii] = ls;
        }
        const float R = row_totals<H>(x, tb, p, q);
        const float L = -__builtin_fmaf(clmax, R, row_totals<H>(l, tb, p, q)) / s;
        err = ms > 0.f ? fabsf(U * R - ms) : 0.f;
        lsum = ms > 0.f ? U * L : 0.f;
    }
    column_product();  // rowv still holds the returned U
    __syncthreads();
    {
        const float S = col_in ? column_total(cp, c) : 0.f;
        err += ns > 0.f ? fabsf(V * S - ns) : 0.f;
    }
    err = wave_sum(err);
    lsum = wave_sum(lsum);
    if (lane == 0) {
        red[0][w][0] = err;
        red[0][w][1] = lsum;
    }
    if (row_in) A.alpha[(size_t)b * d1 + i_own] = kLn2 * lg2(U);
    if (col_in) A.beta[(size_t)b * d2 + c] = kLn2 * (lg2(V) - clmax);
    __syncthreads();
    if (threadIdx.x == 0) {
        A.loss[b] = red[0][0][1] + red[0][1][1];
        A.marg_err[b] = red[0][0][0] + red[0][1][0];
        A.iters[b] = kstop;
    }
    return false;
}

}  // namespace
}  // namespace sk

#endif  // SK_RESIDENT_GEN_H_
