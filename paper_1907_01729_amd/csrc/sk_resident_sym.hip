// sk_resident_sym.hip -- a symmetric cost shared by the batch, d1 = d2 <= 104
// (the label-space case: one set of points on both sides): one work-group of
// two wavefronts per problem, the plain form of eq. (sk_plain) on the vector
// ALU.
//
// With K = 2^(cl - clmax) (cl = -C log2(e)/lambda, clmax = max cl) the
// iteration is R = K V, U = mu / R, S = K^T U, V = nu / S, from u^0 = 1 on
// the support of mu: the same iterates, range guards and outputs as the
// general kernel (alpha = ln2 log2 U, beta = ln2 (log2 V - clmax)), so the
// potentials equal the log-domain iterates up to rounding.
//
// Lane l = p + 8q (p = l & 7, q = l >> 3) of wavefront w holds K[p + 8r][q + 8t]
// for its row blocks (ceil(NC / 2) from 0 for w = 0, floor(NC / 2) after
// them for w = 1) and every column block t < NC (8 NC >= d).  A product
// K w takes w "by columns"
// (register t of lane (p, q) holds w[q + 8t], read from LDS), forms per-lane
// partial row sums over t, and sums them over the 8 lanes q through a small
// per-wavefront LDS transpose: lane (p, q) writes its H partials, lane
// (p, r) reads the 8 partials of its row r and adds them, so that each row
// total ends in one lane.  The update runs on that lane only and publishes the new scaling to
// LDS for the next product; one barrier per product.  Because K is symmetric,
// K^T U is the same product as K U, so one register copy of K serves both
// passes.
//
// The kernel verifies the symmetry of the cost first, pair by pair (bit
// equality); on a cost that is not symmetric every work-group runs the
// general kernel's iteration in place (same outputs, same bits as that
// kernel), so no second launch is needed.  A problem outside the plain
// form's range gets iters = -1 (the log-domain kernel takes it): a cost
// spread wider than the range at the start, or a guard that failed in any
// iteration (checked once, at the end): a sum R_i, S_j outside
// [2^-64, 2^64] or a scaling U_i, V_j outside [2^-100, 2^100] on the supports.
#include "sk_resident_log.h"  // the general iteration, the range guards

namespace sk {
namespace {

// (K w) of the lane's row for the column-layout w (NR row blocks).
template <int NR, int NC>
__device__ __forceinline__ float kmul(const float (&K)[NR][NC], const float (&wc)[NC], float *tb, int p, int q) {
    // The two wavefronts sharing a SIMD belong to different problems: the
    // FMAs run at the lowest issue priority and the rest of the iteration
    // (the transpose, the update, the exchange) at the highest, so that one
    // problem's serial stretch is not queued behind the other's FMAs.
    __builtin_amdgcn_s_setprio(0);
    float x[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) x[r] = K[r][0] * wc[0];
#pragma unroll
    for (int t = 1; t < NC; ++t)
#pragma unroll
        for (int r = 0; r < NR; ++r) x[r] = __builtin_fmaf(K[r][t], wc[t], x[r]);
    __builtin_amdgcn_s_setprio(3);
    return row_totals<NR>(x, tb, p, q);
}

// Buffer descriptor over the d x d cost (reads past its end return 0): a
// lane's column is the register offset, the row a scalar offset.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t cost_rsrc(const float *C, int d) {
    return __builtin_amdgcn_make_buffer_rsrc((void *)C, (short)0, 4 * d * d, 0x00020000);
}

// Column operand in LDS, by column block: row y at [y & 7][y >> 3], so that
// lane (p, q) reads its NC values contiguously (16-byte reads; a stride of
// 20 floats puts the 8 blocks q on distinct banks).
constexpr int XS = 20;
// Set-up staging of the cost: row stride LDC = 8 mod 64, so that row reads
// (p, q + 8t) and transposed reads (q, p + 8a) hit 64 banks.
constexpr int LDC = 136;
// One LDS pool, also the general iteration's when the cost proves not
// symmetric (the two never run at once): float offsets, 16-byte aligned.
constexpr int oXs = 0, oTsum = oXs + 2 * 8 * XS, oCst = oTsum + 2 * kRowTotalsFloats, oRed = oCst + 2 * 8 * LDC,
              oIni = oRed + 8, kSymLdsFloats = oIni + 16;
static_assert(oTsum % 4 == 0 && oCst % 4 == 0 && oRed % 4 == 0, "16-byte offsets");
constexpr int kSymPoolFloats = kSymLdsFloats > kGenLdsFloats ? (kSymLdsFloats > kLogLdsFloats ? kSymLdsFloats : kLogLdsFloats)
                                                              : (kGenLdsFloats > kLogLdsFloats ? kGenLdsFloats : kLogLdsFloats);

// Work-group = one problem, two wavefronts: wavefront W holds H row blocks
// from R0 on (ceil(NC / 2) for the first, floor(NC / 2) for the second, so no
// block lies past the problem) against every column block, so each computes
// whole row sums of its rows; the updated scalings meet in LDS (one barrier
// per product).  Two wavefronts per problem put two per SIMD for a batch of
// one problem per SIMD: a single wavefront issues a vector instruction only
// every few cycles, two interleave.  The two wavefronts run separate
// instantiations (W = 0, 1) of this body, which pass the same barriers.
// Returns, the same on both wavefronts: kSymAsym after a barrier that frees
// the LDS pool when the cost is not symmetric (nothing written);
// kSymHandOver when the problem leaves the plain form's range (nothing
// written); kSymDone otherwise.
constexpr int kSymDone = 0, kSymAsym = 1, kSymHandOver = 2;

template <int NC, int W>
__device__ __forceinline__ int sym_body(const FwdArgs &A, float *pool) {
    constexpr int H = W == 0 ? (NC + 1) / 2 : NC / 2;
    constexpr int R0 = W == 0 ? 0 : (NC + 1) / 2;
    static_assert(R0 + H <= XS, "row blocks per column-block line");
    float(&xs)[2][8 * XS] = lds_at<float[2][8 * XS]>(pool, oXs);  // xs[0] = U, xs[1] = V
    // Per-wavefront error reports of the stop test: [iteration parity]
    // [wavefront][row phase, column phase], one 16-byte read per decision.
    // The parity keeps a report readable until both wavefronts have passed
    // the next iteration's barriers.
    float(&red)[2][2][2] = lds_at<float[2][2][2]>(pool, oRed);
    float(&ini)[2][2][4] = lds_at<float[2][2][4]>(pool, oIni);  // set-up exchanges
    float(&tsum)[2][kRowTotalsFloats] = lds_at<float[2][kRowTotalsFloats]>(pool, oTsum);  // per-wavefront row-total scratch
    float(&cst)[2][8 * LDC] = lds_at<float[2][8 * LDC]>(pool, oCst);

    const int lane = threadIdx.x & 63;
    constexpr int w = W;
    const int p = lane & 7, q = lane >> 3;
    const int b = blockIdx.x;
    const int d = A.d1;
    const float s = A.s;
    constexpr int r0 = R0;  // first row block of this wavefront

    // Raw cost cells of the wavefront's row blocks and the symmetry check, the
    // cost streamed through LDS one row block (8 rows) at a time: thread tau
    // stages column tau of the block (coalesced loads, 0 past d), the
    // wavefront owning the block takes its cells from it, and every pair
    // {(x, y), (y, x)} is compared when the later of its two row blocks is
    // staged, by the owner of the earlier one (whose cells are all loaded by
    // then).  Cells off the problem are masked (row block r holds a row iff
    // r < rlim, column block t a column iff t < tlim).
    const int rlim = (d - p + 7) >> 3, tlim = (d - q + 7) >> 3;
    constexpr int PF = NC < 4 ? NC : 4;  // row blocks in flight
    const int tau = threadIdx.x;
    const __amdgpu_buffer_rsrc_t whole = cost_rsrc(A.C, d);
    // Stream row blocks 0 .. NC-1 through LDS (PF in flight, one barrier per
    // block) and hand each staged block to visit(c, block).  Block c goes
    // into buffer c & 1, whose previous block was read before the last
    // barrier; rows and columns past d are staged as 0.
    auto stream_blocks = [&](auto &&visit) {
        float pf[PF][8];
        auto load_block = [&](int c, float(&v)[8]) {
#pragma unroll
            for (int rr = 0; rr < 8; ++rr)
                v[rr] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(whole, tau * 4, (8 * c + rr) * d * 4, 0));
        };
#pragma unroll
        for (int c = 0; c < PF; ++c) load_block(c, pf[c]);
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            if (tau < 8 * NC)
#pragma unroll
                for (int rr = 0; rr < 8; ++rr) cst[c & 1][rr * LDC + tau] = tau < d ? pf[c % PF][rr] : 0.f;
            if (c + PF < NC) load_block(c + PF, pf[c % PF]);
            __syncthreads();
            visit(c, static_cast<const float *>(cst[c & 1]));
        }
    };
    float K[H][NC];
    bool asym = false;
    stream_blocks([&](int c, const float *ch) {
        bool ne = false;
        if (c >= R0 && c < R0 + H)
#pragma unroll
            for (int t = 0; t < NC; ++t) K[c - R0][t] = ch[p * LDC + q + 8 * t];
#pragma unroll
        for (int a = R0; a < R0 + H; ++a)
            if (a <= c) ne |= (a < rlim) & (__float_as_uint(ch[q * LDC + p + 8 * a]) != __float_as_uint(K[a - R0][c]));
        asym |= (c < tlim) & ne;
    });
    float mx = neg_inf(), mn = __builtin_inff();
    bool nan = false;
#pragma unroll
    for (int i = 0; i < H; ++i) {
        float rmx = neg_inf(), rmn = __builtin_inff();
        bool rnan = false;
#pragma unroll
        for (int t = 0; t < NC; ++t) {
            const bool in = t < tlim;
            rmx = fmaxf(rmx, in ? K[i][t] : neg_inf());
            rmn = fminf(rmn, in ? K[i][t] : __builtin_inff());
            rnan |= in & (K[i][t] != K[i][t]);
        }
        const bool in = r0 + i < rlim;
        mx = fmaxf(mx, in ? rmx : neg_inf());
        mn = fminf(mn, in ? rmn : __builtin_inff());
        nan |= in & rnan;
    }
    // (Wavefront-wide votes and reductions are taken by every lane, before
    // lane 0 publishes them.)
    mx = wave_max(mx);
    mn = -wave_max(-mn);
    const float fasym = __any(asym) ? 1.f : 0.f, fnan = __any(nan) ? 1.f : 0.f;
    if (lane == 0) {
        ini[0][w][0] = fasym;
        ini[0][w][1] = fnan;
        ini[0][w][2] = mn;
        ini[0][w][3] = mx;
    }
    __syncthreads();
    if (ini[0][0][0] + ini[0][1][0] != 0.f) {  // the same verdict for every problem: the cost is shared
        __syncthreads();  // every thread has read the verdict: the pool is free
        return kSymAsym;
    }
    // Raw cost range -> cl range (cl = -s C with s > 0: the extremes swap).
    const float clmax = -s * fminf(ini[0][0][2], ini[0][1][2]);
    const float clmin = -s * fmaxf(ini[0][0][3], ini[0][1][3]);
    if (ini[0][0][1] + ini[0][1][1] != 0.f || !(clmax - clmin <= kRangeBits)) {  // a non-finite cost fails too
        return kSymHandOver;
    }
    // K on the cells of the problem; elsewhere a finite value in (0, 1]
    // (the clamp), which meets only zero operands and unused rows.
#pragma unroll
    for (int i = 0; i < H; ++i)
#pragma unroll
        for (int t = 0; t < NC; ++t) K[i][t] = ex2(fminf(-s * K[i][t] - clmax, 0.f));

    // The lane's row: x = p + 8 (r0 + q) for q < H (the row whose total the
    // lane receives), none for the other lanes.  Marginals are 0 off the
    // problem.
    const bool own = q < H;
    const int x = own ? p + 8 * (r0 + q) : 0;
    const int xl = p * XS + r0 + q;  // its place in the LDS operand
    const float ms = own && x < d ? A.mu[(size_t)b * d + x] : 0.f;
    const float ns = own && x < d ? A.nu[(size_t)b * d + x] : 0.f;
    {
        const float cm = wave_sum(ms > 0.f ? 1.f : 0.f), cn = wave_sum(ns > 0.f ? 1.f : 0.f);
        if (lane == 0) {
            ini[1][w][0] = cm;
            ini[1][w][1] = cn;
        }
    }
    // Column operand of the first product: u^0 = 1 on the support of mu.
    if (own) xs[0][xl] = ms > 0.f ? 1.f : 0.f;
    __syncthreads();
    if (ini[1][0][0] + ini[1][1][0] == 0.f || ini[1][0][1] + ini[1][1][1] == 0.f) {  // empty support
        return kSymHandOver;
    }

    const int n_iter = A.n_iter;
    const float tol = A.tol;
    const bool check = tol > 0.f;
    int kstop = n_iter;
    float U = 0.f, V, Vold = 0.f, X, wc[NC];
    float *const tb = tsum[w];

    // Column layout from LDS: register t of lane (p, q) takes row q + 8t.
    auto gather_lds = [&](const float *src) {
        const float *line = src + q * XS;
#pragma unroll
        for (int t = 0; t + 4 <= NC; t += 4) {
            const float4 v4 = *reinterpret_cast<const float4 *>(line + t);
            wc[t] = v4.x;
            wc[t + 1] = v4.y;
            wc[t + 2] = v4.z;
            wc[t + 3] = v4.w;
        }
#pragma unroll
        for (int t = NC & ~3; t < NC; ++t) wc[t] = line[t];
    };
    // A scaling out of range (or a sum that would push one there) marks the
    // problem for the log-domain kernel.  The mark is kept per lane and
    // exchanged once, after the loop: iterating on after a failure costs
    // time but cannot trap, and a failed problem's outputs are never written.
    bool bad_acc = false;

    // v-update of iteration 1.
    gather_lds(xs[0]);
    X = kmul<H, NC>(K, wc, tb, p, q);
    {
        const float v = ns * __builtin_amdgcn_rcpf(X);
        bad_acc |= (ns > 0.f) & !(sum_ok(X) & scale_ok(v));
        V = ns > 0.f ? v : 0.f;
        if (own) xs[1][xl] = V;
    }
    __syncthreads();
    gather_lds(xs[1]);

    // Iteration k: R = K V and the u-update; then (k < n_iter) S = K^T U = K U,
    // the v-update of k+1 and the stop test of iterate k (its row error from
    // the u-update, its column error from S and the V it was built with).
    // The next product's operand is read before that test, which only
    // discards it.
    for (int k = 1; k <= n_iter; ++k) {
        float(&rd)[2][2] = red[k & 1];
        X = kmul<H, NC>(K, wc, tb, p, q);
        {
            const float u = ms * __builtin_amdgcn_rcpf(X);
            bad_acc |= (ms > 0.f) & !(sum_ok(X) & scale_ok(u));
            U = ms > 0.f ? u : 0.f;
            if (own) xs[0][xl] = U;
            if (check) {
                const float e = wave_sum(ms > 0.f ? fabsf(u * X - ms) : 0.f);
                if (lane == 0) rd[w][0] = e;
            }
        }
        __syncthreads();
        if (k == n_iter) break;

        gather_lds(xs[0]);
        X = kmul<H, NC>(K, wc, tb, p, q);
        {
            const float v = ns * __builtin_amdgcn_rcpf(X);
            bad_acc |= (ns > 0.f) & !(sum_ok(X) & scale_ok(v));
            if (check) {
                const float e = wave_sum(ns > 0.f ? fabsf(V * X - ns) : 0.f);
                if (lane == 0) rd[w][1] = e;
            }
            Vold = V;
            V = ns > 0.f ? v : 0.f;
            if (own) xs[1][xl] = V;
        }
        __syncthreads();
        gather_lds(xs[1]);
        if (check) {
            const float4 e4 = *reinterpret_cast<const float4 *>(&rd[0][0]);
            if ((e4.x + e4.y) + (e4.z + e4.w) <= tol) {
                kstop = k;  // the returned plan is iterate k: U and the V it was built with
                V = Vold;
                break;
            }
        }
    }
    {
        const float fb = __any(bad_acc) ? 1.f : 0.f;
        if (lane == 0) ini[0][w][0] = fb;
    }

    // ---- the returned plan P = U K V, measured (Section 4): its marginals
    // and sum_ij P_ij C_ij from the cost itself.  Past the loop's last
    // barrier a wavefront reads the operand buffers only for a gather whose
    // values it drops (a stop), so rewriting V here is safe. ----
    if (own) xs[1][xl] = V;
    __syncthreads();
    if (ini[0][0][0] + ini[0][1][0] != 0.f) {
        return kSymHandOver;
    }
    gather_lds(xs[1]);
    X = kmul<H, NC>(K, wc, tb, p, q);  // row sums R = K V
    float err = ms > 0.f ? fabsf(U * X - ms) : 0.f, lsum;
    {
        // L_i = sum_j K_ij V_j C_ij with the cost recovered from K itself:
        // on the cells of the problem log2 K = cl - clmax (the spread guard
        // keeps K >= 2^-64), so L_i = -(sum_j K_ij V_j log2 K_ij + clmax R_i) / s
        // -- no second read of the cost.  Cells off the problem meet V = 0
        // (the select keeps a K of 0 from turning 0 * log2 0 into NaN).
        float l[H];
#pragma unroll
        for (int i = 0; i < H; ++i) {
            float acc = 0.f;
#pragma unroll
            for (int t = 0; t < NC; ++t) {
                const float kv = K[i][t] * wc[t];
                acc = __builtin_fmaf(kv, kv > 0.f ? lg2(K[i][t]) : 0.f, acc);
            }
            l[i] = acc;
        }
        const float ls = row_totals<H>(l, tb, p, q);
        lsum = ms > 0.f ? U * (-__builtin_fmaf(clmax, X, ls) / s) : 0.f;
    }
    gather_lds(xs[0]);
    X = kmul<H, NC>(K, wc, tb, p, q);  // column sums S = K^T U
    err += ns > 0.f ? fabsf(V * X - ns) : 0.f;
    err = wave_sum(err);
    lsum = wave_sum(lsum);
    if (lane == 0) {
        red[0][w][0] = err;
        red[0][w][1] = lsum;
    }
    if (own && x < d) {
        A.alpha[(size_t)b * d + x] = kLn2 * lg2(U);
        A.beta[(size_t)b * d + x] = kLn2 * (lg2(V) - clmax);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        A.loss[b] = red[0][0][1] + red[0][1][1];
        A.marg_err[b] = red[0][0][0] + red[0][1][0];
        A.iters[b] = kstop;
    }
    return kSymDone;
}

template <int NC>
__global__ __launch_bounds__(128) void sk_resident_sym_kernel(FwdArgs A) {
    __shared__ __attribute__((aligned(16))) float pool[kSymPoolFloats];
    int r = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) == 0 ? sym_body<NC, 0>(A, pool)
                                                                   : sym_body<NC, 1>(A, pool);
    // the general iteration in place (its own reads of the cost)
    if (r == kSymAsym) r = resident_gen_body<NC>(A, pool) ? kSymHandOver : kSymDone;
    if (r == kSymHandOver) hand_over_to_log<NC>(A, pool);
}

template <int NC>
hipError_t launch_nc(const FwdArgs &a, hipStream_t st) {
    hipLaunchKernelGGL((sk_resident_sym_kernel<NC>), dim3(a.B), dim3(128), 0, st, a);
    return hipGetLastError();
}

}  // namespace

bool launch_resident_sym(const FwdArgs &a, hipStream_t st, hipError_t *err) {
    if (a.n_iter <= 0 || a.c_batched || a.d1 != a.d2) return false;
    const int nc = (a.d1 + 7) / 8;
    if (nc <= 2) *err = launch_nc<2>(a, st);
    else if (nc <= 4) *err = launch_nc<4>(a, st);
    else if (nc <= 8) *err = launch_nc<8>(a, st);
    else if (nc <= 13) *err = launch_nc<13>(a, st);
    else return false;
    return true;
}

}  // namespace sk
