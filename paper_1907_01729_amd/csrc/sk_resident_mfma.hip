// sk_resident_mfma.hip -- a cost shared by the batch (Section 4), max(d1, d2) <= 128:
// the two matrix products of every iteration on the matrix cores.
//
// With one cost for all problems, the iteration of eq. (sk_plain) over a
// group of problems is a pair of matrix products with the same kernel matrix:
//   R = K V   (d1 x G),   U = mu / R,      S = K^T U   (d2 x G),   V = nu / S,
// where column n of U, V holds problem n of the group.  Here K = 2^(cl - clmax)
// with cl = -C log2(e)/lambda, clmax = max cl.  Potentials come back in the
// log form the other kernels use: starting from u = 1 on the support of mu
// (a^0 = -clmax instead of 0, a constant gauge shift that the same map carries
// through every iterate), alpha_i = ln2 log2 U_i and beta_j = ln2 (log2 V_j - clmax),
// so that P_ij = U_i K_ij V_j = exp(alpha_i + beta_j - C_ij/lambda) and both
// potentials equal the log-domain iterates exactly (up to rounding).
//
// Range: the plain form is taken only when max cl - min cl <= 64 bits, and a
// problem is handed to the log-domain kernel (iters = -1, launched next on the
// same stream) as soon as one of its sums R_i, S_j leaves [2^-64, 2^64] or a
// scaling U_i, V_j leaves [2^-100, 2^100] on the supports.  Inside those
// bounds nothing overflows and every product that underflows (< 2^-126) is
// below 2^-55 of the sum it drops out of.
//
// Work-group = 4 problems (n = lane & 3), 4 wavefronts on the CU's 4 SIMDs.
// v_mfma_f32_4x4x1_16b_f32 multiplies 16 blocks of (4 x 1) by (1 x 4): with
// the blocks stacked along the rows, one instruction is a rank-1 update of a
// 64-row slab of R (or S) for the 4 problems.  Wavefront w contracts over its
// quarter of the inner index, [w JI, w JI + JI), with its slice of K held in
// VGPRs as A operands (lane l = row l of the slab):
//   GEMM1: A1[h][jj] = K[l + 64h, w JI + jj],  B = V[w JI + jj, n]
//   GEMM2: A2[h][ii] = K[w JI + ii, l + 64h],  B = U[w JI + ii, n]
// The four partial products meet in LDS; after a barrier wavefront w sums
// the rows (then the columns) of its own quarter, updates U (V) there, and
// feeds them back as its own B operands: two barriers per iteration, no other
// traffic.  Output layout of the instruction: lane l, element v holds row
// 4 (l / 4) + v of the slab for problem l & 3.
#include "sk_device.h"
#include "sk_internal.h"

namespace sk {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr float kLo = 5.42101086242752217e-20f;   // 2^-64
constexpr float kHi = 1.84467440737095516e19f;    // 2^64
constexpr float kSMin = 7.8886090522101181e-31f;  // 2^-100
constexpr float kSMax = 1.2676506002282294e30f;   // 2^100
constexpr float kRangeBits = 64.f;
constexpr int kRowRor4 = 0x124;  // DPP row_ror:4

__device__ __forceinline__ bool sum_ok(float x) { return x >= kLo && x <= kHi; }
__device__ __forceinline__ bool scale_ok(float x) { return x >= kSMin && x <= kSMax; }

// Sum over the 16 lanes of one problem (same lane & 3); lanes 0..3 hold the
// totals of problems 0..3.
__device__ __forceinline__ float sum_n(float v) {
    v += dpp<kRowRor4>(v);
    v += dpp<kRowRor8>(v);
    LanePair a = swap16(v);
    v = a.lo + a.hi;
    LanePair c = swap32(v);
    return c.lo + c.hi;
}

// D[h] = sum over the wavefront's inner quarter of A[h][k] x Bsrc[k] (this
// lane's problem), two accumulator chains per slab.
template <int NH, int JI, int JP>
__device__ __forceinline__ void gemm(const float (&Aop)[NH][JI], const float *Bsrc, f4 (&D)[NH]) {
    float Bv[JP];
#pragma unroll
    for (int k = 0; k < JP; k += 4) {
        const f4 t = *reinterpret_cast<const f4 *>(Bsrc + k);
        Bv[k] = t[0];
        Bv[k + 1] = t[1];
        Bv[k + 2] = t[2];
        Bv[k + 3] = t[3];
    }
    f4 acc[NH][2];
#pragma unroll
    for (int h = 0; h < NH; ++h) acc[h][0] = acc[h][1] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < JI; ++k)
#pragma unroll
        for (int h = 0; h < NH; ++h)
            acc[h][k & 1] = __builtin_amdgcn_mfma_f32_4x4x1f32(Aop[h][k], Bv[k], acc[h][k & 1], 0, 0, 0);
#pragma unroll
    for (int h = 0; h < NH; ++h) D[h] = acc[h][0] + acc[h][1];
}

// Full sum for slot index x (row or column of the matrix, < 64 NH) of this
// lane's problem n from the four wavefronts' partials, in wavefront order.
template <int NH>
__device__ __forceinline__ float gather_partials(const f4 (*P)[NH][64], int x, int n) {
    const int h = x >> 6, xl = x & 63;
    const int src = (xl & ~3) + n, v = xl & 3;
    const float *p0 = reinterpret_cast<const float *>(&P[0][h][src]) + v;
    float s = p0[0];
#pragma unroll
    for (int w = 1; w < 4; ++w) s += reinterpret_cast<const float *>(&P[w][h][src])[v];
    return s;
}

template <int NH, int JP>
union Lds {
    struct {
        f4 P[3][4][NH][64];              // partial products [product][wavefront][slab][lane]
        __align__(16) float Vb[4][4][JP];  // [wavefront][problem][k]: B operands of GEMM1
        __align__(16) float Ub[4][4][JP];  // same for GEMM2
        float F[3][4][4][2];             // per-problem sums and flags [stage][wavefront][problem]
    } loop;
    float cl[64 * NH * 64 * NH];         // scaled cost, row-major d1 x d2
};

// Wave flag of this lane's problem n (lanes 0..3 = problems 0..3) from a
// ballot: lanes n, n + 4, ... belong to problem n.
__device__ __forceinline__ float flag_n(bool bad, int l) {
    const unsigned long long m = __ballot(bad);
    return ((m >> (l & 3)) & 0x1111111111111111ull) ? 1.f : 0.f;
}

// Problem states (per lane, for its problem n; identical on every lane of n).
constexpr int kLive = 0, kStopped = 1, kFailed = 2;

template <int NH, int JI>
__global__ __launch_bounds__(256) void sk_resident_mfma_kernel(FwdArgs A) {
    constexpr int JP = (JI + 3) & ~3;   // B-operand stride in LDS (16-byte reads)
    constexpr int NS = (JI + 15) / 16;  // update slots per lane
    static_assert(16 * NS >= JP, "update slots must cover the padded operand rows");
    // The scaled cost is staged through LDS for the set-up only; the loop's
    // buffers reuse the same bytes afterwards.
    __shared__ Lds<NH, JP> lds;
    __shared__ float red[2][4];
    auto &P = lds.loop.P;
    auto &Vb = lds.loop.Vb;
    auto &Ub = lds.loop.Ub;
    auto &F = lds.loop.F;

    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int n = l & 3;
    const int b = 4 * blockIdx.x + n;  // this lane's problem
    // only_flagged == 2: the symmetric-cost kernel ran first and handed over
    // the problems it marked with iters = -2; the others are left untouched.
    const bool real = b < A.B && (A.only_flagged != 2 || A.iters[b] == -2);
    if (A.only_flagged == 2 && !__any(real)) return;  // one verdict for the work-group: its lanes span its 4 problems
    const int d1 = A.d1, d2 = A.d2;
    const float s = A.s;
    const float *C = A.C;

    // Range of cl over the shared cost, staged in LDS on the way.
    float mx = neg_inf(), mn = __builtin_inff();
    for (int x = threadIdx.x; x < d1 * d2; x += 256) {
        const float c = -s * C[x];
        lds.cl[x] = c;
        mx = fmaxf(mx, c);
        mn = fminf(mn, c);
    }
    mx = wave_max(mx);
    mn = -wave_max(-mn);
    if (l == 0) {
        red[0][w] = mx;
        red[1][w] = mn;
    }
    __syncthreads();
    mx = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
    mn = fminf(fminf(red[1][0], red[1][1]), fminf(red[1][2], red[1][3]));
    if (!(mx - mn <= kRangeBits)) {
        if (threadIdx.x < 4 && real) A.iters[b] = -1;  // lanes 0..3 hold problems 0..3
        return;
    }
    const float clmax = mx;

    // This wavefront's slice of K as A operands.
    float A1[NH][JI], A2[NH][JI];
#pragma unroll
    for (int h = 0; h < NH; ++h)
#pragma unroll
        for (int k = 0; k < JI; ++k) {
            const int i = l + 64 * h, j = w * JI + k;
            A1[h][k] = (i < d1 && j < d2) ? ex2(lds.cl[i * d2 + j] - clmax) : 0.f;
            const int i2 = w * JI + k, j2 = l + 64 * h;
            A2[h][k] = (i2 < d1 && j2 < d2) ? ex2(lds.cl[i2 * d2 + j2] - clmax) : 0.f;
        }
    __syncthreads();  // the staged cost is dead from here on

    // Update slots: lane (n, l / 4) owns rows (and columns) x = w JI + l/4 + 16 t.
    float mu_s[NS], nu_s[NS], U_s[NS], V_s[NS], Vold_s[NS];
    int x_s[NS];
    bool in_s[NS];
    float msum = 0.f, nsum = 0.f;
#pragma unroll
    for (int t = 0; t < NS; ++t) {
        const int k = (l >> 2) + 16 * t;
        in_s[t] = k < JI;
        x_s[t] = w * JI + k;
        mu_s[t] = (real && in_s[t] && x_s[t] < d1) ? A.mu[(size_t)b * d1 + x_s[t]] : 0.f;
        nu_s[t] = (real && in_s[t] && x_s[t] < d2) ? A.nu[(size_t)b * d2 + x_s[t]] : 0.f;
        msum += mu_s[t] > 0.f ? 1.f : 0.f;
        nsum += nu_s[t] > 0.f ? 1.f : 0.f;
        U_s[t] = mu_s[t] > 0.f ? 1.f : 0.f;  // u^0 = 1 on the support of mu
        V_s[t] = Vold_s[t] = 0.f;
        if (k < JP) {  // the wavefront's own operand rows, padding included
            Ub[w][n][k] = U_s[t];
            Vb[w][n][k] = 0.f;
        }
    }

    const int n_iter = A.n_iter;
    const float tol = A.tol;
    const bool check = tol > 0.f;
    int state = real ? kLive : kStopped;
    int kstop = n_iter;
    float rowerr_prev = 0.f;
    f4 D[NH];

    // v-update of iteration 1.
    gemm<NH, JI, JP>(A2, &Ub[w][n][0], D);
#pragma unroll
    for (int h = 0; h < NH; ++h) P[1][w][h][l] = D[h];
    msum = sum_n(msum);
    nsum = sum_n(nsum);
    if (l < 4) {
        F[2][w][l][0] = msum;
        F[2][w][l][1] = nsum;
    }
    __syncthreads();
    {
        const float ms = F[2][0][n][0] + F[2][1][n][0] + F[2][2][n][0] + F[2][3][n][0];
        const float ns = F[2][0][n][1] + F[2][1][n][1] + F[2][2][n][1] + F[2][3][n][1];
        if (state == kLive && (ms == 0.f || ns == 0.f)) state = kFailed;  // empty support: log-domain kernel
        bool bad = false;
#pragma unroll
        for (int t = 0; t < NS; ++t) {
            const float S = gather_partials<NH>(P[1], x_s[t], n);
            if (nu_s[t] > 0.f) {
                V_s[t] = nu_s[t] * __builtin_amdgcn_rcpf(S);
                bad |= !(sum_ok(S) && scale_ok(V_s[t]));
            }
            if (in_s[t]) Vb[w][n][x_s[t] - w * JI] = V_s[t];
        }
        const float fb = flag_n(bad, l);
        if (l < 4) {
            F[1][w][l][0] = 0.f;
            F[1][w][l][1] = fb;
        }
    }

    for (int k = 1;; ++k) {
        // ---- GEMM1: R = K V for the 4 problems ----
        gemm<NH, JI, JP>(A1, &Vb[w][n][0], D);
#pragma unroll
        for (int h = 0; h < NH; ++h) P[0][w][h][l] = D[h];
        __syncthreads();

        // Column-stage results of the previous sweep: failures, and the stop
        // test of iterate k-1 (row part measured then, column part now).
        {
            const float cerr = check ? F[1][0][n][0] + F[1][1][n][0] + F[1][2][n][0] + F[1][3][n][0] : 0.f;
            const float cbad = F[1][0][n][1] + F[1][1][n][1] + F[1][2][n][1] + F[1][3][n][1];
            if (state == kLive) {
                if (cbad != 0.f) {
                    state = kFailed;
                } else if (check && k >= 2 && rowerr_prev + cerr <= tol) {
                    state = kStopped;
                    kstop = k - 1;
#pragma unroll
                    for (int t = 0; t < NS; ++t) V_s[t] = Vold_s[t];
                }
            }
        }
        if (!__any(state == kLive)) break;  // all four problems finished

        // ---- u-update of iteration k on this wavefront's rows ----
        float rerr = 0.f;
        bool bad = false;
#pragma unroll
        for (int t = 0; t < NS; ++t) {
            const float R = gather_partials<NH>(P[0], x_s[t], n);
            if (state == kLive && mu_s[t] > 0.f) {
                U_s[t] = mu_s[t] * __builtin_amdgcn_rcpf(R);
                bad |= !(sum_ok(R) && scale_ok(U_s[t]));
                if (check) rerr += fabsf(U_s[t] * R - mu_s[t]);
            }
            if (in_s[t]) Ub[w][n][x_s[t] - w * JI] = U_s[t];
        }
        const float fb = flag_n(bad, l);
        if (check) rerr = sum_n(rerr);
        if (l < 4) {
            F[0][w][l][0] = rerr;
            F[0][w][l][1] = fb;
        }
        if (k == n_iter) break;

        // ---- GEMM2: S = K^T U ----
        gemm<NH, JI, JP>(A2, &Ub[w][n][0], D);
#pragma unroll
        for (int h = 0; h < NH; ++h) P[1][w][h][l] = D[h];
        __syncthreads();

        {
            const float re = check ? F[0][0][n][0] + F[0][1][n][0] + F[0][2][n][0] + F[0][3][n][0] : 0.f;
            const float rb = F[0][0][n][1] + F[0][1][n][1] + F[0][2][n][1] + F[0][3][n][1];
            if (state == kLive && rb != 0.f) state = kFailed;
            rowerr_prev = re;
        }
        // ---- plan column sums of iterate k, then the v-update of iteration k+1 ----
        float cerr = 0.f;
        bad = false;
#pragma unroll
        for (int t = 0; t < NS; ++t) {
            const float S = gather_partials<NH>(P[1], x_s[t], n);
            if (state == kLive && nu_s[t] > 0.f) {
                if (check) cerr += fabsf(V_s[t] * S - nu_s[t]);
                Vold_s[t] = V_s[t];
                V_s[t] = nu_s[t] * __builtin_amdgcn_rcpf(S);
                bad |= !(sum_ok(S) && scale_ok(V_s[t]));
            }
            if (in_s[t]) Vb[w][n][x_s[t] - w * JI] = V_s[t];
        }
        const float fc = flag_n(bad, l);
        if (check) cerr = sum_n(cerr);
        if (l < 4) {
            F[1][w][l][0] = cerr;
            F[1][w][l][1] = fc;
        }
    }
    __syncthreads();
    {
        // Failures of the last u-update (harmless to re-read an older stage).
        const float rb = F[0][0][n][1] + F[0][1][n][1] + F[0][2][n][1] + F[0][3][n][1];
        if (state == kLive && rb != 0.f) state = kFailed;
    }

    // ---- the returned plan P = U K V, measured (Section 4) ----
#pragma unroll
    for (int t = 0; t < NS; ++t)
        if (in_s[t]) {
            Ub[w][n][x_s[t] - w * JI] = U_s[t];
            Vb[w][n][x_s[t] - w * JI] = V_s[t];
        }
    gemm<NH, JI, JP>(A1, &Vb[w][n][0], D);
#pragma unroll
    for (int h = 0; h < NH; ++h) P[0][w][h][l] = D[h];
    gemm<NH, JI, JP>(A2, &Ub[w][n][0], D);
#pragma unroll
    for (int h = 0; h < NH; ++h) P[1][w][h][l] = D[h];
    {
        // sum_j K_ij cl_ij V_j: the loss weights, with cl from the cost itself
        float AL[NH][JI];
#pragma unroll
        for (int h = 0; h < NH; ++h)
#pragma unroll
            for (int k = 0; k < JI; ++k) {
                const int i = l + 64 * h, j = w * JI + k;
                AL[h][k] = (i < d1 && j < d2) ? A1[h][k] * (-s * C[(size_t)i * d2 + j]) : 0.f;
            }
        gemm<NH, JI, JP>(AL, &Vb[w][n][0], D);
#pragma unroll
        for (int h = 0; h < NH; ++h) P[2][w][h][l] = D[h];
    }
    __syncthreads();
    float err = 0.f, lsum = 0.f;
#pragma unroll
    for (int t = 0; t < NS; ++t) {
        const float R = gather_partials<NH>(P[0], x_s[t], n);
        const float S = gather_partials<NH>(P[1], x_s[t], n);
        const float L = gather_partials<NH>(P[2], x_s[t], n);
        if (mu_s[t] > 0.f) {
            err += fabsf(U_s[t] * R - mu_s[t]);
            lsum = __builtin_fmaf(U_s[t], L, lsum);
        }
        if (nu_s[t] > 0.f) err += fabsf(V_s[t] * S - nu_s[t]);
    }
    err = sum_n(err);
    lsum = sum_n(lsum);
    if (l < 4) {
        F[2][w][l][0] = err;
        F[2][w][l][1] = lsum;
    }
    __syncthreads();

    if (!real) return;
    if (state == kFailed) {
        if (w == 0 && l < 4) A.iters[b] = -1;
        return;
    }
#pragma unroll
    for (int t = 0; t < NS; ++t) {
        if (!in_s[t]) continue;
        const int x = x_s[t];
        if (x < d1) A.alpha[(size_t)b * d1 + x] = kLn2 * lg2(U_s[t]);
        if (x < d2) A.beta[(size_t)b * d2 + x] = kLn2 * (lg2(V_s[t]) - clmax);
    }
    if (w == 0 && l < 4) {
        A.loss[b] = -(F[2][0][n][1] + F[2][1][n][1] + F[2][2][n][1] + F[2][3][n][1]) / s;
        A.marg_err[b] = F[2][0][n][0] + F[2][1][n][0] + F[2][2][n][0] + F[2][3][n][0];
        A.iters[b] = kstop;
    }
}

template <int NH, int JI>
hipError_t launch_shape(const FwdArgs &a, hipStream_t st) {
    hipLaunchKernelGGL((sk_resident_mfma_kernel<NH, JI>), dim3((a.B + 3) / 4), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace

bool launch_resident_mfma(const FwdArgs &a, hipStream_t st, hipError_t *err) {
    if (a.n_iter <= 0 || a.c_batched) return false;
    const int dm = a.d1 > a.d2 ? a.d1 : a.d2;
    if (dm <= 16) *err = launch_shape<1, 4>(a, st);
    else if (dm <= 32) *err = launch_shape<1, 8>(a, st);
    else if (dm <= 64) *err = launch_shape<1, 16>(a, st);
    else if (dm <= 100) *err = launch_shape<2, 25>(a, st);
    else if (dm <= 128) *err = launch_shape<2, 32>(a, st);
    else return false;
    return true;
}

}  // namespace sk
