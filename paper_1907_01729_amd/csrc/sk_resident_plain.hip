// sk_resident_plain.hip -- small problems in the plain form, the kernel matrix in VGPRs.
//
// The same iterates as the log-domain resident kernel (v-update first, then
// u-update), computed in the plain form of eq. (sk_plain),
//   u = mu / (K v),   v = nu / (K^T u),
// with the potentials tracked in the log domain and a shift per iteration so
// that every fp32 quantity stays normal.  Section 3 motivates the log domain
// by exactly this range problem; here a range test per problem decides, and a
// problem that fails it (or any guard below, at any iteration) is marked with
// iters = -1 and solved from the start by the log-domain kernel launched right
// after on the same stream.
//
// Base-2 notation: cl = -C log2(e)/lambda, clmax = max cl over the problem and
// K = 2^(cl - clmax) in [2^-64, 1] (range test: max cl - min cl <= 64).  With
// B = max_j b_j over the support of nu:
//   V_j = 2^(b_j - B),   R_i = sum_j K_ij V_j,   U_i = mu_i / R_i,
//   a_i = log2 U_i - (B + clmax),   S_j = sum_i K_ij U_i,
//   b_j' = log2 nu_j + B - log2 S_j,
// so that P_ij = U_i K_ij V_j = 2^(a_i + b_j + cl_ij), as in the log form.
// Guards: R_i, S_j in [2^-64, 2^64] and log2 U_i in [-100, 100] on the
// supports.  Then U_i <= 2^100, S_j <= 2^107 never overflow, and every product
// that underflows (< 2^-126) is below 2^-55 of the sum it drops out of.
//
// Work-group = one problem, H wavefronts, lane = 8p + q.  Two register copies
// of K, one per pass, so that both matrix-vector products reduce over the 8
// lanes q (three DPP adds) and never across DPP rows:
//   row pass    (layout A): wave h owns rows i = H(p + 8r) + h, all columns j = q + 8t;
//   column pass (layout B): wave h owns columns j = H(p + 8t) + h, all rows i = q + 8r.
// The vectors cross between the layouts (and the wavefronts) through LDS:
// U after the row pass, b after the column pass; one barrier each.
#include "sk_device.h"
#include "sk_internal.h"

namespace sk {
namespace {

constexpr float kLo = 5.42101086242752217e-20f;   // 2^-64
constexpr float kHi = 1.84467440737095516e19f;    // 2^64
constexpr float kRangeBits = 64.f;                // largest spread of cl the plain form takes
constexpr float kLogUMax = 100.f;                 // |log2 U_i| bound on the support

__device__ __forceinline__ bool in_range(float x) { return x >= kLo && x <= kHi; }

// Scalars a wavefront publishes per phase: [0] error part, [1] guard failure,
// [2] loss part.
constexpr int kScal = 4;

template <int N, int H>
struct Shape {
    static constexpr int NR = (N + H - 1) / H;  // rows per lane (layout A) = columns per lane (layout B)
    static constexpr int NP = (N + 3) & ~3;     // padded vector stride in LDS (16-byte reads)
};

// Sum over q of this lane's products with the vector, per owned row (layout A)
// or column (layout B): out[x] = sum_q sum_y M[x][y] w[y].
template <int NX, int NY>
__device__ __forceinline__ void matvec(const float (&M)[NX][NY], const float (&w)[NY], float (&out)[NX]) {
#pragma unroll
    for (int x = 0; x < NX; ++x) {
        float s0 = 0.f, s1 = 0.f;
#pragma unroll
        for (int y = 0; y < NY; ++y) {
            if (y & 1)
                s1 = __builtin_fmaf(M[x][y], w[y], s1);
            else
                s0 = __builtin_fmaf(M[x][y], w[y], s0);
        }
        out[x] = sum_q(s0 + s1);
    }
}

// Wave-uniform sum of published scalars over the H wavefronts, in wave order.
template <int H>
__device__ __forceinline__ float gather(const float (*slot)[kScal], int k) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < H; ++w) s += slot[w][k];
    return s;
}

template <int N, int H>
__global__ __launch_bounds__(64 * H) __attribute__((amdgpu_waves_per_eu(2))) void sk_resident_plain_kernel(FwdArgs A) {
    using S = Shape<N, H>;
    constexpr int NR = S::NR, NP = S::NP;
    // xb: b_j at [(j & 7) * NP + (j >> 3)], two buffers (current iterate and
    // the next);  xu: U_i at [(i & 7) * NP + (i >> 3)].
    __shared__ __align__(16) float xb[2][8 * NP];
    __shared__ __align__(16) float xu[8 * NP];
    __shared__ float mus[8 * N], nus[8 * N];
    __shared__ float scal[4][H][kScal];  // 0 range, 1 row pass, 2 column pass, 3 final

    const int lane = threadIdx.x & 63, h = threadIdx.x >> 6;
    const int p = lane >> 3, q = lane & 7;
    const int b = blockIdx.x;
    const int d1 = A.d1, d2 = A.d2;
    const float *Cb = A.C + (A.c_batched ? (size_t)b * d1 * d2 : 0);
    const float *mub = A.mu + (size_t)b * d1;
    const float *nub = A.nu + (size_t)b * d2;
    const float s = A.s;

    for (int x = threadIdx.x; x < 8 * N; x += 64 * H) {
        mus[x] = x < d1 ? mub[x] : 0.f;
        nus[x] = x < d2 ? nub[x] : 0.f;
    }

    // Layout A cost cells (scaled) and their range; every cell of the problem
    // sits in exactly one lane of one wavefront in this layout.
    float KA[NR][N];
    float mx = neg_inf(), mn = __builtin_inff();
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int i = H * (p + 8 * r) + h;
#pragma unroll
        for (int t = 0; t < N; ++t) {
            const int j = q + 8 * t;
            // Cells outside the problem hold -inf (K = 0 there), so no mask
            // per cell has to stay alive past this loop.
            const bool v = i < d1 && j < d2;
            const float c = v ? -s * Cb[(size_t)i * d2 + j] : neg_inf();
            KA[r][t] = c;
            mx = fmaxf(mx, c);
            mn = fminf(mn, v ? c : __builtin_inff());
        }
    }
    mx = wave_max(mx);
    mn = -wave_max(-mn);
    if (lane == 0) {
        scal[0][h][0] = mx;
        scal[0][h][1] = mn;
    }
    __syncthreads();
#pragma unroll
    for (int w = 0; w < H; ++w) {
        mx = fmaxf(mx, scal[0][w][0]);
        mn = fminf(mn, scal[0][w][1]);
    }
    if (!(mx - mn <= kRangeBits)) {  // also catches an empty or non-finite cost
        if (threadIdx.x == 0) A.iters[b] = -1;
        return;
    }
    const float clmax = mx;
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int i = H * (p + 8 * r) + h;
#pragma unroll
        for (int t = 0; t < N; ++t) KA[r][t] = ex2(KA[r][t] - clmax);
    }
    float KB[NR][N];  // KB[t][r] = K[q + 8r, H(p + 8t) + h]
#pragma unroll
    for (int t = 0; t < NR; ++t) {
        const int j = H * (p + 8 * t) + h;
#pragma unroll
        for (int r = 0; r < N; ++r) {
            const int i = q + 8 * r;
            KB[t][r] = (i < d1 && j < d2) ? ex2(-s * Cb[(size_t)i * d2 + j] - clmax) : 0.f;
        }
    }

    // log2 of the marginals on the owned rows (layout A) and columns (layout B).
    float la[NR], lb[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int i = H * (p + 8 * r) + h;  // also the column index j of layout B
        const float m = i < d1 ? mub[i] : 0.f;
        la[r] = m > 0.f ? log2f(m) : neg_inf();
        const float n = i < d2 ? nub[i] : 0.f;
        lb[r] = n > 0.f ? log2f(n) : neg_inf();
    }

    const int n_iter = A.n_iter;
    const float tol = A.tol;
    const bool check = tol > 0.f;
    int K = n_iter;
    bool fail = false;
    int cur = 0;         // xb[cur] holds the column potentials of the current iterate
    float Bsh = -clmax;  // shift of the U just used: U_i = 2^(a_i + Bsh + clmax)

    // v-update of iteration 1 from a^0 = 0 on the support of mu (U_i = 1 there).
    {
        float U[N];
#pragma unroll
        for (int r = 0; r < N; ++r) {
            const int i = q + 8 * r;
            U[r] = (i < d1 && mub[i] > 0.f) ? 1.f : 0.f;
        }
        float Sc[NR];
        matvec<NR, N>(KB, U, Sc);
        bool bad = false;
#pragma unroll
        for (int t = 0; t < NR; ++t) {
            const bool act = lb[t] != neg_inf();
            bad |= act && !in_range(Sc[t]);
            const int j = H * (p + 8 * t) + h;
            if (q == 0 && j < 8 * N) xb[0][(j & 7) * NP + (j >> 3)] = act ? (lb[t] + Bsh) - lg2(Sc[t]) : neg_inf();
        }
        if (lane == 0) scal[2][h][1] = __any(bad) ? 1.f : 0.f;
        __syncthreads();
        fail = gather<H>(scal[2], 1) != 0.f;
    }

    float V[N];
    for (int k = 1; k <= n_iter && !fail; ++k) {
        // ---- row pass: u-update of iteration k ----
        float bmax = neg_inf();
#pragma unroll
        for (int t = 0; t < N; ++t) {
            V[t] = xb[cur][q * NP + t];
            bmax = fmaxf(bmax, V[t]);
        }
        Bsh = max_q(bmax);
#pragma unroll
        for (int t = 0; t < N; ++t) V[t] = ex2(V[t] - Bsh);
        float R[NR];
        matvec<NR, N>(KA, V, R);
        float rerr = 0.f;
        bool bad = !(Bsh > neg_inf());
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const int i = H * (p + 8 * r) + h;
            const bool act = la[r] != neg_inf();
            const float g = la[r] - lg2(R[r]);
            bad |= act && !(in_range(R[r]) && fabsf(g) <= kLogUMax);
            const float U = act ? ex2(g) : 0.f;
            if (q == 0) {
                if (check && act) rerr += fabsf(U * R[r] - mus[i]);
                if (i < 8 * N) xu[(i & 7) * NP + (i >> 3)] = U;
            }
        }
        rerr = wave_sum(rerr);
        const bool wbad = __any(bad);
        if (lane == 0) {
            scal[1][h][0] = rerr;
            scal[1][h][1] = wbad ? 1.f : 0.f;
        }
        __syncthreads();
        const float row_err = gather<H>(scal[1], 0);
        if (gather<H>(scal[1], 1) != 0.f) {
            fail = true;
            break;
        }
        if (k == n_iter) break;

        // ---- column pass: plan column sums, then the v-update of iteration
        // k+1 into the other buffer ----
        float U[N];
#pragma unroll
        for (int r = 0; r < N; ++r) U[r] = xu[q * NP + r];
        float Sc[NR];
        matvec<NR, N>(KB, U, Sc);
        float cerr = 0.f;
        bad = false;
#pragma unroll
        for (int t = 0; t < NR; ++t) {
            const int j = H * (p + 8 * t) + h;
            const int x = (j & 7) * NP + (j >> 3);
            const bool act = lb[t] != neg_inf();
            bad |= act && !in_range(Sc[t]);
            if (check && act && q == 0) cerr += fabsf(ex2(xb[cur][x] - Bsh) * Sc[t] - nus[j]);
            if (q == 0 && j < 8 * N) xb[cur ^ 1][x] = act ? (lb[t] + Bsh) - lg2(Sc[t]) : neg_inf();
        }
        cerr = wave_sum(cerr);
        const bool cbad = __any(bad);
        if (lane == 0) {
            scal[2][h][0] = cerr;
            scal[2][h][1] = cbad ? 1.f : 0.f;
        }
        __syncthreads();
        if (gather<H>(scal[2], 1) != 0.f) {
            fail = true;
            break;
        }
        if (check && row_err + gather<H>(scal[2], 0) <= tol) {
            K = k;  // stop at iterate k: xb[cur] still holds its column potentials
            break;
        }
        cur ^= 1;
    }
    if (fail) {
        if (threadIdx.x == 0) A.iters[b] = -1;
        return;
    }

    // The returned plan P = U K V, measured entry by entry (Section 4): its
    // marginal error and sum P cl.
    float bmax = neg_inf();
#pragma unroll
    for (int t = 0; t < N; ++t) {
        V[t] = xb[cur][q * NP + t];
        bmax = fmaxf(bmax, V[t]);
    }
    Bsh = max_q(bmax);
#pragma unroll
    for (int t = 0; t < N; ++t) V[t] = ex2(V[t] - Bsh);
    float rerr = 0.f, lsum = 0.f;
    float aout[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int i = H * (p + 8 * r) + h;
        float s0 = 0.f, l0 = 0.f;
#pragma unroll
        for (int t = 0; t < N; ++t) {
            // K is 0 on cells outside the problem: read a clamped (in-bounds)
            // cost there instead of keeping a mask per cell alive.
            const int j = q + 8 * t;
            const int ic = i < d1 ? i : d1 - 1, jc = j < d2 ? j : d2 - 1;
            const float kv = KA[r][t] * V[t];
            s0 += kv;
            l0 = __builtin_fmaf(kv, -s * Cb[(size_t)ic * d2 + jc], l0);
        }
        const float R = sum_q(s0);
        const float Lr = sum_q(l0);
        const bool act = la[r] != neg_inf();
        const float g = la[r] - lg2(R);
        const float U = act ? ex2(g) : 0.f;
        aout[r] = act ? g - (Bsh + clmax) : neg_inf();
        if (q == 0) {
            if (act) rerr += fabsf(U * R - mus[i]);
            lsum = __builtin_fmaf(U, Lr, lsum);
            if (i < 8 * N) xu[(i & 7) * NP + (i >> 3)] = U;
        }
    }
    __syncthreads();
    float bout[NR];
    {
        float U[N];
#pragma unroll
        for (int r = 0; r < N; ++r) U[r] = xu[q * NP + r];
        float Sc[NR];
        matvec<NR, N>(KB, U, Sc);
        float cerr = 0.f;
#pragma unroll
        for (int t = 0; t < NR; ++t) {
            const int j = H * (p + 8 * t) + h;
            bout[t] = j < 8 * N ? xb[cur][(j & 7) * NP + (j >> 3)] : neg_inf();
            if (lb[t] != neg_inf() && q == 0) cerr += fabsf(ex2(bout[t] - Bsh) * Sc[t] - nus[j]);
        }
        rerr = wave_sum(rerr);
        cerr = wave_sum(cerr);
        lsum = wave_sum(lsum);
        if (lane == 0) {
            scal[3][h][0] = rerr + cerr;
            scal[3][h][2] = lsum;
        }
    }
    __syncthreads();

    if (q == 0) {
        float *al = A.alpha + (size_t)b * d1;
        float *be = A.beta + (size_t)b * d2;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const int i = H * (p + 8 * r) + h;
            if (i < d1) al[i] = aout[r] * kLn2;
            if (i < d2) be[i] = bout[r] * kLn2;  // column index of layout B has the same form
        }
    }
    if (threadIdx.x == 0) {
        A.loss[b] = -gather<H>(scal[3], 2) / s;  // sum P C = -(1/s) sum P cl
        A.marg_err[b] = gather<H>(scal[3], 0);
        A.iters[b] = K;
    }
}

template <int N, int H>
hipError_t launch_shape(const FwdArgs &a, hipStream_t st) {
    hipLaunchKernelGGL((sk_resident_plain_kernel<N, H>), dim3(a.B), dim3(64 * H), 0, st, a);
    return hipGetLastError();
}

}  // namespace

bool launch_resident_plain(const FwdArgs &a, hipStream_t st, hipError_t *err) {
    if (a.n_iter <= 0) return false;
    const int dm = a.d1 > a.d2 ? a.d1 : a.d2;
    const int n = (dm + 7) / 8;
    if (n <= 2) *err = launch_shape<2, 1>(a, st);
    else if (n <= 4) *err = launch_shape<4, 1>(a, st);
    else if (n <= 8) *err = launch_shape<8, 2>(a, st);
    else if (n <= 13) *err = launch_shape<13, 4>(a, st);
    else if (n <= 16) *err = launch_shape<16, 4>(a, st);
    else return false;
    return true;
}

}  // namespace sk
