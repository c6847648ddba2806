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
// One work-group of two wavefronts per problem, max(d1, d2) <= 8 N <= 128;
// the plan lives in VGPRs (the products are those of sk_device.h).  Lane l = p + 8q (p = l & 7, q = l >> 3) of
// wavefront w holds P[p + 8r][q + 8t] for its row blocks r in [w H, w H + H)
// (H = ceil(N / 2)) and every column block t < N.  One pass over the
// registers forms both halves of H p:
//   rows:    partial sums over the lane's columns, summed over the 8 lanes q
//            through a per-wavefront LDS transpose (lane (p, q < H) gets row
//            p + 8 (w H + q));
//   columns: partial sums over the lane's rows, summed over the 8 lanes p and
//            the two wavefronts through LDS (thread c gets column c).
// So a row i lives on one lane and a column j on thread j: every vector of
// the conjugate-gradient iteration is kept there, and published to LDS for
// the next product.  Reductions are fixed-order block sums (deterministic).
#include "sk_device.h"
#include "sk_internal.h"

namespace sk {
namespace {

constexpr int kShWaves = 2;
constexpr int kVS = 20;  // LDS line stride of the published vectors (16-byte reads, 8 lines on distinct banks)

template <int N>
__global__ __launch_bounds__(64 * kShWaves) __attribute__((amdgpu_waves_per_eu(2))) void sk_sharp_kernel(SharpArgs A) {
    constexpr int H = (N + 1) / 2;
    static_assert(8 * N <= 128 && H <= 8, "one thread per column, one lane per row");
    // Published vectors: column j at colv[(j & 7) * kVS + (j >> 3)] (lane
    // (p, q) reads line q), row p + 8 (w H + r) at rowv[p * kVS + 8 w + r]
    // (lane (p, q) of wavefront w reads line p from entry 8w).
    __shared__ __attribute__((aligned(16))) float colv[8 * kVS];
    __shared__ __attribute__((aligned(16))) float rowv[8 * kVS];
    __shared__ __attribute__((aligned(16))) float cp[2][kColumnPartialsFloats];
    __shared__ __attribute__((aligned(16))) float tsum[kShWaves][kRowTotalsFloats];
    __shared__ float bs[2][kShWaves][4];  // block-sum slots, alternating

    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int p = lane & 7, q = lane >> 3;
    const int b = blockIdx.x;
    const int d1 = A.d1, d2 = A.d2;
    const float s = A.s;
    const float *Cb = A.C + (A.c_batched ? (size_t)b * d1 * d2 : 0);
    float *const tb = tsum[w];
    // Fixed-order sum over the work-group of n <= 4 values per thread; one
    // barrier (a wavefront can be at most one sum ahead of the other, so two
    // alternating slots suffice).
    int slot = 0;
    auto block_sum = [&](float(&v)[4], int n) {
        for (int k = 0; k < n; ++k) v[k] = wave_sum(v[k]);
        if (lane == 0)
            for (int k = 0; k < n; ++k) bs[slot][w][k] = v[k];
        __syncthreads();
        for (int k = 0; k < n; ++k) v[k] = bs[slot][0][k] + bs[slot][1][k];
        slot ^= 1;
    };

    // The lane's cells: rows i = p + 8 (w H + ii), columns j = q + 8t.
    float a2[H];  // base-2 potentials of the lane's rows
#pragma unroll
    for (int ii = 0; ii < H; ++ii) {
        const int i = p + 8 * (w * H + ii);
        a2[ii] = i < d1 ? A.alpha[(size_t)b * d1 + i] * kLog2e : 0.f;
    }
    // The plan P_ij = 2^(a_i + b_j - s C_ij) (0 off the problem), column
    // block by column block, with the row partials of P and of P o C in
    // registers and the column partials written out as each block is done.
    float P[H][N];
    float rP[H], rPC[H];
#pragma unroll
    for (int ii = 0; ii < H; ++ii) rP[ii] = rPC[ii] = 0.f;
#pragma unroll
    for (int t = 0; t < N; ++t) {
        const int j = q + 8 * t;
        const float bj = j < d2 ? A.beta[(size_t)b * d2 + j] * kLog2e : 0.f;
        float cs = 0.f, csc = 0.f;
#pragma unroll
        for (int ii = 0; ii < H; ++ii) {
            const int i = p + 8 * (w * H + ii);
            const bool in = i < d1 && j < d2;
            const float cij = in ? Cb[(size_t)i * d2 + j] : 0.f;
            const float v = in ? ex2((a2[ii] + bj) - s * cij) : 0.f;
            P[ii][t] = v;
            rP[ii] += v;
            rPC[ii] = __builtin_fmaf(v, cij, rPC[ii]);
            cs += v;
            csc = __builtin_fmaf(v, cij, csc);
        }
        cp[0][partial_at(w, p, q, t)] = cs;
        cp[1][partial_at(w, p, q, t)] = csc;
    }

    // Owners: lane (p, q < H) owns row i = p + 8 (w H + q); thread c owns column c.
    const int c = threadIdx.x;
    const int i_own = p + 8 * (w * H + q);
    const bool row_on = q < H && i_own < d1;
    const bool col_on = c < d2;
    // Diagonal of H (the plan's marginals) and the right-hand side (a, b).
    float dgf = row_totals<H>(rP, tb, p, q);
    float rf = row_totals<H>(rPC, tb, p, q);
    __syncthreads();
    float dgg = col_on ? column_total(cp[0], c) : 0.f;
    float rg = col_on ? column_total(cp[1], c) : 0.f;
    const float mf = row_on ? A.mu[(size_t)b * d1 + i_own] : 0.f;
    const float mg = col_on ? A.nu[(size_t)b * d2 + c] : 0.f;
    const bool supf = row_on && mf > 0.f && dgf > 0.f;
    const bool supg = col_on && mg > 0.f && dgg > 0.f;
    if (!supf) dgf = rf = 0.f;
    if (!supg) dgg = rg = 0.f;
    // Project the right-hand side off (1, -1) over the supports.
    {
        float v[4] = {(supf ? rf : 0.f) - (supg ? rg : 0.f), (supf ? 1.f : 0.f) + (supg ? 1.f : 0.f), 0.f, 0.f};
        block_sum(v, 2);
        if (supf) rf -= v[0] / v[1];
        if (supg) rg += v[0] / v[1];
    }

    // Jacobi-preconditioned conjugate gradients; every scalar is a block sum,
    // so the control flow is uniform across the work-group.
    float xf = 0.f, xg = 0.f;
    float zf = supf ? rf / dgf : 0.f, zg = supg ? rg / dgg : 0.f;
    float pf = zf, pg = zg;
    float rz;
    {
        float v[4] = {rf * zf + rg * zg, 0.f, 0.f, 0.f};
        block_sum(v, 1);
        rz = v[0];
    }
    const float stop = A.cg_tol * A.cg_tol * rz;
    int it = 0;
    if (rz > 0.f) {
        while (it < A.max_cg) {
            // Publish p; its row half and its column half meet the plan.
            if (q < H) rowv[p * kVS + 8 * w + q] = pf;
            if (c < 8 * N) colv[(c & 7) * kVS + (c >> 3)] = pg;
            __syncthreads();
            float wc[N], wr[H];
#pragma unroll
            for (int t = 0; t < N; ++t) wc[t] = colv[q * kVS + t];
#pragma unroll
            for (int ii = 0; ii < H; ++ii) wr[ii] = rowv[p * kVS + 8 * w + ii];
            // One pass over the plan: row partials against the column half
            // of p, column partials against the row half (written out per
            // column block).
            // (At the lowest issue priority: the wavefronts sharing a SIMD
            // belong to different problems, and the serial rest of an
            // iteration -- transposes, block sums -- should not queue
            // behind another problem's FMAs.)
            __builtin_amdgcn_s_setprio(0);
            float yr[H];
#pragma unroll
            for (int ii = 0; ii < H; ++ii) yr[ii] = 0.f;
#pragma unroll
            for (int t = 0; t < N; ++t) {
                float yc = 0.f;
#pragma unroll
                for (int ii = 0; ii < H; ++ii) {
                    yr[ii] = __builtin_fmaf(P[ii][t], wc[t], yr[ii]);
                    yc = __builtin_fmaf(P[ii][t], wr[ii], yc);
                }
                cp[0][partial_at(w, p, q, t)] = yc;
            }
            __builtin_amdgcn_s_setprio(3);
            const float Pp = row_totals<H>(yr, tb, p, q);  // (P p_g)_i on the row owner
            __syncthreads();
            const float PTp = col_on ? column_total(cp[0], c) : 0.f;  // (P^T p_f)_j on the column owner
            const float qf = supf ? __builtin_fmaf(dgf, pf, Pp) : 0.f;
            const float qg = supg ? __builtin_fmaf(dgg, pg, PTp) : 0.f;
            float v[4] = {pf * qf + pg * qg, 0.f, 0.f, 0.f};
            block_sum(v, 1);  // its barrier also retires this product's reads of cp, colv and rowv
            const float pq = v[0];
            if (!(pq > 0.f)) break;
            const float step = rz / pq;
            xf = __builtin_fmaf(step, pf, xf);
            xg = __builtin_fmaf(step, pg, xg);
            rf = __builtin_fmaf(-step, qf, rf);
            rg = __builtin_fmaf(-step, qg, rg);
            zf = supf ? rf / dgf : 0.f;
            zg = supg ? rg / dgg : 0.f;
            float u[4] = {rf * zf + rg * zg, 0.f, 0.f, 0.f};
            block_sum(u, 1);
            const float rzn = u[0];
            ++it;
            if (!(rzn > stop)) break;
            pf = __builtin_fmaf(rzn / rz, pf, zf);
            pg = __builtin_fmaf(rzn / rz, pg, zg);
            rz = rzn;
        }
    }

    // Centre each block over its support, scale by the upstream gradient.
    float v[4] = {supf ? xf : 0.f, supf ? 1.f : 0.f, supg ? xg : 0.f, supg ? 1.f : 0.f};
    block_sum(v, 4);
    const float g = A.grad_loss[b];
    if (row_on) {
        const float mean = v[1] > 0.f ? v[0] / v[1] : 0.f;
        A.grad_mu[(size_t)b * d1 + i_own] = supf ? g * (xf - mean) : 0.f;
    }
    if (col_on) {
        const float mean = v[3] > 0.f ? v[2] / v[3] : 0.f;
        A.grad_nu[(size_t)b * d2 + c] = supg ? g * (xg - mean) : 0.f;
    }
    if (threadIdx.x == 0 && A.cg_iters) A.cg_iters[b] = it;
}

template <int N>
hipError_t launch_n(const SharpArgs &a, hipStream_t st) {
    hipLaunchKernelGGL((sk_sharp_kernel<N>), dim3(a.B), dim3(64 * kShWaves), 0, st, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_sharp(const SharpArgs &a, hipStream_t st) {
    const int nb = ((a.d1 > a.d2 ? a.d1 : a.d2) + 7) / 8;  // at most kSharpMaxD / 8 = 16
    if (nb <= 2) return launch_n<2>(a, st);
    if (nb <= 4) return launch_n<4>(a, st);
    if (nb <= 8) return launch_n<8>(a, st);
    if (nb <= 13) return launch_n<13>(a, st);
    return launch_n<16>(a, st);
}

}  // namespace sk
