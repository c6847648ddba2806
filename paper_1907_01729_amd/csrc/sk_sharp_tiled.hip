// sk_sharp_tiled.hip -- gradient of the sharp loss E^0 for supports larger
// than the resident kernel takes (max(d1, d2) > 128): the same implicit
// differentiation and preconditioned conjugate gradients as sk_sharp.hip, with
// the plan never stored.
//
// With P_ij = 2^(a_i + b_j + cl_ij) rebuilt cell by cell (one exponential),
// every product of the iteration is one sweep over the cells, a work-group
// per (row block, problem), wavefronts taking whole rows and lanes the
// columns:
//   setup:  r = P 1 and (P o C) 1 per row (wavefront all-reduce), the column
//           sums of P and P o C as row-block partials;
//   CG:     (P p_g)_i per row and the row-block partials of P^T p_f, both
//           halves of H p from the same exponentials.
// One work-group per problem then merges the partials in a fixed order and
// takes the conjugate-gradient step (dot products are fixed-order block
// sums), with the vectors of the iteration in the workspace.  A problem that
// has converged (or whose step broke down) is marked done, and every later
// launch skips it; the host launches max_cg iterations.
#include "sk_device.h"
#include "sk_internal.h"

namespace sk {
namespace {

constexpr int kShtThreads = 256;  // sweep: 4 wavefronts, whole rows each
constexpr int kShtWaves = kShtThreads / 64;
constexpr int kShuThreads = 1024;  // per-problem merge and update
constexpr float kShtPadCost = -1.0e30f;  // scaled cost past d2: plan entry 0

struct ShtArgs {
    const float *grad_loss, *mu, *nu, *C, *alpha, *beta;
    float *grad_mu, *grad_nu;
    int32_t *cg_iters;  // may be null
    // workspace: per problem [B][d1] or [B][d2p] vectors
    float *a2, *b2;      // base-2 potentials (b2: 0 past d2)
    float *dgf, *dgg;    // diagonal of H: the plan's marginals (0 off the supports)
    float *xf, *xg;      // solution
    float *rf, *rg;      // residual (setup: the right-hand side)
    float *pf, *pg;      // search direction
    float *Pp;           // (P p_g)_i of the last product
    float *part;         // [2][R][B][d2p] column partials
    float *sc;           // [B][4]: rz, stop threshold, iterations, done
    int B, d1, d2, d2p, R, RBS, c_batched, max_cg;
    float s, cg_tol;
};

__device__ __forceinline__ size_t ppart(const ShtArgs &T, int plane, int r, int b, int j) {
    return (((size_t)plane * T.R + r) * T.B + b) * (size_t)T.d2p + j;
}

template <int NT>
__device__ __forceinline__ float block_sum_sh(float v, float *red) {
    v = wave_sum(v);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) s += red[w];
    return s;
}

// Base-2 potentials of the forward's output (0 past d2).
__global__ __launch_bounds__(kShuThreads) void sk_sht_prep(ShtArgs T) {
    const int b = blockIdx.x;
    for (int i = threadIdx.x; i < T.d1; i += kShuThreads)
        T.a2[(size_t)b * T.d1 + i] = T.alpha[(size_t)b * T.d1 + i] * kLog2e;
    for (int j = threadIdx.x; j < T.d2p; j += kShuThreads)
        T.b2[(size_t)b * T.d2p + j] = j < T.d2 ? T.beta[(size_t)b * T.d2 + j] * kLog2e : 0.f;
    if (threadIdx.x == 0) T.sc[(size_t)b * 4 + 3] = 0.f;
}

// One sweep over the cells of row block r of problem b.
// SETUP: row i -> dgf_i = sum_j P_ij, rf_i = sum_j P_ij C_ij; column partials
//        of P (plane 0) and P o C (plane 1).
// else:  row i -> Pp_i = sum_j P_ij pg_j; column partials of sum_i P_ij pf_i
//        (plane 0); problems marked done are skipped.
template <int NCW, bool SETUP>
__global__ __launch_bounds__(kShtThreads) void sk_sht_sweep(ShtArgs T) {
    extern __shared__ float lds[];  // [kShtWaves][NCW * 64] column partials of the wavefronts
    const int r = blockIdx.x, b = blockIdx.y;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (!SETUP && T.sc[(size_t)b * 4 + 3] != 0.f) return;  // work-group-uniform
    const int d1 = T.d1, d2 = T.d2;
    const float *Cb = T.C + (T.c_batched ? (size_t)b * d1 * d2 : 0);
    const float ns = -T.s;
    float bv[NCW], pg[NCW], c0[NCW], c1[NCW];
#pragma unroll
    for (int c = 0; c < NCW; ++c) {
        const int j = lane + 64 * c;
        bv[c] = T.b2[(size_t)b * T.d2p + j];
        pg[c] = SETUP ? 0.f : T.pg[(size_t)b * T.d2p + j];
        c0[c] = c1[c] = 0.f;
    }
    const int i0 = r * T.RBS, i1 = min(d1, i0 + T.RBS);
    for (int i = i0 + w; i < i1; i += kShtWaves) {
        const float ai = T.a2[(size_t)b * d1 + i];
        const float pfi = SETUP ? 0.f : T.pf[(size_t)b * d1 + i];
        const float *crow = Cb + (size_t)i * d2;
        float x0 = 0.f, x1 = 0.f;
#pragma unroll
        for (int c = 0; c < NCW; ++c) {
            const int j = lane + 64 * c;
            const float cij = j < d2 ? crow[j] : 0.f;
            const float e = ex2((ai + bv[c]) + (j < d2 ? ns * cij : kShtPadCost));
            if (SETUP) {
                x0 += e;
                x1 = __builtin_fmaf(e, cij, x1);
                c0[c] += e;
                c1[c] = __builtin_fmaf(e, cij, c1[c]);
            } else {
                x0 = __builtin_fmaf(e, pg[c], x0);
                c0[c] = __builtin_fmaf(e, pfi, c0[c]);
            }
        }
        x0 = wave_sum(x0);
        if (SETUP) x1 = wave_sum(x1);
        if (lane == 0) {
            if (SETUP) {
                T.dgf[(size_t)b * d1 + i] = x0;
                T.rf[(size_t)b * d1 + i] = x1;
            } else {
                T.Pp[(size_t)b * d1 + i] = x0;
            }
        }
    }
    // Combine the wavefronts' partials in a fixed order and store.
#pragma unroll
    for (int plane = 0; plane < (SETUP ? 2 : 1); ++plane) {
        __syncthreads();
#pragma unroll
        for (int c = 0; c < NCW; ++c) lds[w * NCW * 64 + c * 64 + lane] = plane ? c1[c] : c0[c];
        __syncthreads();
        for (int j = threadIdx.x; j < T.d2p && j < NCW * 64; j += kShtThreads) {
            float v = 0.f;
#pragma unroll
            for (int q = 0; q < kShtWaves; ++q) v += lds[q * NCW * 64 + j];
            T.part[ppart(T, plane, r, b, j)] = v;
        }
    }
}

// Rows wider than one wavefront's registers hold (d2 > kTiledMaxD2): each
// product takes two passes over the cells, one exponential per cell in each.
// The rows pass (one wavefront per row, looping over the columns) forms the
// row half (SETUP: the plan's row marginal and (P o C) 1); the columns pass
// (one thread per column, looping over a row block) the row blocks' column
// partials.  Setup, update and final are those of the one-pass sweep.
constexpr int kShtWideWaves = 16;

template <bool SETUP>
__global__ __launch_bounds__(64 * kShtWideWaves) void sk_sht_rows(ShtArgs T) {
    const int r = blockIdx.x, b = blockIdx.y;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (!SETUP && T.sc[(size_t)b * 4 + 3] != 0.f) return;  // work-group-uniform
    const int d1 = T.d1, d2 = T.d2;
    const float *Cb = T.C + (T.c_batched ? (size_t)b * d1 * d2 : 0);
    const float *bv = T.b2 + (size_t)b * T.d2p;
    const float *pg = T.pg + (size_t)b * T.d2p;
    const float ns = -T.s;
    const int i0 = r * T.RBS, i1 = min(d1, i0 + T.RBS);
    for (int i = i0 + w; i < i1; i += kShtWideWaves) {
        const float ai = T.a2[(size_t)b * d1 + i];
        const float *crow = Cb + (size_t)i * d2;
        float x0 = 0.f, x1 = 0.f;
        for (int j = lane; j < d2; j += 64) {
            const float cij = crow[j];
            const float e = ex2((ai + bv[j]) + ns * cij);
            if (SETUP) {
                x0 += e;
                x1 = __builtin_fmaf(e, cij, x1);
            } else {
                x0 = __builtin_fmaf(e, pg[j], x0);
            }
        }
        x0 = wave_sum(x0);
        if (SETUP) x1 = wave_sum(x1);
        if (lane == 0) {
            if (SETUP) {
                T.dgf[(size_t)b * d1 + i] = x0;
                T.rf[(size_t)b * d1 + i] = x1;
            } else {
                T.Pp[(size_t)b * d1 + i] = x0;
            }
        }
    }
}

template <bool SETUP>
__global__ __launch_bounds__(kShtThreads) void sk_sht_cols(ShtArgs T) {
    const int j = blockIdx.x * kShtThreads + threadIdx.x;
    const int r = blockIdx.y, b = blockIdx.z;
    if (!SETUP && T.sc[(size_t)b * 4 + 3] != 0.f) return;  // work-group-uniform
    const int d1 = T.d1, d2 = T.d2;
    const int i0 = r * T.RBS, i1 = min(d1, i0 + T.RBS);
    float c0 = 0.f, c1 = 0.f;
    if (j < d2) {
        const float bj = T.b2[(size_t)b * T.d2p + j];
        const float *col = T.C + (T.c_batched ? (size_t)b * d1 * d2 : 0) + j;
        const float *ab = T.a2 + (size_t)b * d1;
        const float *pf = T.pf + (size_t)b * d1;
        const float ns = -T.s;
        for (int i = i0; i < i1; ++i) {
            const float cij = col[(size_t)i * d2];
            const float e = ex2((ab[i] + bj) + ns * cij);
            if (SETUP) {
                c0 += e;
                c1 = __builtin_fmaf(e, cij, c1);
            } else {
                c0 = __builtin_fmaf(e, pf[i], c0);
            }
        }
    }
    T.part[ppart(T, 0, r, b, j)] = c0;
    if (SETUP) T.part[ppart(T, 1, r, b, j)] = c1;
}

// Fixed-order sum over the row blocks of column j's partial in plane pl.
__device__ __forceinline__ float merge_col(const ShtArgs &T, int pl, int b, int j) {
    float v = 0.f;
    for (int r = 0; r < T.R; ++r) v += T.part[ppart(T, pl, r, b, j)];
    return v;
}

// Setup per problem: the column marginals and right-hand side from the
// partials, the supports (mass > 0 and a positive plan marginal), the
// right-hand side projected off (1, -1), and the first conjugate-gradient
// vectors.
__global__ __launch_bounds__(kShuThreads) void sk_sht_setup(ShtArgs T) {
    __shared__ float red[kShuThreads / 64];
    const int b = blockIdx.x;
    const int d1 = T.d1, d2 = T.d2;
    float *dgf = T.dgf + (size_t)b * d1, *rf = T.rf + (size_t)b * d1;
    float *dgg = T.dgg + (size_t)b * T.d2p, *rg = T.rg + (size_t)b * T.d2p;
    const float *mu = T.mu + (size_t)b * d1, *nu = T.nu + (size_t)b * d2;
    float dsum = 0.f, cnt = 0.f;
    for (int i = threadIdx.x; i < d1; i += kShuThreads) {
        const bool sup = mu[i] > 0.f && dgf[i] > 0.f;
        if (!sup) dgf[i] = rf[i] = 0.f;
        dsum += sup ? rf[i] : 0.f;
        cnt += sup ? 1.f : 0.f;
    }
    for (int j = threadIdx.x; j < T.d2p; j += kShuThreads) {
        float dg = 0.f, rhs = 0.f;
        if (j < d2) {
            dg = merge_col(T, 0, b, j);
            rhs = merge_col(T, 1, b, j);
        }
        const bool sup = j < d2 && nu[j] > 0.f && dg > 0.f;
        dgg[j] = sup ? dg : 0.f;
        rg[j] = sup ? rhs : 0.f;
        dsum -= sup ? rhs : 0.f;
        cnt += sup ? 1.f : 0.f;
    }
    dsum = block_sum_sh<kShuThreads>(dsum, red);
    cnt = block_sum_sh<kShuThreads>(cnt, red);
    const float shift = cnt > 0.f ? dsum / cnt : 0.f;
    float rz = 0.f;
    for (int i = threadIdx.x; i < d1; i += kShuThreads) {
        const size_t u = (size_t)b * d1 + i;
        const bool sup = dgf[i] > 0.f;
        const float rv = sup ? rf[i] - shift : 0.f;
        const float z = sup ? rv / dgf[i] : 0.f;
        rf[i] = rv;
        T.xf[u] = 0.f;
        T.pf[u] = z;
        rz = __builtin_fmaf(rv, z, rz);
    }
    for (int j = threadIdx.x; j < T.d2p; j += kShuThreads) {
        const size_t u = (size_t)b * T.d2p + j;
        const bool sup = dgg[j] > 0.f;
        const float rv = sup ? rg[j] + shift : 0.f;
        const float z = sup ? rv / dgg[j] : 0.f;
        rg[j] = rv;
        T.xg[u] = 0.f;
        T.pg[u] = z;
        rz = __builtin_fmaf(rv, z, rz);
    }
    rz = block_sum_sh<kShuThreads>(rz, red);
    if (threadIdx.x == 0) {
        float *sc = T.sc + (size_t)b * 4;
        sc[0] = rz;
        sc[1] = T.cg_tol * T.cg_tol * rz;
        sc[2] = 0.f;
        sc[3] = rz > 0.f ? 0.f : 1.f;
    }
}

// One conjugate-gradient step per problem after its product sweep:
// q = H p, step = rz / <p, q>, x += step p, r -= step q, z = r / diag(H),
// and the next direction; stops when the preconditioned residual <r, z>
// falls to cg_tol^2 of its start, or when <p, q> is not positive.
__global__ __launch_bounds__(kShuThreads) void sk_sht_update(ShtArgs T) {
    __shared__ float red[kShuThreads / 64];
    const int b = blockIdx.x;
    float *sc = T.sc + (size_t)b * 4;
    if (sc[3] != 0.f) return;  // work-group-uniform
    const int d1 = T.d1, d2 = T.d2;
    const size_t of = (size_t)b * d1, og = (size_t)b * T.d2p;
    // q = H p over the supports: q_f in place of Pp, q_g in the first
    // row-block slot of partial plane 1 (free after the setup).
    float pq = 0.f;
    for (int i = threadIdx.x; i < d1; i += kShuThreads) {
        const float dg = T.dgf[of + i];
        const float qf = dg > 0.f ? __builtin_fmaf(dg, T.pf[of + i], T.Pp[of + i]) : 0.f;
        T.Pp[of + i] = qf;
        pq = __builtin_fmaf(T.pf[of + i], qf, pq);
    }
    for (int j = threadIdx.x; j < d2; j += kShuThreads) {
        const float dg = T.dgg[og + j];
        const float qg = dg > 0.f ? __builtin_fmaf(dg, T.pg[og + j], merge_col(T, 0, b, j)) : 0.f;
        T.part[ppart(T, 1, 0, b, j)] = qg;  // plane 1 is free after the setup
        pq = __builtin_fmaf(T.pg[og + j], qg, pq);
    }
    pq = block_sum_sh<kShuThreads>(pq, red);
    const float rz = sc[0];
    if (!(pq > 0.f)) {
        if (threadIdx.x == 0) sc[3] = 1.f;
        return;
    }
    const float step = rz / pq;
    float rzn = 0.f;
    for (int i = threadIdx.x; i < d1; i += kShuThreads) {
        const float dg = T.dgf[of + i];
        T.xf[of + i] = __builtin_fmaf(step, T.pf[of + i], T.xf[of + i]);
        const float rv = __builtin_fmaf(-step, T.Pp[of + i], T.rf[of + i]);
        T.rf[of + i] = rv;
        rzn = __builtin_fmaf(rv, dg > 0.f ? rv / dg : 0.f, rzn);
    }
    for (int j = threadIdx.x; j < d2; j += kShuThreads) {
        const float dg = T.dgg[og + j];
        T.xg[og + j] = __builtin_fmaf(step, T.pg[og + j], T.xg[og + j]);
        const float rv = __builtin_fmaf(-step, T.part[ppart(T, 1, 0, b, j)], T.rg[og + j]);
        T.rg[og + j] = rv;
        rzn = __builtin_fmaf(rv, dg > 0.f ? rv / dg : 0.f, rzn);
    }
    rzn = block_sum_sh<kShuThreads>(rzn, red);
    const bool done = !(rzn > sc[1]);
    if (!done) {
        const float beta = rzn / rz;
        for (int i = threadIdx.x; i < d1; i += kShuThreads) {
            const float dg = T.dgf[of + i];
            T.pf[of + i] = __builtin_fmaf(beta, T.pf[of + i], dg > 0.f ? T.rf[of + i] / dg : 0.f);
        }
        for (int j = threadIdx.x; j < d2; j += kShuThreads) {
            const float dg = T.dgg[og + j];
            T.pg[og + j] = __builtin_fmaf(beta, T.pg[og + j], dg > 0.f ? T.rg[og + j] / dg : 0.f);
        }
    }
    __syncthreads();  // every thread has read sc before it changes
    if (threadIdx.x == 0) {
        sc[0] = rzn;
        sc[2] += 1.f;
        if (done) sc[3] = 1.f;
    }
}

// Each block of the solution centred over its support (0 off it), scaled by
// the upstream gradient.
__global__ __launch_bounds__(kShuThreads) void sk_sht_final(ShtArgs T) {
    __shared__ float red[kShuThreads / 64];
    const int b = blockIdx.x;
    const int d1 = T.d1, d2 = T.d2;
    const size_t of = (size_t)b * d1, og = (size_t)b * T.d2p;
    float sf = 0.f, cf = 0.f, sg = 0.f, cg = 0.f;
    for (int i = threadIdx.x; i < d1; i += kShuThreads)
        if (T.dgf[of + i] > 0.f) {
            sf += T.xf[of + i];
            cf += 1.f;
        }
    for (int j = threadIdx.x; j < d2; j += kShuThreads)
        if (T.dgg[og + j] > 0.f) {
            sg += T.xg[og + j];
            cg += 1.f;
        }
    sf = block_sum_sh<kShuThreads>(sf, red);
    cf = block_sum_sh<kShuThreads>(cf, red);
    sg = block_sum_sh<kShuThreads>(sg, red);
    cg = block_sum_sh<kShuThreads>(cg, red);
    const float g = T.grad_loss[b];
    const float mf = cf > 0.f ? sf / cf : 0.f, mg = cg > 0.f ? sg / cg : 0.f;
    for (int i = threadIdx.x; i < d1; i += kShuThreads)
        T.grad_mu[of + i] = T.dgf[of + i] > 0.f ? g * (T.xf[of + i] - mf) : 0.f;
    for (int j = threadIdx.x; j < d2; j += kShuThreads)
        T.grad_nu[(size_t)b * d2 + j] = T.dgg[og + j] > 0.f ? g * (T.xg[og + j] - mg) : 0.f;
    if (threadIdx.x == 0 && T.cg_iters) T.cg_iters[b] = (int32_t)T.sc[(size_t)b * 4 + 2];
}

int sht_ncw(int d2) {
    const int n = (d2 + 63) / 64;
    return n <= 4 ? 4 : n <= 8 ? 8 : n <= 13 ? 13 : n <= 16 ? 16 : n <= 32 ? 32 : 64;
}

// Row blocks: about 512 work-groups in all, rows per block a multiple of the
// wavefronts per work-group.
void sht_row_blocks(int B, int d1, int d2, int *R, int *RBS) {
    int want = (512 + B - 1) / (B > 0 ? B : 1);
    // Wide rows: at most 64 row blocks (the update merges R d2 partials per
    // problem with one work-group).
    if (d2 > kTiledMaxD2 && want > 64) want = 64;
    const int maxR = (d1 + kShtWaves - 1) / kShtWaves;
    want = want < 1 ? 1 : (want > maxR ? maxR : want);
    int rbs = (d1 + want - 1) / want;
    rbs = (rbs + kShtWaves - 1) / kShtWaves * kShtWaves;
    *RBS = rbs;
    *R = (d1 + rbs - 1) / rbs;
}

struct ShtLayout {
    size_t a2, b2, dgf, dgg, xf, xg, rf, rg, pf, pg, Pp, part, sc, total;
};

size_t al256(size_t x) { return (x + 255) & ~size_t(255); }

ShtLayout sht_layout(int B, int d1, int d2, int *R, int *RBS, int *d2p) {
    sht_row_blocks(B, d1, d2, R, RBS);
    *d2p = d2 > kTiledMaxD2 ? (d2 + kShtThreads - 1) / kShtThreads * kShtThreads : 64 * sht_ncw(d2);
    const size_t f1 = sizeof(float) * (size_t)B * d1, f2 = sizeof(float) * (size_t)B * *d2p;
    ShtLayout L;
    size_t off = 0;
    L.a2 = off;
    off = al256(off + f1);
    L.b2 = off;
    off = al256(off + f2);
    L.dgf = off;
    off = al256(off + f1);
    L.dgg = off;
    off = al256(off + f2);
    L.xf = off;
    off = al256(off + f1);
    L.xg = off;
    off = al256(off + f2);
    L.rf = off;
    off = al256(off + f1);
    L.rg = off;
    off = al256(off + f2);
    L.pf = off;
    off = al256(off + f1);
    L.pg = off;
    off = al256(off + f2);
    L.Pp = off;
    off = al256(off + f1);
    L.part = off;
    off = al256(off + 2 * (size_t)*R * f2);
    L.sc = off;
    off = al256(off + sizeof(float) * 4 * (size_t)B);
    L.total = off;
    return L;
}

hipError_t run_sht_wide(const ShtArgs &T, hipStream_t st) {
    const dim3 rg(T.R, T.B), rblk(64 * kShtWideWaves), cg(T.d2p / kShtThreads, T.R, T.B), cblk(kShtThreads);
    hipLaunchKernelGGL(sk_sht_prep, dim3(T.B), dim3(kShuThreads), 0, st, T);
    hipLaunchKernelGGL(sk_sht_rows<true>, rg, rblk, 0, st, T);
    hipLaunchKernelGGL(sk_sht_cols<true>, cg, cblk, 0, st, T);
    hipLaunchKernelGGL(sk_sht_setup, dim3(T.B), dim3(kShuThreads), 0, st, T);
    for (int it = 0; it < T.max_cg; ++it) {
        hipLaunchKernelGGL(sk_sht_rows<false>, rg, rblk, 0, st, T);
        hipLaunchKernelGGL(sk_sht_cols<false>, cg, cblk, 0, st, T);
        hipLaunchKernelGGL(sk_sht_update, dim3(T.B), dim3(kShuThreads), 0, st, T);
    }
    hipLaunchKernelGGL(sk_sht_final, dim3(T.B), dim3(kShuThreads), 0, st, T);
    return hipGetLastError();
}

template <int NCW>
hipError_t run_sht(const ShtArgs &T, hipStream_t st) {
    const size_t lds = sizeof(float) * kShtWaves * NCW * 64;
    const dim3 grid(T.R, T.B), blk(kShtThreads);
    hipLaunchKernelGGL(sk_sht_prep, dim3(T.B), dim3(kShuThreads), 0, st, T);
    hipLaunchKernelGGL((sk_sht_sweep<NCW, true>), grid, blk, lds, st, T);
    hipLaunchKernelGGL(sk_sht_setup, dim3(T.B), dim3(kShuThreads), 0, st, T);
    for (int it = 0; it < T.max_cg; ++it) {
        hipLaunchKernelGGL((sk_sht_sweep<NCW, false>), grid, blk, lds, st, T);
        hipLaunchKernelGGL(sk_sht_update, dim3(T.B), dim3(kShuThreads), 0, st, T);
    }
    hipLaunchKernelGGL(sk_sht_final, dim3(T.B), dim3(kShuThreads), 0, st, T);
    return hipGetLastError();
}

// One chunk (at most kTiledMaxBatch problems) of the solve.
hipError_t launch_sharp_tiled_chunk(const SharpArgs &a, void *ws, hipStream_t st) {
    ShtArgs T;
    int R, RBS, d2p;
    const ShtLayout L = sht_layout(a.B, a.d1, a.d2, &R, &RBS, &d2p);
    char *base = static_cast<char *>(ws);
    T.grad_loss = a.grad_loss;
    T.mu = a.mu;
    T.nu = a.nu;
    T.C = a.C;
    T.alpha = a.alpha;
    T.beta = a.beta;
    T.grad_mu = a.grad_mu;
    T.grad_nu = a.grad_nu;
    T.cg_iters = a.cg_iters;
    T.a2 = reinterpret_cast<float *>(base + L.a2);
    T.b2 = reinterpret_cast<float *>(base + L.b2);
    T.dgf = reinterpret_cast<float *>(base + L.dgf);
    T.dgg = reinterpret_cast<float *>(base + L.dgg);
    T.xf = reinterpret_cast<float *>(base + L.xf);
    T.xg = reinterpret_cast<float *>(base + L.xg);
    T.rf = reinterpret_cast<float *>(base + L.rf);
    T.rg = reinterpret_cast<float *>(base + L.rg);
    T.pf = reinterpret_cast<float *>(base + L.pf);
    T.pg = reinterpret_cast<float *>(base + L.pg);
    T.Pp = reinterpret_cast<float *>(base + L.Pp);
    T.part = reinterpret_cast<float *>(base + L.part);
    T.sc = reinterpret_cast<float *>(base + L.sc);
    T.B = a.B;
    T.d1 = a.d1;
    T.d2 = a.d2;
    T.d2p = d2p;
    T.R = R;
    T.RBS = RBS;
    T.c_batched = a.c_batched;
    T.max_cg = a.max_cg;
    T.s = a.s;
    T.cg_tol = a.cg_tol;
    if (a.d2 > kTiledMaxD2) return run_sht_wide(T, st);
    switch (sht_ncw(a.d2)) {
        case 4: return run_sht<4>(T, st);
        case 8: return run_sht<8>(T, st);
        case 13: return run_sht<13>(T, st);
        case 16: return run_sht<16>(T, st);
        case 32: return run_sht<32>(T, st);
        default: return run_sht<64>(T, st);
    }
}

}  // namespace

size_t sharp_tiled_workspace_bytes(int B, int d1, int d2) {
    int R, RBS, d2p;
    return sht_layout(tiled_chunk(B), d1, d2, &R, &RBS, &d2p).total;
}

bool sharp_tiled_fits(int B, int d1, int d2) {
    int R, RBS;
    sht_row_blocks(tiled_chunk(B), d1, d2, &R, &RBS);
    if (R > 65535) return false;
    if (B > kTiledMaxBatch && B % kTiledMaxBatch) {
        sht_row_blocks(B % kTiledMaxBatch, d1, d2, &R, &RBS);
        if (R > 65535) return false;
    }
    return true;
}

hipError_t launch_sharp_tiled(const SharpArgs &a, void *ws, hipStream_t st) {
    return for_each_chunk(a.B, [&](int off, int n) {
        SharpArgs c = a;
        const size_t o1 = (size_t)off * a.d1, o2 = (size_t)off * a.d2;
        c.grad_loss += off;
        c.mu += o1;
        c.alpha += o1;
        c.grad_mu += o1;
        c.nu += o2;
        c.beta += o2;
        c.grad_nu += o2;
        if (a.c_batched) c.C += o1 * a.d2;
        if (a.cg_iters) c.cg_iters += off;
        c.B = n;
        return launch_sharp_tiled_chunk(c, ws, st);
    });
}

}  // namespace sk
