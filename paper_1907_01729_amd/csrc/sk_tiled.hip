// sk_tiled.hip -- the forward for supports larger than the resident kernel takes.
//
// The batch is cut into (problem, row block) work-groups.  Per iteration ONE
// sweep streams every cost row once: each wavefront takes whole rows, its 64
// lanes cover the columns (coalesced), and for a row i it
//   * builds e_ij = 2^(a_i + b_j + cl_ij) for all j and all-reduces the row sum
//     over the wavefront (DPP / lane shuffles)           -> u-update of row i,
//   * scales by f_i = 2^(a_i' - a_i) and accumulates the column sums of the
//     updated plan in registers                           -> column partials.
// (One exponential per cell per iteration; see the resident kernel for why the
// current potential is a valid logsumexp shift.)  Column partials of a
// work-group's wavefronts are combined in LDS; the row blocks' partials are
// summed in a fixed order (no float atomics) by one work-group per problem and
// 1024 columns (sk_tiled_merge_cols), which also performs the v-update and
// takes the marginal error.  The streaming sweep (per-sample cost) folds that
// merge into the start of the next sweep instead.
//
// Launch sequence for n iterations:
//   init                 a^0 = 0 on supp(mu), -inf off it; stop flags cleared
//   col_exact + merge    v-update of iteration 1: online (max, sumexp) over i
//                        per row block (Section 4's single-pass stabilised
//                        logsumexp), merged across row blocks
//   sweep(k), merge(k)   k = 1..n (no merge after the last sweep)
//   sweep(stats), final  loss E^0 and marginal error of the returned iterate,
//                        outputs in natural-log units
// Early stop (tol > 0): the merge of problem b gathers b's whole error after
// iteration k (column part summed there, by several work-groups above 1024
// columns that combine their parts in one fixed-point atomic; row part from
// the sweep's double-buffered row-block partials) and records K = k in the
// stop flag, which every later sweep and merge honours.  In the streaming sweep every
// work-group of b sums the same partials in the same order, so all take the
// same decision, and the first row block records it.
#include <stdio.h>

#include <cmath>

#include "sk_device.h"
#include "sk_internal.h"

namespace sk {
namespace {

constexpr int kThreads = 256;  // 4 wavefronts per work-group
constexpr int kWaves = kThreads / 64;
constexpr int kMergeThreads = 64;  // merge: one wavefront per (problem, 64 columns)
constexpr int kMergeColsThreads = 256;  // merge after a sweep: 4 columns per thread
constexpr int kFxCountShift = 49;       // split merge's stop accumulator: count above, sum below
constexpr float kPadCost = -1.0e30f;  // cost of cells beyond d2: plan entry 0, finite so 0*cl = 0
constexpr float kNegBig = -1.0e30f;   // finite "minus infinity" seed of the online max

struct TiledArgs {
    const float *mu, *nu, *C;
    // Point clouds instead of C (C is then null): X [B, d1, D], Y [B, d2, D];
    // cl_ij = -|rs x_i - rs y_j|^2 with rs = sqrt(log2(e) / lambda), evaluated
    // as 2 x'.y' - |x'|^2 - |y'|^2 on coordinates x' = rs (x - c_b) centred on
    // the problem's mean point c_b (ctr, [B][4], computed by sk_tiled_center).
    const float *X, *Y;
    float *ctr;
    int D;
    float rs;
    float *a;        // [B, d1] base-2 potentials (the alpha output buffer)
    float *a2;       // [B, d1] second plane of the potentials (streaming sweep: odd iterations), or null
    float *bbuf;     // [2][B, d2p] base-2 column potentials, ping-pong by iteration parity
    float *part;     // [2][R][B, d2p] column partials (plane 1 only for the exact pass)
    float *rowerr;   // [3][R][B] row-error partials: planes 0/1 by iteration parity, 2 for stats
    float *lossp;    // [R][B] loss partials (stats)
    const float *a0;  // warm start: alpha^0 [B, d1] (natural log), else null
    int32_t *state;  // [B] 0 = running, K > 0 = stopped after iteration K
    // Early stop with a compacted batch: sync[0] counts the problems stopped
    // since the running list was last rebuilt.
    int32_t *sync;
    // Compaction of the shared-cost sweep's batch (early stop only; else
    // null): order[0, nlive) lists the running problems in increasing order;
    // the identity at first, rebuilt by the merge after a problem stops.
    int32_t *order, *nlive;
    // Merge split into MS work-groups per problem (MS > 1, early stop only):
    // each adds its share of the marginal error, in fixed point, and a count
    // of one to stopacc[b] in one 64-bit atomic; the one that completes the
    // count takes the stop decision (see sk_tiled_merge_cols).
    unsigned long long *stopacc;
    int MS;
    float fx_cap;     // parts are clamped to [0, fx_cap] (NaN counts as fx_cap)
    double fx_scale;  // fixed-point units per unit of error
    double fx_tol;    // tol in fixed-point units
    float *alpha_out, *beta_out, *loss_out, *merr_out;
    int32_t *iters_out;
    int B, d1, d2, R, RBS, JC, n_iter, c_batched;
    int d2p;  // row stride of bbuf and part: d2 rounded up to the sweep's column width
              // (entries past d2 stay 0), so sweeps load and store whole rows unmasked
    float s, tol;
};

__device__ __forceinline__ size_t pidx(const TiledArgs &T, int plane, int r, int b, int j) {
    return (((size_t)plane * T.R + r) * T.B + b) * (size_t)T.d2p + j;
}

// Work-group sum in a fixed order (deterministic); `red` holds NT/64 floats.
template <int NT>
__device__ __forceinline__ float block_sum_n(float v, float *red) {
    v = wave_sum(v);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) s += red[w];
    return s;
}
__device__ __forceinline__ float block_sum(float v, float *red) { return block_sum_n<kThreads>(v, red); }

__global__ __launch_bounds__(kThreads) void sk_tiled_init(TiledArgs T) {
    const size_t n = (size_t)T.B * T.d1;
    for (size_t u = (size_t)blockIdx.x * kThreads + threadIdx.x; u < n; u += (size_t)gridDim.x * kThreads)
        T.a[u] = T.mu[u] > 0.f ? (T.a0 ? T.a0[u] * kLog2e : 0.f) : neg_inf();
    // Both planes: b^0 in plane 0 (only read when n_iter == 0), zeros past d2.
    const size_t m = (size_t)2 * T.B * T.d2p;
    for (size_t u = (size_t)blockIdx.x * kThreads + threadIdx.x; u < m; u += (size_t)gridDim.x * kThreads) {
        const size_t row = u / T.d2p;
        const int j = (int)(u - row * T.d2p);
        float v = 0.f;
        if (row < (size_t)T.B && j < T.d2 && !(T.nu[row * T.d2 + j] > 0.f)) v = neg_inf();
        T.bbuf[u] = v;
    }
    for (size_t u = (size_t)blockIdx.x * kThreads + threadIdx.x; u < (size_t)T.B; u += (size_t)gridDim.x * kThreads) {
        T.state[u] = 0;
        if (T.order) T.order[u] = (int32_t)u;
        if (T.stopacc) T.stopacc[u] = 0;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        T.sync[0] = 0;
        if (T.nlive) *T.nlive = T.B;
    }
}

// Scaled cost of one cell from the point clouds, in the centred expansion
// form every kernel uses: with x' = rs (x_i - c), y' = rs (y_j - c),
//   cl_ij = fma(2x'_0, y'_0, fma(2x'_1, y'_1, ... fma(2x'_{D-1}, y'_{D-1}, -|y'|^2))) - |x'|^2.
// Centring keeps the three terms of the size of the clouds' spread, so the
// rounding error stays that of the distance itself.
template <int DM>
__device__ __forceinline__ void centred(const float *p, const float *c, float rs, int D, float (&o)[DM]) {
#pragma unroll
    for (int k = 0; k < DM; ++k) o[k] = k < D ? rs * (p[k] - c[k]) : 0.f;
}
template <int DM>
__device__ __forceinline__ float sqnorm(const float (&o)[DM]) {
    float acc = 0.f;
#pragma unroll
    for (int k = 0; k < DM; ++k) acc = __builtin_fmaf(o[k], o[k], acc);
    return acc;
}
template <int DM>
__device__ __forceinline__ float dot2_from(const float (&x)[DM], const float (&y)[DM], float init) {
    float acc = init;
#pragma unroll
    for (int k = DM - 1; k >= 0; --k) acc = __builtin_fmaf(2.f * x[k], y[k], acc);
    return acc;
}
__device__ __forceinline__ float cl_points(const TiledArgs &T, int b, int i, int j) {
    float x[kPointsMaxD], y[kPointsMaxD];
    const float *c = T.ctr + (size_t)b * 4;
    centred(T.X + ((size_t)b * T.d1 + i) * T.D, c, T.rs, T.D, x);
    centred(T.Y + ((size_t)b * T.d2 + j) * T.D, c, T.rs, T.D, y);
    return dot2_from(x, y, -sqnorm(y)) - sqnorm(x);
}
__device__ __forceinline__ float cl_at(const TiledArgs &T, const float *Cb, int b, int i, int j) {
    return T.X ? cl_points(T, b, i, j) : -T.s * Cb[(size_t)i * T.d2 + j];
}

// v-update of iteration 1, per row block: online (max, sumexp) of
// a^0_i + cl_ij over the block's rows for every column j (one thread per
// column, reading cost rows coalesced across threads; the work-group is one
// wavefront).  A shared cost is read once for W problems: each thread carries
// the W problems' (max, sum) pairs, each updated in row order as alone.  The
// row potentials of 64 rows are loaded one per lane (-inf at zero mass: the
// row contributes nothing) and read with readlane, so the row loop waits on
// no scalar load.
template <int W>
__global__ __launch_bounds__(kMergeThreads) void sk_tiled_col_exact(TiledArgs T) {
    const int lane = threadIdx.x;
    const int j = blockIdx.x * kMergeThreads + lane;
    const int r = blockIdx.y, b0 = blockIdx.z * W;
    const int i0 = r * T.RBS, i1 = min(T.d1, i0 + T.RBS);
    const bool col_in = j < T.d2;
    const float *Cb = T.C ? T.C + (T.c_batched ? (size_t)b0 * T.d1 * T.d2 : 0) : nullptr;
    float m[W], s[W];
#pragma unroll
    for (int w = 0; w < W; ++w) {
        m[w] = kNegBig;
        s[w] = 0.f;
    }
    for (int c0 = i0; c0 < i1; c0 += 64) {
        float av[W];  // a^0 of row c0 + lane (0 unless warm-started), -inf at zero mass
#pragma unroll
        for (int w = 0; w < W; ++w) {
            const size_t u = (size_t)(b0 + w) * T.d1 + c0 + lane;
            av[w] = b0 + w < T.B && c0 + lane < i1 && T.mu[u] > 0.f ? T.a[u] : neg_inf();
        }
        const int n = min(64, i1 - c0);
        for (int q = 0; q < n; ++q) {
            const int i = c0 + q;
            // W > 1: a shared cost, the same for every problem
            const float cl = col_in ? (W > 1 ? -T.s * Cb[(size_t)i * T.d2 + j] : cl_at(T, Cb, b0, i, j)) : 0.f;
#pragma unroll
            for (int w = 0; w < W; ++w) {
                const float aw = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(av[w]), q));
                if (aw == neg_inf()) continue;  // wavefront-uniform
                const float x = aw + cl;
                const float mn = fmaxf(m[w], x);
                s[w] = s[w] * ex2(m[w] - mn) + ex2(x - mn);
                m[w] = mn;
            }
        }
    }
    if (!col_in) return;
#pragma unroll
    for (int w = 0; w < W; ++w) {
        if (b0 + w >= T.B) break;
        T.part[pidx(T, 0, r, b0 + w, j)] = m[w];
        T.part[pidx(T, 1, r, b0 + w, j)] = s[w];
    }
}

// Exact logsumexp (base 2) over all rows i of a_i + cl_ij for one column:
// the fallback of the merge when the shifted column sum left [2^-64, 2^64].
__device__ float col_lse_exact(const TiledArgs &T, int b, int j) {
    const float *Cb = T.C ? T.C + (T.c_batched ? (size_t)b * T.d1 * T.d2 : 0) : nullptr;
    const float *ab = T.a + (size_t)b * T.d1;
    float m = neg_inf();
    for (int i = 0; i < T.d1; ++i) m = fmaxf(m, ab[i] + cl_at(T, Cb, b, i, j));
    if (m == neg_inf()) return m;
    float s = 0.f;
    for (int i = 0; i < T.d1; ++i) s += ex2(ab[i] + cl_at(T, Cb, b, i, j) - m);
    return m + lg2(s);
}

// Merge of the row blocks' (max, sumexp) partials of the first v-update
// (fixed order): beta of iteration 1.
__global__ __launch_bounds__(kMergeThreads) void sk_tiled_merge_exact(TiledArgs T) {
    const int j = blockIdx.x * kMergeThreads + threadIdx.x;
    const int b = blockIdx.y;
    if (j >= T.d2) return;
    const float nuj = T.nu[(size_t)b * T.d2 + j];
    float bnew = neg_inf();
    float M = kNegBig;
    for (int r = 0; r < T.R; ++r) M = fmaxf(M, T.part[pidx(T, 0, r, b, j)]);
    float S = 0.f;
    for (int r = 0; r < T.R; ++r) S += T.part[pidx(T, 1, r, b, j)] * ex2(T.part[pidx(T, 0, r, b, j)] - M);
    if (nuj > 0.f) bnew = log2f(nuj) - (M + lg2(S));
    T.bbuf[(size_t)1 * T.B * T.d2p + (size_t)b * T.d2p + j] = bnew;
}

typedef float f4v __attribute__((ext_vector_type(4)));

// Running list of a compacted batch: order[0, nlive) = the problems with
// state 0, increasing (one work-group of NT threads, ballot prefix sums).  It
// runs beside the merges of the same launch, so a problem those merges stop
// may or may not be listed yet; the sweep skips stopped problems either way,
// and which slot a problem takes never changes its bits.
template <int NT>
__device__ void relist_running(const TiledArgs &T) {
    __shared__ int wsum[NT / 64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int base = 0;
    for (int b0 = 0; b0 < T.B; b0 += NT) {
        const int b = b0 + threadIdx.x;
        const bool live = b < T.B && T.state[b] == 0;
        const unsigned long long m = __ballot(live);
        if (lane == 0) wsum[w] = __popcll(m);
        __syncthreads();
        int off = base, tot = 0;
#pragma unroll
        for (int q = 0; q < NT / 64; ++q) {
            off += q < w ? wsum[q] : 0;
            tot += wsum[q];
        }
        if (live) T.order[off + __popcll(m & ((1ull << lane) - 1ull))] = b;
        base += tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) *T.nlive = base;
}

// Merge after sweep k (k < n_iter), work-group (b, slice) for problem b's
// columns [4 NT slice, 4 NT (slice + 1)): column sums of the plan after the
// u-update of iteration k, summed over the row blocks in a fixed order; the
// v-update of iteration k+1; iterate k's marginal error.  Each thread takes one
// group of four consecutive columns (16-byte loads of the padded rows; padding
// columns keep 0).
//
// Early stop (tol > 0): problem b's error is the column part summed here plus
// the row part from the sweep's row-block partials (added by slice 0).  With
// one slice the work-group stops b at K = k when the error is <= tol.  With
// MS slices each adds its part to stopacc[b] in one 64-bit atomic: bits 0..48
// hold the sum in fixed point (integer addition, so the total has the same
// bits whatever the order of arrival), bits 49..63 count the slices.  The
// slice whose add completes the count takes the decision from the sum; no
// work-group waits for another, and no other memory is shared between them.
// Parts are clamped to fx_cap >= 2 tol, which leaves every decision unchanged
// (a clamped part alone exceeds tol).  Every later launch skips a stopped b.
// With a compacted batch, stops are counted in sync[0], and one extra
// work-group (index B, slice 0) rebuilds the running list from the stops of
// earlier launches when the count is nonzero.
template <int NT>
__global__ __launch_bounds__(NT) void sk_tiled_merge_cols(TiledArgs T, int k) {
    __shared__ float red[NT / 64];
    const int b = blockIdx.x, sl = blockIdx.y;
    if (b == T.B) {  // the relist work-group of a compacted batch
        if (sl != 0) return;
        const int seen = T.sync[0];
        if (seen == 0) return;  // nothing stopped since the last rebuild
        relist_running<NT>(T);
        if (threadIdx.x == 0) atomicSub(&T.sync[0], seen);
        return;
    }
    if (T.state[b] != 0) return;  // block-uniform
    const size_t rstride = (size_t)T.B * T.d2p / 4;  // one row block, in f4v
    float err = 0.f;
    const int j0 = 4 * (sl * NT + (int)threadIdx.x);
    if (j0 < T.d2) {
        const f4v *col = reinterpret_cast<const f4v *>(T.part + pidx(T, 0, 0, b, j0));
        f4v cs = {0.f, 0.f, 0.f, 0.f};
        for (int r0 = 0; r0 < T.R; r0 += 16) {
            f4v v[16];
#pragma unroll
            for (int q = 0; q < 16; ++q)
                v[q] = r0 + q < T.R ? col[(size_t)(r0 + q) * rstride] : f4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < 16; ++q) cs += v[q];
        }
        const f4v bold = *reinterpret_cast<const f4v *>(T.bbuf + (size_t)(k & 1) * T.B * T.d2p + (size_t)b * T.d2p + j0);
        f4v bnew;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int j = j0 + c;
            float v = 0.f;  // padding columns
            if (j < T.d2) {
                const float nuj = T.nu[(size_t)b * T.d2 + j];
                err += fabsf(cs[c] - nuj);
                v = neg_inf();
                if (nuj > 0.f) {
                    if (cs[c] >= kSumLo && cs[c] <= kSumHi)
                        v = bold[c] + log2f(nuj) - lg2(cs[c]);
                    else
                        v = log2f(nuj) - col_lse_exact(T, b, j);
                }
            }
            bnew[c] = v;
        }
        *reinterpret_cast<f4v *>(T.bbuf + (size_t)((k + 1) & 1) * T.B * T.d2p + (size_t)b * T.d2p + j0) = bnew;
    }
    if (!(T.tol > 0.f)) return;
    if (sl == 0) {
        const float *re = T.rowerr + (size_t)(k & 1) * T.R * T.B;
        for (int q = threadIdx.x; q < T.R; q += NT) err += re[(size_t)q * T.B + b];
    }
    err = block_sum_n<NT>(err, red);
    if (threadIdx.x != 0) return;
    bool stop = err <= T.tol;
    if (T.MS > 1) {
        const float part = err <= T.fx_cap ? err : T.fx_cap;  // NaN -> fx_cap
        const unsigned long long add =
            (1ull << kFxCountShift) + (unsigned long long)__builtin_rint((double)part * T.fx_scale);
        const unsigned long long got = atomicAdd(T.stopacc + b, add) + add;
        if ((got >> kFxCountShift) != (unsigned long long)T.MS) return;
        T.stopacc[b] = 0;  // for the next merge (a later launch)
        stop = (double)(got & ((1ull << kFxCountShift) - 1ull)) <= T.fx_tol;
    }
    if (stop) {
        T.state[b] = k;
        if (T.order) atomicAdd(&T.sync[0], 1);
    }
}

// Cost of this lane's columns j = lane + 64 c of one row, read from global
// memory and scaled on the fly (kPadCost beyond d2).  A per-sample cost is
// streamed once per iteration, so it bypasses the caches.
template <bool BATCHED>
struct GlobalCost {
    const float *row;
    int lane, d2;
    float s;
    __device__ __forceinline__ float operator()(int c) const {
        const int j = lane + 64 * c;
        if (j >= d2) return kPadCost;
        return -s * (BATCHED ? __builtin_nontemporal_load(row + j) : row[j]);
    }
};
// The same from a row staged (already scaled and padded) in LDS.
struct LdsCost {
    const float *row;  // already offset by lane
    __device__ __forceinline__ float operator()(int c) const { return row[64 * c]; }
};

// One cost row i of one problem in one wavefront: e_j = 2^(a_i + b_j + cl_ij),
// row sum by wavefront all-reduce, u-update of a_i, and the column sums of the
// updated plan accumulated into colpart.  STATS: the plan of the current (a, b)
// without update, with sum P*cl.  rowerr (wavefront-uniform) gathers the rows'
// marginal error.
template <int NCW, bool STATS, class Cost>
__device__ __forceinline__ void row_step(const Cost &cost, float ai, float mui, float *a_row,
                                         const float (&bv)[NCW], float (&colpart)[NCW], float &rowerr,
                                         float &losspart, int lane) {
    float e[NCW];
#pragma unroll
    for (int c = 0; c < NCW; ++c) e[c] = cost(c);
#pragma unroll
    for (int c = 0; c < NCW; ++c) {
        const float cl = e[c];
        const float v = ex2((ai + bv[c]) + cl);
        if (STATS) losspart = __builtin_fmaf(v, cl, losspart);
        e[c] = v;
    }
    const float rs = wave_sum(tree_sum<NCW>(e));
    if (STATS) {
        if (mui > 0.f) rowerr += fabsf(rs - mui);
#pragma unroll
        for (int c = 0; c < NCW; ++c) colpart[c] += e[c];
        return;
    }
    if (!(mui > 0.f)) return;  // zero-mass row: a_i = -inf, all its entries 0
    const float lmu = log2f(mui);
    float an, f;
    if (rs >= kSumLo && rs <= kSumHi) {
        an = ai + lmu - lg2(rs);
        f = ex2(an - ai);
        rowerr += fabsf(f * rs - mui);
    } else {
        // Exact u-update of this row (max, then sum), plan entries rebuilt
        // from the new potential.
        float m = neg_inf();
#pragma unroll
        for (int c = 0; c < NCW; ++c) m = fmaxf(m, bv[c] + cost(c));
        m = wave_max(m);
        float s2 = 0.f;
#pragma unroll
        for (int c = 0; c < NCW; ++c) s2 += ex2(bv[c] + cost(c) - m);
        s2 = wave_sum(s2);
        an = lmu - (m + lg2(s2));
#pragma unroll
        for (int c = 0; c < NCW; ++c) e[c] = ex2((an + bv[c]) + cost(c));
        f = 1.f;
        rowerr += fabsf(wave_sum(tree_sum<NCW>(e)) - mui);
    }
#pragma unroll
    for (int c = 0; c < NCW; ++c) colpart[c] = __builtin_fmaf(e[c], f, colpart[c]);
    if (lane == 0) *a_row = an;
}

// Sweep, one problem per work-group (per-sample costs, or tiny batches).
// Work-group (row block r, problem b); wavefront w takes rows i0 + w,
// i0 + w + 4, ...; lane l owns columns j = l + 64 c, c < NCW.  The
// wavefronts' column partials are combined in LDS in a fixed order.
template <int NCW, bool STATS, bool BATCHED>
__global__ __launch_bounds__(kThreads) void sk_tiled_sweep(TiledArgs T, int k) {
    extern __shared__ float lds[];  // [kWaves][NCW*64] column partials
    __shared__ float scal[2 * kWaves];
    const int r = blockIdx.x, b = blockIdx.y;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int d1 = T.d1, d2 = T.d2;

    const int st = T.state[b];
    if (!STATS && st != 0) return;  // stopped by an earlier merge's test
    const int K = STATS ? (st ? st : T.n_iter) : k;
    const float *bsrc = T.bbuf + (size_t)(K & 1) * T.B * T.d2p + (size_t)b * T.d2p;
    const float *Cb = T.C + (T.c_batched ? (size_t)b * d1 * d2 : 0);
    float *ab = T.a + (size_t)b * d1;
    const float *mub = T.mu + (size_t)b * d1;

    float bv[NCW], colpart[NCW];
#pragma unroll
    for (int c = 0; c < NCW; ++c) {
        const int j = lane + 64 * c;
        bv[c] = bsrc[j];  // 0 past d2 (padded stride)
        colpart[c] = 0.f;
    }
    float rowerr = 0.f, losspart = 0.f;
    const int i0 = r * T.RBS, i1 = min(d1, i0 + T.RBS);
    for (int i = i0 + w; i < i1; i += kWaves) {
        const GlobalCost<BATCHED> cost{Cb + (size_t)i * d2, lane, d2, T.s};
        row_step<NCW, STATS>(cost, ab[i], mub[i], ab + i, bv, colpart, rowerr, losspart, lane);
    }

    // Combine the wavefronts' partials in LDS, fixed order, and store.
#pragma unroll
    for (int c = 0; c < NCW; ++c) lds[w * NCW * 64 + c * 64 + lane] = colpart[c];
    // rowerr is wavefront-uniform (built from all-reduced sums); losspart is per lane
    const float lw = STATS ? wave_sum(losspart) : 0.f;
    if (lane == 0) {
        scal[w] = rowerr;
        scal[kWaves + w] = lw;
    }
    __syncthreads();
    for (int j = threadIdx.x; j < d2; j += kThreads) {
        float s = 0.f;
#pragma unroll
        for (int q = 0; q < kWaves; ++q) s += lds[q * NCW * 64 + j];
        T.part[pidx(T, 0, r, b, j)] = s;
    }
    if (threadIdx.x == 0) {
        float re = 0.f, lo = 0.f;
#pragma unroll
        for (int q = 0; q < kWaves; ++q) {
            re += scal[q];
            lo += scal[kWaves + q];
        }
        const int plane = STATS ? 2 : (k & 1);
        T.rowerr[((size_t)plane * T.R + r) * T.B + b] = re;
        if (STATS) T.lossp[(size_t)r * T.B + b] = lo;
    }
}

// ---- Rows wider than one wavefront's registers hold (d2 > kTiledMaxD2) ----
//
// The one-pass sweeps keep a row's plan entries in registers between its row
// sum and its column sums.  A wider row takes two passes per iteration over
// the cost, one exponential per cell in each, with the same shifted sums and
// exact fallbacks (so the same iterates):
//   sk_wide_rows  one wavefront per row, looping over the columns: the row
//                 sum of the plan after the last v-update, the u-update in
//                 place, the row part of the marginal error;
//   sk_wide_cols  one thread per column, looping over a row block: the column
//                 partials of the plan after that u-update, merged by
//                 sk_tiled_merge_cols like every other sweep's.
// STATS: the plan of the returned iterate, without update (row error and
// loss partials, column partials) for sk_tiled_final.
constexpr int kWideRowWaves = 16;  // rows kernel: 16 wavefronts, one row each at a time

template <bool STATS>
__global__ __launch_bounds__(64 * kWideRowWaves) void sk_wide_rows(TiledArgs T, int k) {
    __shared__ float scal[2 * kWideRowWaves];
    const int r = blockIdx.x, b = blockIdx.y;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int st = T.state[b];
    if (!STATS && st != 0) return;  // stopped by an earlier merge's test (block-uniform)
    const int K = STATS ? (st ? st : T.n_iter) : k;
    const int d1 = T.d1, d2 = T.d2;
    const float s = T.s;
    const float *bsrc = T.bbuf + (size_t)(K & 1) * T.B * T.d2p + (size_t)b * T.d2p;
    const float *Cb = T.C + (T.c_batched ? (size_t)b * d1 * d2 : 0);
    float *ab = T.a + (size_t)b * d1;
    const float *mub = T.mu + (size_t)b * d1;
    float rowerr = 0.f, losspart = 0.f;  // rowerr wavefront-uniform, losspart per lane
    const int i0 = r * T.RBS, i1 = min(d1, i0 + T.RBS);
    for (int i = i0 + w; i < i1; i += kWideRowWaves) {
        const float mui = mub[i];
        if (!STATS && !(mui > 0.f)) continue;  // zero-mass row: a_i = -inf, its entries 0
        const float ai = ab[i];
        const float *row = Cb + (size_t)i * d2;
        float acc = 0.f;
        for (int j = lane; j < d2; j += 64) {
            const float cl = -s * row[j];
            const float v = ex2((ai + bsrc[j]) + cl);
            acc += v;
            if (STATS) losspart = __builtin_fmaf(v, cl, losspart);
        }
        const float rs = wave_sum(acc);
        if (STATS) {
            if (mui > 0.f) rowerr += fabsf(rs - mui);
            continue;
        }
        const float lmu = log2f(mui);
        float an;
        if (rs >= kSumLo && rs <= kSumHi) {
            an = ai + lmu - lg2(rs);
            rowerr += fabsf(ex2(an - ai) * rs - mui);
        } else {
            // Exact u-update of this row (max, then sum); the row error from
            // the entries rebuilt with the new potential.
            float m = neg_inf();
            for (int j = lane; j < d2; j += 64) m = fmaxf(m, bsrc[j] - s * row[j]);
            m = wave_max(m);
            float s2 = 0.f;
            for (int j = lane; j < d2; j += 64) s2 += ex2(bsrc[j] - s * row[j] - m);
            an = lmu - (m + lg2(wave_sum(s2)));
            float s3 = 0.f;
            for (int j = lane; j < d2; j += 64) s3 += ex2((an + bsrc[j]) - s * row[j]);
            rowerr += fabsf(wave_sum(s3) - mui);
        }
        if (lane == 0) ab[i] = an;
    }
    const float lw = STATS ? wave_sum(losspart) : 0.f;
    if (lane == 0) {
        scal[w] = rowerr;
        scal[kWideRowWaves + w] = lw;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float re = 0.f, lo = 0.f;
#pragma unroll
        for (int q = 0; q < kWideRowWaves; ++q) {
            re += scal[q];
            lo += scal[kWideRowWaves + q];
        }
        const int plane = STATS ? 2 : (k & 1);
        T.rowerr[((size_t)plane * T.R + r) * T.B + b] = re;
        if (STATS) T.lossp[(size_t)r * T.B + b] = lo;
    }
}

// Column partials over row block r of the plan (a, b) (after the rows pass's
// u-update; STATS: the returned iterate), one thread per column; the entries
// past d2 are written 0.  Four rows per step in separate accumulators, summed
// in a fixed order.
template <bool STATS>
__global__ __launch_bounds__(kThreads) void sk_wide_cols(TiledArgs T, int k) {
    const int j = blockIdx.x * kThreads + threadIdx.x;
    const int r = blockIdx.y, b = blockIdx.z;
    const int st = T.state[b];
    if (!STATS && st != 0) return;  // block-uniform
    const int K = STATS ? (st ? st : T.n_iter) : k;
    const int d1 = T.d1, d2 = T.d2;
    const int i0 = r * T.RBS, i1 = min(d1, i0 + T.RBS);
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    if (j < d2) {
        const float s = T.s;
        const float bj = T.bbuf[(size_t)(K & 1) * T.B * T.d2p + (size_t)b * T.d2p + j];
        const float *col = T.C + (T.c_batched ? (size_t)b * d1 * d2 : 0) + j;
        const float *ab = T.a + (size_t)b * d1;
        int i = i0;
        for (; i + 4 <= i1; i += 4) {
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[q] += ex2((ab[i + q] + bj) - s * col[(size_t)(i + q) * d2]);
        }
        for (; i < i1; ++i) acc[0] += ex2((ab[i] + bj) - s * col[(size_t)i * d2]);
    }
    T.part[pidx(T, 0, r, b, j)] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

// Mean point of each problem's two clouds (fixed-order sums): the centre of
// the expansion form above.  One work-group per problem.
__global__ __launch_bounds__(kThreads) void sk_tiled_center(TiledArgs T) {
    __shared__ float red[kWaves];
    const int b = blockIdx.x;
    for (int k = 0; k < T.D; ++k) {
        float acc = 0.f;
        for (int i = threadIdx.x; i < T.d1; i += kThreads) acc += T.X[((size_t)b * T.d1 + i) * T.D + k];
        for (int j = threadIdx.x; j < T.d2; j += kThreads) acc += T.Y[((size_t)b * T.d2 + j) * T.D + k];
        acc = block_sum(acc, red);
        if (threadIdx.x == 0) T.ctr[(size_t)b * 4 + k] = acc / (float)(T.d1 + T.d2);
    }
}

// Padding columns sit at kFarCoord: |y'|^2 = 3e36, the plan entry is 0 and
// the cost finite (0 * cl = 0).
constexpr float kFarCoord = 1.0e18f;

// RB rows of a point-cloud problem in one wavefront (the structure of
// row_step, with the rows' reductions interleaved so their latencies
// overlap): u_c = b_j + cl_ij + |x'_i|^2 = fma chain of 2x'.y' on
// bp_c = b_j - |y'_j|^2, so a cell costs three fmas, one add and the exp2.
// Row q takes part only if live[q] (wavefront-uniform).
template <int NCW, int D, int RB, bool STATS>
__device__ __forceinline__ void rows_step_points(const float (&ys)[NCW][D], const float (&bp)[NCW],
                                                 const float (&xc)[RB][D], const float (&ai)[RB],
                                                 const float (&mui)[RB], const bool (&live)[RB], float *const (&a_row)[RB],
                                                 float (&colpart)[NCW], float &rowerr, float &losspart, int lane) {
    float xx[RB], e[RB][NCW], rs[RB];
    __builtin_amdgcn_s_setprio(0);  // exponentials low, the row reductions high
#pragma unroll
    for (int q = 0; q < RB; ++q) {
        xx[q] = sqnorm(xc[q]);
        const float ax = ai[q] - xx[q];
#pragma unroll
        for (int c = 0; c < NCW; ++c) e[q][c] = live[q] ? ex2(dot2_from(xc[q], ys[c], bp[c]) + ax) : 0.f;
    }
    __builtin_amdgcn_s_setprio(3);
#pragma unroll
    for (int q = 0; q < RB; ++q) rs[q] = wave_sum(tree_sum<NCW>(e[q]));
    if (STATS) {
#pragma unroll
        for (int q = 0; q < RB; ++q) {
#pragma unroll
            for (int c = 0; c < NCW; ++c) {
                const float cl = dot2_from(xc[q], ys[c], -sqnorm(ys[c])) - xx[q];
                losspart = __builtin_fmaf(e[q][c], cl, losspart);
                colpart[c] += e[q][c];
            }
            if (live[q] && mui[q] > 0.f) rowerr += fabsf(rs[q] - mui[q]);
        }
        return;
    }
    float f[RB];
#pragma unroll
    for (int q = 0; q < RB; ++q) {
        f[q] = 0.f;  // zero-mass or idle row: a_i = -inf, all its entries 0
        if (!live[q] || !(mui[q] > 0.f)) continue;
        const float lmu = log2f(mui[q]);
        float an;
        if (rs[q] >= kSumLo && rs[q] <= kSumHi) {
            an = ai[q] + lmu - lg2(rs[q]);
            f[q] = ex2(an - ai[q]);
            rowerr += fabsf(f[q] * rs[q] - mui[q]);
        } else {
            // Exact u-update (max, then sum) over b_j + cl_ij = u_c - |x'|^2
            // (u_c recomputed in each pass: this path is rare and keeps
            // no extra registers).
            float m = neg_inf();
#pragma unroll
            for (int c = 0; c < NCW; ++c) m = fmaxf(m, dot2_from(xc[q], ys[c], bp[c]));
            m = wave_max(m);
            float s2 = 0.f;
#pragma unroll
            for (int c = 0; c < NCW; ++c) s2 += ex2(dot2_from(xc[q], ys[c], bp[c]) - m);
            s2 = wave_sum(s2);
            an = lmu - ((m - xx[q]) + lg2(s2));
            const float ax2 = an - xx[q];
#pragma unroll
            for (int c = 0; c < NCW; ++c) e[q][c] = ex2(dot2_from(xc[q], ys[c], bp[c]) + ax2);
            f[q] = 1.f;
            rowerr += fabsf(wave_sum(tree_sum<NCW>(e[q])) - mui[q]);
        }
        if (lane == 0) *a_row[q] = an;
    }
#pragma unroll
    for (int c = 0; c < NCW; ++c) {
        float acc = colpart[c];
#pragma unroll
        for (int q = 0; q < RB; ++q) acc = __builtin_fmaf(e[q][c], f[q], acc);
        colpart[c] = acc;
    }
}

// Rows reduced together by the points sweep (their plan entries stay in
// registers until the row sums are known).
template <int NCW>
struct PointsShape {
    static constexpr int RB = NCW <= 8 ? 4 : (NCW <= 16 ? 2 : 1);
};

// Sweep over per-sample point clouds (the on-the-fly cost of Section 4's
// closing remark: cost entries are recreated from the points, no cost matrix
// exists).  Work-group (row block r, problem b) as in sk_tiled_sweep; lane l
// keeps the centred, scaled coordinates of its columns j = l + 64 c in
// registers.  The row's coordinates, potential and mass are loaded one row
// ahead (vector loads through a lane-varying index, kept in flight over the
// current row's work).
template <int NCW, int D, bool STATS>
__global__ __launch_bounds__(kThreads) void sk_tiled_sweep_points(TiledArgs T, int k) {
    extern __shared__ float lds[];  // [kWaves][NCW*64] column partials
    __shared__ float scal[2 * kWaves];
    const int r = blockIdx.x, b = blockIdx.y;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int d1 = T.d1, d2 = T.d2;

    const int st = T.state[b];
    if (!STATS && st != 0) return;  // stopped by an earlier merge's test
    const int K = STATS ? (st ? st : T.n_iter) : k;
    const float *bsrc = T.bbuf + (size_t)(K & 1) * T.B * T.d2p + (size_t)b * T.d2p;
    float *ab = T.a + (size_t)b * d1;
    const float *mub = T.mu + (size_t)b * d1;
    const float *xb = T.X + (size_t)b * d1 * D;
    const float *yb = T.Y + (size_t)b * d2 * D;
    const float rs = T.rs;
    float cen[D];  // the centre, in registers (a memory operand would be re-read after every store)
#pragma unroll
    for (int q = 0; q < D; ++q) cen[q] = T.ctr[(size_t)b * 4 + q];

    // The columns' raw coordinates first (clamped index: all loads in
    // flight together), then centred and scaled; padding columns go far away.
    float bp[NCW], colpart[NCW], ys[NCW][D];
#pragma unroll
    for (int c = 0; c < NCW; ++c) {
        const int jj = min(lane + 64 * c, d2 - 1);
#pragma unroll
        for (int q = 0; q < D; ++q) ys[c][q] = yb[(size_t)jj * D + q];
        bp[c] = bsrc[lane + 64 * c];  // 0 past d2 (padded stride)
    }
#pragma unroll
    for (int c = 0; c < NCW; ++c) {
        const bool in = lane + 64 * c < d2;
#pragma unroll
        for (int q = 0; q < D; ++q) ys[c][q] = in ? rs * (ys[c][q] - cen[q]) : kFarCoord;
        bp[c] -= sqnorm(ys[c]);
        colpart[c] = 0.f;
    }
    // Rows i0 + w + kWaves t, RB at a time; the next batch's coordinates,
    // potentials and masses are loaded one batch ahead.
    constexpr int RB = PointsShape<NCW>::RB;
    int vz = 0;
    __asm__ volatile("" : "+v"(vz));  // a zero the compiler cannot see as uniform
    float xn[RB][D], an[RB], mn[RB];
    const int i0 = r * T.RBS, i1 = min(d1, i0 + T.RBS);
    // Raw values only: the arithmetic on them waits for the next batch, so
    // the loads stay in flight over this batch's work.
    auto load_rows = [&](int i) {
#pragma unroll
        for (int q = 0; q < RB; ++q) {
            const int ii = min(i + q * kWaves, i1 - 1) + vz;  // an idle slot re-reads the last row
#pragma unroll
            for (int d = 0; d < D; ++d) xn[q][d] = xb[(size_t)ii * D + d];
            an[q] = ab[ii];
            mn[q] = mub[ii];
        }
    };
    float rowerr = 0.f, losspart = 0.f;
    if (i0 + w < i1) load_rows(i0 + w);
    for (int i = i0 + w; i < i1; i += RB * kWaves) {
        float xc[RB][D], ai[RB], mui[RB];
        bool live[RB];
        float *arow[RB];
#pragma unroll
        for (int q = 0; q < RB; ++q) {
#pragma unroll
            for (int d = 0; d < D; ++d) xc[q][d] = rs * (xn[q][d] - cen[d]);
            ai[q] = an[q];
            mui[q] = mn[q];
            live[q] = i + q * kWaves < i1;
            arow[q] = ab + min(i + q * kWaves, i1 - 1);
        }
        // Other rows of this wavefront (no conflict with the stores below);
        // unconditional, clamped to the last row, so the waits stay exact.
        load_rows(i + RB * kWaves);
        rows_step_points<NCW, D, RB, STATS>(ys, bp, xc, ai, mui, live, arow, colpart, rowerr, losspart, lane);
    }

    // Combine the wavefronts' partials in LDS, fixed order, and store.
#pragma unroll
    for (int c = 0; c < NCW; ++c) lds[w * NCW * 64 + c * 64 + lane] = colpart[c];
    const float lw = STATS ? wave_sum(losspart) : 0.f;
    if (lane == 0) {
        scal[w] = rowerr;
        scal[kWaves + w] = lw;
    }
    __syncthreads();
    for (int j = threadIdx.x; j < d2; j += kThreads) {
        float sum = 0.f;
#pragma unroll
        for (int q = 0; q < kWaves; ++q) sum += lds[q * NCW * 64 + j];
        T.part[pidx(T, 0, r, b, j)] = sum;
    }
    if (threadIdx.x == 0) {
        float re = 0.f, lo = 0.f;
#pragma unroll
        for (int q = 0; q < kWaves; ++q) {
            re += scal[q];
            lo += scal[kWaves + q];
        }
        const int plane = STATS ? 2 : (k & 1);
        T.rowerr[((size_t)plane * T.R + r) * T.B + b] = re;
        if (STATS) T.lossp[(size_t)r * T.B + b] = lo;
    }
}

// Sweep for a cost shared by the batch (Section 4's setting).
//
// A work-group of W wavefronts = W problems of group g walks the rows of row
// block r.  Chunks of RS raw cost rows are copied into LDS by direct
// global->LDS loads (no registers, no VALU work), double-buffered: the next
// chunk is in flight while the current one is computed, and every staged
// element is read by all W wavefronts, so the cost leaves L2 once per W
// problems.  Work-groups of the same row block share an XCD (block index
// r + R g with R a multiple of 8), so a row block leaves HBM once.
//
// Per cell: one add (a_i + b_j), one fma (- s C_ij), one exp, one add (row
// sum) and one fma (column sum).  RB rows are reduced together: their row
// sums share one transposed wavefront all-reduce (permlane swaps pack the RB
// partial vectors into one register before the 16-lane DPP stages).  The row
// potentials a_i and log2 mu_i of 64 rows sit in one register each (lane =
// row), are read with readlane and prefetched a segment ahead; the updated
// a_i are collected the same way and stored once per 64 rows.
constexpr float kPadC = 1.0e30f;  // raw cost of padding cells: exp underflows to 0, 0 * cl stays finite
constexpr int kSegs = 4;          // row blocks of the shared-cost sweep hold at most 64 kSegs rows

// All-reduce of RB per-lane partials (RB = 1, 2 or 4).  Packing: a permlane32
// swap pairs (p0, p1) so that lanes < 32 carry p0's half-sums and lanes >= 32
// p1's; a permlane16 swap then packs four vectors into the four 16-lane rows
// (p0, p2, p1, p3); the 16-lane DPP stages finish every row at once, each
// lane of a row with the same bits.
__device__ __forceinline__ LanePair swap32x(float x, float y) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(y), false, false);
    return {__uint_as_float(r[0]), __uint_as_float(r[1])};
}
__device__ __forceinline__ LanePair swap16x(float x, float y) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(y), false, false);
    return {__uint_as_float(r[0]), __uint_as_float(r[1])};
}
__device__ __forceinline__ float sum16(float v) {  // all-reduce within each 16-lane row
    v = sum_q(v);
    return v + dpp<kRowRor8>(v);
}
__device__ __forceinline__ float uni(float v, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}
// The result stays in the packed layout: the 16-lane group (lane >> 4) holds
// the sum of row row_of_lane(lane); lane_of_row(q) is the first lane holding
// row q.
template <int RB>
__device__ __forceinline__ float allreduce_rows_packed(const float (&p)[RB]) {
    if constexpr (RB == 1) {
        return wave_sum(p[0]);
    } else if constexpr (RB == 2) {
        const LanePair a = swap32x(p[0], p[1]);
        const LanePair b = swap16(a.lo + a.hi);
        return sum16(b.lo + b.hi);
    } else {
        static_assert(RB == 4, "RB must be 1, 2 or 4");
        const LanePair a = swap32x(p[0], p[1]);
        const LanePair b = swap32x(p[2], p[3]);
        const LanePair c = swap16x(a.lo + a.hi, b.lo + b.hi);
        return sum16(c.lo + c.hi);
    }
}
template <int RB>
__device__ __forceinline__ int row_of_lane(int lane) {
    return RB == 4 ? ((lane >> 4) & 1) * 2 + (lane >> 5) : (RB == 2 ? lane >> 5 : 0);
}
template <int RB>
__device__ __forceinline__ int lane_of_row(int q) {
    return RB == 4 ? (q & 1) * 32 + (q >> 1) * 16 : (RB == 2 ? 32 * q : 0);
}
// Value of register v in lane src (any lane, per-lane index).
__device__ __forceinline__ float lane_get(float v, int src) {
    return __int_as_float(__builtin_amdgcn_ds_bpermute(src << 2, __float_as_int(v)));
}

template <int NCW, int W, int RS, int RB, bool VEC4, bool STATS>
__global__ __launch_bounds__(64 * W) void sk_tiled_sweep_shared(TiledArgs T, int k) {
    constexpr int D2P = NCW * 64;  // LDS row length (columns beyond d2 hold kPadC)
    constexpr int NT = 64 * W;
    constexpr int VW = VEC4 ? 4 : 1;  // floats per lane per global->LDS load
    static_assert(RS % RB == 0 && 64 % RS == 0, "chunks must tile 64-row segments");
    extern __shared__ float lds[];  // [2][RS][D2P]
    const int r = blockIdx.x, g = blockIdx.y;
    // The wavefront index is uniform: read it into a scalar register so that
    // everything derived from it (problem, staging assignments) is scalar.
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int d1 = T.d1, d2 = T.d2;
    // Problem of this wavefront: slot g W + w of the running list when the
    // batch is compacted, else problem g W + w.
    const bool compacted = !STATS && T.order;
    const int slot = g * W + w;
    const int nslot = compacted ? __builtin_amdgcn_readfirstlane(*T.nlive) : T.B;
    const int b_raw = slot < nslot ? (compacted ? __builtin_amdgcn_readfirstlane(T.order[slot]) : slot) : T.B;
    // Inactive wavefronts (past the batch, or stopped) keep staging and
    // reaching the barriers; they compute nothing and store nothing.
    const int b = b_raw < T.B ? b_raw : T.B - 1;
    const int st = T.state[b];
    const bool skip = b_raw >= T.B || (!STATS && st != 0);
    if (!__syncthreads_or(!skip)) return;

    // Columns past d2 hold the padding cost (plan entries exactly 0); loads
    // never touch them.  Rows past the block are never read (see below).
    if (d2 < D2P)
        for (int u = threadIdx.x; u < 2 * RS * (D2P - d2); u += NT)
            lds[(u / (D2P - d2)) * D2P + d2 + u % (D2P - d2)] = kPadC;
    __syncthreads();

    const int i0 = r * T.RBS, i1 = min(d1, i0 + T.RBS);
    const int nrows = i1 - i0;
    const int nchunk = (nrows + RS - 1) / RS;
    const int lpr = (d2 + 64 * VW - 1) / (64 * VW);  // wavefront loads per cost row
    // Wavefront w issues the loads (row rr, 64-lane segment sg) numbered
    // w, w + W, w + 2W, ... of the chunk (scalar index arithmetic).
    const int ld_rr0 = w / lpr, ld_sg0 = w - (w / lpr) * lpr;
    auto issue_chunk = [&](int ch) {
        float *base = lds + (ch & 1) * RS * D2P;
        int rr = ld_rr0, sg = ld_sg0;
        for (int q = w; q < RS * lpr; q += W) {
            const int i = i0 + ch * RS + rr;
            const int u = sg * 64 + lane;
            if (i < i1 && u * VW < d2) {
                const float *src = T.C + (size_t)i * d2 + (size_t)u * VW;
                auto *dst = (__attribute__((address_space(3))) void *)(base + rr * D2P + sg * 64 * VW);
                if constexpr (VEC4)
                    __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
                else
                    __builtin_amdgcn_global_load_lds(src, dst, 4, 0, 0);
            }
            for (sg += W; sg >= lpr; sg -= lpr) ++rr;
        }
    };
    issue_chunk(0);

    const int K = STATS ? (st ? st : T.n_iter) : k;
    const float *bsrc = T.bbuf + (size_t)(K & 1) * T.B * T.d2p + (size_t)b * T.d2p;
    float *ab = T.a + (size_t)b * d1;
    const float *mub = T.mu + (size_t)b * d1;
    const float ns = -T.s;
    float bv[NCW], colpart[NCW];
#pragma unroll
    for (int c = 0; c < NCW; ++c) {
        const int j = lane + 64 * c;
        bv[c] = bsrc[j];  // 0 past d2 (padded stride)
        colpart[c] = 0.f;
    }
    // Row state of the block, 64 rows per register (lane = row), loaded
    // before the first barrier; row blocks of this sweep have <= 64 kSegs rows.
    float a_s[kSegs], mu_s[kSegs];
#pragma unroll
    for (int q = 0; q < kSegs; ++q) {
        const int i = i0 + 64 * q + lane;
        a_s[q] = i < i1 ? ab[i] : neg_inf();
        mu_s[q] = i < i1 ? mub[i] : 0.f;
    }
    float a_seg = 0.f, mu_seg = 0.f, lmu_seg = 0.f, a_out = 0.f;
    float rowerr = 0.f, losspart = 0.f;

    for (int ch = 0; ch < nchunk; ++ch) {
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wavefront's loads of chunk ch have landed
        __syncthreads();                     // ... and every other wavefront's
        if (ch + 1 < nchunk) issue_chunk(ch + 1);
        const float *cbuf = lds + (ch & 1) * RS * D2P + lane;
        // One row per batch (the widest rows): the next row's first 4 staged
        // values are read before this row's reduction, so their latency is
        // hidden instead of exposed at the next row's start (1.8 % on 4096
        // columns).  Narrower rows gain too little to pay its registers.
        constexpr int PF = 4;
        float pre[PF];
#pragma unroll
        for (int rb = 0; rb < RS; rb += RB) {
            const int rel = ch * RS + rb;
            if (rel >= nrows) break;
            if ((rel & 63) == 0) {  // next 64-row segment
                const int sg = rel >> 6;
                a_seg = a_s[0];
                mu_seg = mu_s[0];
#pragma unroll
                for (int q = 1; q < kSegs; ++q) {
                    a_seg = sg == q ? a_s[q] : a_seg;
                    mu_seg = sg == q ? mu_s[q] : mu_seg;
                }
                lmu_seg = mu_seg > 0.f ? lg2(mu_seg) : neg_inf();
                a_out = a_seg;
            }
            if (!skip) {
                const int rr0 = rel & 63;
                float ai[RB], e[RB][NCW], p[RB], f[RB];
                // The staged cost values of the batch go into the plan-entry
                // registers and are turned into plan entries in place, in
                // groups of G: group g + 1 is read from LDS while group g's
                // exponentials run, so the LDS reads of every wavefront spread
                // over its arithmetic instead of stalling it once per batch.
                // Rows past the block (a = -inf) read the batch's first row,
                // which is staged.
                constexpr int NE = RB * NCW, G = RB > 1 ? NCW : 16, NG = (NE + G - 1) / G;
                int rq[RB];
#pragma unroll
                for (int q = 0; q < RB; ++q) {
                    rq[q] = rel + q < nrows ? rb + q : rb;
                    ai[q] = uni(a_seg, rr0 + q);
                }
                auto read_group = [&](int g) {
#pragma unroll
                    for (int n = g * G; n < (g + 1) * G && n < NE; ++n)
                        e[n / NCW][n % NCW] = cbuf[rq[n / NCW] * D2P + 64 * (n % NCW)];
                };
                if (RB == 1 && rb > 0) {  // group 0 of the batch is row rb's first G values
#pragma unroll
                    for (int n = 0; n < PF; ++n) e[0][n] = pre[n];
#pragma unroll
                    for (int n = PF; n < G; ++n) e[0][n] = cbuf[rb * D2P + 64 * n];
                } else {
                    read_group(0);
                }
                __builtin_amdgcn_sched_barrier(0);
                // Issue priority falls with the batch's place in the chunk
                // (3 for the first rows, 0 for the last): of the wavefronts
                // sharing a SIMD, the one behind issues first, so they reach
                // the chunk's barrier together instead of the oldest one
                // finishing early and leaving the SIMD to the other.  With
                // two batches per chunk the second bit is the block's
                // progress: the last quarter of the chunks run two levels
                // lower, so that of two work-groups sharing a CU the one
                // ahead yields to the other near the end (3.8 % on the image
                // batch, whose CUs hold two work-groups each).
                set_issue_priority(RS / RB == 2 ? (rb == 0 ? 1 : 0) + (ch < nchunk - (nchunk + 3) / 4 ? 2 : 0)
                                                : 3 - rb * 4 / RS);
#pragma unroll
                for (int g = 0; g < NG; ++g) {
                    if (g + 1 < NG) read_group(g + 1);
#pragma unroll
                    for (int n = g * G; n < (g + 1) * G && n < NE; ++n) {
                        const int q = n / NCW, c = n % NCW;
                        e[q][c] = ex2(__builtin_fmaf(e[q][c], ns, ai[q] + bv[c]));
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
                if (RB == 1 && rb + 1 < RS) {  // the next row of this chunk (staged; unused if past the block)
#pragma unroll
                    for (int n = 0; n < PF; ++n) pre[n] = cbuf[(rb + 1) * D2P + 64 * n];
                }
#pragma unroll
                for (int q = 0; q < RB; ++q) p[q] = tree_sum<NCW>(e[q]);
                // Row updates of the batch, one row per 16-lane group (the
                // all-reduce's packed layout): each lane fetches its row's
                // potential and mass from the segment registers.
                const float rsv = allreduce_rows_packed<RB>(p);
                // Each lane's row of the packed layout: its potential and mass
                // (one row per batch: wave-uniform, read with readlane instead
                // of an LDS permute).
                const int src = rr0 + row_of_lane<RB>(lane);
                const float av = RB == 1 ? ai[0] : lane_get(a_seg, src);
                const float muv = RB == 1 ? uni(mu_seg, rr0) : lane_get(mu_seg, src);
                bool exact_any = false;
                if (STATS) {
                    rowerr += muv > 0.f ? fabsf(rsv - muv) : 0.f;
#pragma unroll
                    for (int q = 0; q < RB; ++q) {
                        const int rq = rel + q < nrows ? rb + q : rb;
                        __asm__ volatile("" ::: "memory");  // re-read the staged row
#pragma unroll
                        for (int c = 0; c < NCW; ++c)
                            losspart = __builtin_fmaf(e[q][c], cbuf[rq * D2P + 64 * c] * ns, losspart);
                        f[q] = 1.f;
                    }
                } else {
                    const bool inr = rsv >= kSumLo && rsv <= kSumHi;
                    const bool upd = muv > 0.f && inr;
                    const float an = av + (RB == 1 ? uni(lmu_seg, rr0) : lane_get(lmu_seg, src)) - lg2(rsv);
                    const float fv = upd ? ex2(an - av) : 0.f;
                    rowerr += upd ? fabsf(fv * rsv - muv) : 0.f;
                    exact_any = __any(muv > 0.f && !inr);
#pragma unroll
                    for (int q = 0; q < RB; ++q) f[q] = RB == 1 ? fv : uni(fv, lane_of_row<RB>(q));
                    // lane rr0 + q takes row q's new potential
                    const int dq = lane - rr0;
                    const float got =
                        RB == 1 ? (upd ? an : av) : lane_get(upd ? an : av, lane_of_row<RB>(dq >= 0 && dq < RB ? dq : 0));
                    a_out = dq >= 0 && dq < RB ? got : a_out;
                }
#pragma unroll
                for (int q = 0; q < RB; ++q)
#pragma unroll
                    for (int c = 0; c < NCW; ++c) colpart[c] = __builtin_fmaf(e[q][c], f[q], colpart[c]);
                if (!STATS && exact_any) {
#pragma unroll
                    for (int q = 0; q < RB; ++q) {
                        const float mui = uni(mu_seg, rr0 + q), rsq = uni(rsv, lane_of_row<RB>(q));
                        if (!(mui > 0.f) || (rsq >= kSumLo && rsq <= kSumHi)) continue;
                        // The shifted row sum left [2^-64, 2^64]: exact u-update
                        // of this row (max, then sum) from the staged cost, and
                        // its plan entries rebuilt from the new potential.
                        const float *crow = cbuf + (rb + q) * D2P;
                        float m = neg_inf();
#pragma unroll
                        for (int c = 0; c < NCW; ++c) m = fmaxf(m, __builtin_fmaf(crow[64 * c], ns, bv[c]));
                        m = wave_max(m);
                        // Re-read the staged row in each pass rather than keep
                        // it in registers (it would not fit beside bv and colpart).
                        __asm__ volatile("" ::: "memory");
                        float s2 = 0.f;
#pragma unroll
                        for (int c = 0; c < NCW; ++c) s2 += ex2(__builtin_fmaf(crow[64 * c], ns, bv[c]) - m);
                        s2 = wave_sum(s2);
                        const float an = uni(lmu_seg, rr0 + q) - (m + lg2(s2));
                        __asm__ volatile("" ::: "memory");
                        float rsum = 0.f;
#pragma unroll
                        for (int c = 0; c < NCW; ++c) {
                            const float v = ex2(__builtin_fmaf(crow[64 * c], ns, an + bv[c]));
                            rsum += v;
                            colpart[c] += v;
                        }
                        rowerr += lane == lane_of_row<RB>(q) ? fabsf(wave_sum(rsum) - mui) : 0.f;
                        a_out = lane == rr0 + q ? an : a_out;
                    }
                }
            }
            if (!STATS && !skip && (((rel + RB) & 63) == 0 || rel + RB >= nrows)) {
                const int i = i0 + (rel & ~63) + lane;
                if (i < i1) ab[i] = a_out;
            }
        }
    }
    if (skip) return;
#pragma unroll
    for (int c = 0; c < NCW; ++c) {
        const int j = lane + 64 * c;
        T.part[pidx(T, 0, r, b, j)] = colpart[c];  // 0 past d2
    }
    const float lw = STATS ? wave_sum(losspart) : 0.f;
    // rowerr is per 16-lane group (one batch row each): add the groups' totals
    // in a fixed order.
    float re = 0.f;
#pragma unroll
    for (int q = 0; q < RB; ++q) re += uni(rowerr, lane_of_row<RB>(q));
    if (lane == 0) {
        const int plane = STATS ? 2 : (k & 1);
        T.rowerr[((size_t)plane * T.R + r) * T.B + b] = re;
        if (STATS) T.lossp[(size_t)r * T.B + b] = lw;
    }
}

// Sweep for per-sample costs (each C_b read once per iteration: HBM bound).
//
// Work-group (row block r, problem b) of W wavefronts; wavefront w streams the
// rows i0 + w, i0 + w + W, ... of its block through its own LDS ring of NB
// rows, filled by direct 16-byte global->LDS loads, NB - 1 rows ahead of the
// row it computes: many bytes in flight per CU and no staging registers.  No
// barrier is needed inside the row loop (each ring belongs to one wavefront;
// its loads are waited for with vmcnt).  Lane l holds the columns
// j = 256 c + 4 l + q (c < NC4, q < 4), read from the ring as float4.
//
// The merge of the previous sweep's column partials (the v-update of this
// iteration, fixed order over row blocks) is done at the start by every
// work-group of the problem, for all columns, so no separate merge kernel
// runs between sweeps.  Its inputs are double-buffered by iteration parity:
// sweep k reads partials plane (k-1)&1, row potentials aplane(k-1), and writes
// plane k&1 and aplane(k) (an exact column logsumexp may read any row).  The
// same fixed-order sums give every work-group of the problem the same
// early-stop decision.
template <int NC4>
struct StreamShape {
    static constexpr int W = NC4 <= 8 ? 4 : 2;  // wavefronts per work-group
    static constexpr int NB = 4;                // ring depth (rows) per wavefront
};

__device__ __forceinline__ float *aplane(const TiledArgs &T, int k) { return (T.a2 && (k & 1)) ? T.a2 : T.a; }

// Exact logsumexp (base 2) over all rows of a_i + cl_ij for one column of a
// per-sample cost, reading the row potentials from a.
__device__ float col_lse_exact_from(const TiledArgs &T, const float *a, int b, int j) {
    const float *Cb = T.C + (size_t)b * T.d1 * T.d2;
    float m = neg_inf();
    for (int i = 0; i < T.d1; ++i) m = fmaxf(m, a[i] - T.s * Cb[(size_t)i * T.d2 + j]);
    if (m == neg_inf()) return m;
    float s = 0.f;
    for (int i = 0; i < T.d1; ++i) s += ex2(a[i] - T.s * Cb[(size_t)i * T.d2 + j] - m);
    return m + lg2(s);
}

template <int NC4, bool STATS>
__global__ __launch_bounds__(64 * StreamShape<NC4>::W) void sk_tiled_sweep_stream(TiledArgs T, int k) {
    constexpr int W = StreamShape<NC4>::W, NB = StreamShape<NC4>::NB;
    constexpr int NCW = 4 * NC4, D2S = 256 * NC4, NT = 64 * W;
    extern __shared__ float lds[];  // [D2S] merged potentials, then [W][NB][D2S] rings, then [W][D2S] partials
    __shared__ float red[2 * W];
    const int r = blockIdx.x, b = blockIdx.y;
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int d1 = T.d1, d2 = T.d2;
    const float *Cb = T.C + (size_t)b * d1 * d2;
    const int st = T.state[b];
    if (!STATS && st != 0) return;  // stopped after an earlier iteration (work-group uniform)
    const int K = STATS ? (st ? st : T.n_iter) : k;

    // ---- column potentials of this iteration (v-update folded in for k >= 2)
    float *bl = lds;  // [D2S], reused by the rings below
    const float *bsrc = T.bbuf + (size_t)(K & 1) * T.B * T.d2p + (size_t)b * T.d2p;
    if (!STATS && k >= 2) {
        const float *bold = T.bbuf + (size_t)((k - 1) & 1) * T.B * T.d2p + (size_t)b * T.d2p;
        float *bnew = T.bbuf + (size_t)(k & 1) * T.B * T.d2p + (size_t)b * T.d2p;
        const float *aprev = aplane(T, k - 1) + (size_t)b * d1;
        // Column sums of the plan after iteration k-1, fixed order over the row
        // blocks; the loads of QB row blocks x MPT columns are in flight together.
        constexpr int MPT = (D2S + NT - 1) / NT;        // columns per thread
        constexpr int QB = MPT >= 64 ? 1 : 64 / MPT;    // row blocks per batch of loads
        float cs[MPT];
#pragma unroll
        for (int m = 0; m < MPT; ++m) cs[m] = 0.f;
        for (int q0 = 0; q0 < T.R; q0 += QB) {
            float v[QB][MPT];
#pragma unroll
            for (int qq = 0; qq < QB; ++qq)
#pragma unroll
                for (int m = 0; m < MPT; ++m) {
                    const int j = threadIdx.x + NT * m;
                    v[qq][m] = (q0 + qq < T.R && j < d2) ? T.part[pidx(T, (k - 1) & 1, q0 + qq, b, j)] : 0.f;
                }
#pragma unroll
            for (int qq = 0; qq < QB; ++qq)
#pragma unroll
                for (int m = 0; m < MPT; ++m) cs[m] += v[qq][m];
        }
        float cerr = 0.f;
#pragma unroll
        for (int m = 0; m < MPT; ++m) {
            const int j = threadIdx.x + NT * m;
            float v = 0.f;
            if (j < d2) {
                const float nuj = T.nu[(size_t)b * d2 + j];
                cerr += fabsf(cs[m] - nuj);
                v = neg_inf();
                if (nuj > 0.f) {
                    if (cs[m] >= kSumLo && cs[m] <= kSumHi)
                        v = bold[j] + log2f(nuj) - lg2(cs[m]);
                    else
                        v = log2f(nuj) - col_lse_exact_from(T, aprev, b, j);
                }
                if (r == 0) bnew[j] = v;
            }
            if (j < D2S) bl[j] = v;  // 0 past d2
        }
        // Early stop on the marginal error of iterate k-1: its row part from
        // the previous sweep's row-block partials, its column part just summed.
        float re = 0.f;
        if (T.tol > 0.f)
            for (int q = 0; q < T.R; ++q) re += T.rowerr[((size_t)((k - 1) & 1) * T.R + q) * T.B + b];
        cerr = wave_sum(cerr);
        if (lane == 0) red[w] = cerr;
        __syncthreads();
        if (T.tol > 0.f) {
            float err = re;
#pragma unroll
            for (int q = 0; q < W; ++q) err += red[q];
            if (err <= T.tol) {
                if (r == 0 && threadIdx.x == 0) T.state[b] = k - 1;
                return;  // work-group uniform
            }
        }
    } else {
        for (int j = threadIdx.x; j < D2S; j += NT) bl[j] = bsrc[j];  // 0 past d2 (padded stride)
        __syncthreads();
    }
    float bv[NCW], colpart[NCW];
#pragma unroll
    for (int c = 0; c < NC4; ++c) {
        const f4v v = *reinterpret_cast<const f4v *>(bl + 256 * c + 4 * lane);
        bv[4 * c + 0] = v.x;
        bv[4 * c + 1] = v.y;
        bv[4 * c + 2] = v.z;
        bv[4 * c + 3] = v.w;
    }
#pragma unroll
    for (int c = 0; c < NCW; ++c) colpart[c] = 0.f;
    __syncthreads();  // the rings below reuse bl

    // ---- rows of this wavefront: i = i0 + w + W t
    float *ring = lds + (size_t)w * NB * D2S;
    if (d2 < D2S)  // padding columns of every ring slot: plan entry exactly 0
        for (int u = lane; u < NB * (D2S - d2); u += 64) ring[(u / (D2S - d2)) * D2S + d2 + u % (D2S - d2)] = kPadC;
    const int i0 = r * T.RBS, i1 = min(d1, i0 + T.RBS);
    const int nrow = i0 + w < i1 ? (i1 - i0 - w + W - 1) / W : 0;
    auto issue_row = [&](int t) {
        const float *src = Cb + (size_t)(i0 + w + W * t) * d2 + 4 * lane;
        float *slot = ring + (t % NB) * D2S;
#pragma unroll
        for (int c = 0; c < NC4; ++c)
            if (256 * c + 4 * lane < d2)
                __builtin_amdgcn_global_load_lds(src + 256 * c, (__attribute__((address_space(3))) void *)(slot + 256 * c),
                                                 16, 0, 0);
    };
    const float *a_in = aplane(T, STATS ? K : k - 1) + (size_t)b * d1;
    float *a_wr = aplane(T, k) + (size_t)b * d1;
    const float *mub = T.mu + (size_t)b * d1;
    // Row potentials and masses of 64 rows per register (lane = row t).
    float a_s[kSegs], mu_s[kSegs];
#pragma unroll
    for (int q = 0; q < kSegs; ++q) {
        const int t = 64 * q + lane;
        a_s[q] = t < nrow ? a_in[i0 + w + W * t] : neg_inf();
        mu_s[q] = t < nrow ? mub[i0 + w + W * t] : 0.f;
    }
    for (int t = 0; t < NB - 1 && t < nrow; ++t) issue_row(t);
    const float ns = -T.s;
    float rowerr = 0.f, losspart = 0.f;
    float a_seg = 0.f, mu_seg = 0.f, a_o = 0.f;
    for (int t = 0; t < nrow; ++t) {
        if ((t & 63) == 0) {
            const int sg = t >> 6;
            a_seg = a_s[0];
            mu_seg = mu_s[0];
#pragma unroll
            for (int q = 1; q < kSegs; ++q) {
                a_seg = sg == q ? a_s[q] : a_seg;
                mu_seg = sg == q ? mu_s[q] : mu_seg;
            }
            a_o = a_seg;
        }
        // Rows t+1 .. t+NB-1 may stay in flight (NC4 loads each); the last
        // rows of the wavefront wait for everything.
        if (t + NB - 1 < nrow) {
            issue_row(t + NB - 1);
            __asm__ volatile("s_waitcnt vmcnt(%0)" ::"n"(NC4 * (NB - 1)) : "memory");
        } else {
            __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
        }
        const float *slot = ring + (t % NB) * D2S + 4 * lane;
        float e[NCW];
#pragma unroll
        for (int c = 0; c < NC4; ++c) {
            const f4v v = *reinterpret_cast<const f4v *>(slot + 256 * c);
            e[4 * c + 0] = v.x;
            e[4 * c + 1] = v.y;
            e[4 * c + 2] = v.z;
            e[4 * c + 3] = v.w;
        }
        __builtin_amdgcn_sched_barrier(0);
        const int tt = t & 63;
        const float ai = uni(a_seg, tt), mui = uni(mu_seg, tt);
#pragma unroll
        for (int c = 0; c < NCW; ++c) e[c] = ex2(__builtin_fmaf(e[c], ns, ai + bv[c]));
        const float rs = uni(wave_sum(tree_sum<NCW>(e)), 0);
        float f = 0.f;
        bool exact = false;
        if (STATS) {
            if (mui > 0.f) rowerr += fabsf(rs - mui);
            __asm__ volatile("" ::: "memory");  // re-read the ring slot
#pragma unroll
            for (int c = 0; c < NC4; ++c) {
                const f4v v = *reinterpret_cast<const f4v *>(slot + 256 * c);
                losspart = __builtin_fmaf(e[4 * c + 0], v.x * ns, losspart);
                losspart = __builtin_fmaf(e[4 * c + 1], v.y * ns, losspart);
                losspart = __builtin_fmaf(e[4 * c + 2], v.z * ns, losspart);
                losspart = __builtin_fmaf(e[4 * c + 3], v.w * ns, losspart);
            }
            f = 1.f;
        } else if (mui > 0.f) {
            if (rs >= kSumLo && rs <= kSumHi) {
                const float an = ai + lg2(mui) - lg2(rs);
                f = ex2(an - ai);
                rowerr += fabsf(f * rs - mui);
                a_o = lane == tt ? an : a_o;
            } else {
                exact = true;
            }
        }
#pragma unroll
        for (int c = 0; c < NCW; ++c) colpart[c] = __builtin_fmaf(e[c], f, colpart[c]);
        if (!STATS && exact) {
            // Exact u-update of this row (max, then sum) from the ring slot.
            float m = neg_inf();
#pragma unroll
            for (int c = 0; c < NC4; ++c) {
                const f4v v = *reinterpret_cast<const f4v *>(slot + 256 * c);
                m = fmaxf(m, __builtin_fmaf(v.x, ns, bv[4 * c + 0]));
                m = fmaxf(m, __builtin_fmaf(v.y, ns, bv[4 * c + 1]));
                m = fmaxf(m, __builtin_fmaf(v.z, ns, bv[4 * c + 2]));
                m = fmaxf(m, __builtin_fmaf(v.w, ns, bv[4 * c + 3]));
            }
            m = wave_max(m);
            __asm__ volatile("" ::: "memory");
            float s2 = 0.f;
#pragma unroll
            for (int c = 0; c < NC4; ++c) {
                const f4v v = *reinterpret_cast<const f4v *>(slot + 256 * c);
                s2 += ex2(__builtin_fmaf(v.x, ns, bv[4 * c + 0]) - m);
                s2 += ex2(__builtin_fmaf(v.y, ns, bv[4 * c + 1]) - m);
                s2 += ex2(__builtin_fmaf(v.z, ns, bv[4 * c + 2]) - m);
                s2 += ex2(__builtin_fmaf(v.w, ns, bv[4 * c + 3]) - m);
            }
            s2 = wave_sum(s2);
            const float an = lg2(mui) - (m + lg2(s2));
            __asm__ volatile("" ::: "memory");
            float rsum = 0.f;
#pragma unroll
            for (int c = 0; c < NC4; ++c) {
                const f4v v = *reinterpret_cast<const f4v *>(slot + 256 * c);
                const float x[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float p = ex2(__builtin_fmaf(x[q], ns, an + bv[4 * c + q]));
                    rsum += p;
                    colpart[4 * c + q] += p;
                }
            }
            rowerr += fabsf(wave_sum(rsum) - mui);
            a_o = lane == tt ? an : a_o;
        }
        if (!STATS && (((t + 1) & 63) == 0 || t + 1 == nrow)) {
            const int tw = (t & ~63) + lane;
            if (tw < nrow) a_wr[i0 + w + W * tw] = a_o;
        }
    }

    // ---- combine the wavefronts' column partials (fixed order) and store
    __syncthreads();  // every ring is drained
    float *pl = lds;  // [W][D2S]
#pragma unroll
    for (int c = 0; c < NC4; ++c) {
        f4v v = {colpart[4 * c + 0], colpart[4 * c + 1], colpart[4 * c + 2], colpart[4 * c + 3]};
        *reinterpret_cast<f4v *>(pl + (size_t)w * D2S + 256 * c + 4 * lane) = v;
    }
    const float lw = STATS ? wave_sum(losspart) : 0.f;
    if (lane == 0) {
        red[w] = rowerr;
        red[W + w] = lw;
    }
    __syncthreads();
    const int plane = STATS ? 0 : (k & 1);
    for (int j = threadIdx.x; j < D2S; j += NT) {
        float s = 0.f;
#pragma unroll
        for (int q = 0; q < W; ++q) s += pl[q * D2S + j];
        T.part[pidx(T, plane, r, b, j)] = s;
    }
    if (threadIdx.x == 0) {
        float re = 0.f, lo = 0.f;
#pragma unroll
        for (int q = 0; q < W; ++q) {
            re += red[q];
            lo += red[W + q];
        }
        T.rowerr[((size_t)(STATS ? 2 : (k & 1)) * T.R + r) * T.B + b] = re;
        if (STATS) T.lossp[(size_t)r * T.B + b] = lo;
    }
}

// Outputs of the returned iterate: marginal error, E^0, natural-log potentials.
template <int NT>
__global__ __launch_bounds__(NT) void sk_tiled_final(TiledArgs T) {
    __shared__ float red[NT / 64];
    const int b = blockIdx.x;
    const int st = T.state[b];
    const int K = st ? st : T.n_iter;
    const float *bsrc = T.bbuf + (size_t)(K & 1) * T.B * T.d2p + (size_t)b * T.d2p;
    const size_t rstride = (size_t)T.B * T.d2p / 4;  // one row block, in f4v
    float colerr = 0.f;
    // Column sums of the returned plan over the row blocks (in block order,
    // 16 loads in flight), four consecutive columns per thread.
    for (int j0 = 4 * threadIdx.x; j0 < T.d2; j0 += 4 * NT) {
        const f4v *col = reinterpret_cast<const f4v *>(T.part + pidx(T, 0, 0, b, j0));
        f4v cs = {0.f, 0.f, 0.f, 0.f};
        for (int r0 = 0; r0 < T.R; r0 += 16) {
            f4v v[16];
#pragma unroll
            for (int q = 0; q < 16; ++q)
                v[q] = r0 + q < T.R ? col[(size_t)(r0 + q) * rstride] : f4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < 16; ++q) cs += v[q];
        }
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int j = j0 + c;
            if (j < T.d2) {
                colerr += fabsf(cs[c] - T.nu[(size_t)b * T.d2 + j]);
                T.beta_out[(size_t)b * T.d2 + j] = bsrc[j] * kLn2;
            }
        }
    }
    for (int i = threadIdx.x; i < T.d1; i += NT) {
        const size_t u = (size_t)b * T.d1 + i;
        T.alpha_out[u] = aplane(T, K)[u] * kLn2;
    }
    colerr = block_sum_n<NT>(colerr, red);
    if (threadIdx.x == 0) {
        float re = 0.f, lo = 0.f;
        for (int r = 0; r < T.R; ++r) {
            re += T.rowerr[((size_t)2 * T.R + r) * T.B + b];
            lo += T.lossp[(size_t)r * T.B + b];
        }
        T.loss_out[b] = -lo / T.s;
        T.merr_out[b] = re + colerr;
        T.iters_out[b] = K;
    }
}

// Cost kinds of the tiled regime: a shared cost, a per-sample cost, per-sample
// point clouds (cost computed on the fly).
constexpr int kKindShared = 0, kKindBatched = 1, kKindPoints = 2;
// Rows wider than one wavefront's registers hold (d2 > kTiledMaxD2), shared
// or per-sample cost: two passes per iteration (sk_wide_rows, sk_wide_cols).
constexpr int kKindWide = 3;
int tiled_kind(int d2, int c_batched) {
    return d2 > kTiledMaxD2 ? kKindWide : (c_batched ? kKindBatched : kKindShared);
}

// Which sweep serves a problem: the shared-cost sweep with W problems per
// work-group when C is shared and the batch fills at least four wavefronts,
// otherwise one problem per work-group.
int shared_width(int B, int kind) {
    if (kind != kKindShared) return 0;
    if (B >= 8) return 8;
    if (B >= 4) return 4;
    return 0;
}

// Row blocks.  One problem per work-group: enough work-groups for ~2048
// wavefronts, rows per block a multiple of the wavefronts per group.  Shared
// cost: ~256 (wide rows) or ~512 work-groups, the count of row blocks a
// multiple of 8 when the rows allow it so that a row block stays on one XCD.
bool stream_shape(int d2, int kind);
int stream_waves(int d2);

void row_blocks(int B, int d1, int d2, int kind, int *R, int *RBS) {
    const int W = shared_width(B, kind);
    int want, unit;
    if (stream_shape(d2, kind)) {
        // Streaming sweep: about one work-group per CU, and at most
        // 64 kSegs rows per wavefront (row potentials held in registers).
        want = (256 + B - 1) / (B > 0 ? B : 1);
        const int minR = (d1 + 64 * kSegs * stream_waves(d2) - 1) / (64 * kSegs * stream_waves(d2));
        want = want < minR ? minR : want;
        unit = 1;
    } else if (W) {
        const int G = (B + W - 1) / W;
        const int target = d2 > 1024 ? 256 : 512;
        want = (target + G - 1) / G;
        want = (want + 7) / 8 * 8;
        unit = 1;
    } else if (kind == kKindWide) {
        // Wide rows: ~512 row blocks over the batch, at most 64 per problem
        // (the merge reads R d2 partials per problem with one work-group).
        want = (512 + B - 1) / (B > 0 ? B : 1);
        want = want > 64 ? 64 : want;
        unit = kWaves;
    } else {
        want = (2048 / kWaves + B - 1) / (B > 0 ? B : 1);
        unit = kWaves;
    }
    const int maxR = (d1 + unit - 1) / unit;
    int r = want < 1 ? 1 : (want > maxR ? maxR : want);
    if (W) {
        const int minR = (d1 + 64 * kSegs - 1) / (64 * kSegs);  // the shared sweep holds <= 64 kSegs rows
        r = r < minR ? minR : r;
    }
    int rbs = (d1 + r - 1) / r;
    rbs = (rbs + unit - 1) / unit * unit;
    *RBS = rbs;
    *R = (d1 + rbs - 1) / rbs;
}

struct Layout {
    size_t bbuf, part, rowerr, lossp, state, order, a2, ctr, stopacc, total;
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Column registers per lane of the one-row-per-wavefront sweeps (64 lanes x
// NCW columns), and float4 groups per lane of the streaming sweep; the padded
// row stride of the workspace covers the widest sweep a shape may take.
int ncw_bucket(int d2) {
    const int n = (d2 + 63) / 64;
    return n <= 4 ? 4 : n <= 8 ? 8 : n <= 13 ? 13 : n <= 16 ? 16 : n <= 32 ? 32 : 64;
}
int nc4_bucket(int d2) {
    const int n = (d2 + 255) / 256;
    return n <= 1 ? 1 : n <= 2 ? 2 : n <= 4 ? 4 : n <= 8 ? 8 : 16;
}
bool stream_shape(int d2, int kind) { return kind == kKindBatched && d2 % 4 == 0; }
int stream_nc4(int d2) { return (d2 + 255) / 256; }
int stream_waves(int d2) { return stream_nc4(d2) <= 8 ? 4 : 2; }
int padded_width(int d2, int kind) {
    if (kind == kKindWide) return (d2 + 255) / 256 * 256;  // the column pass's work-group width
    int w = 64 * ncw_bucket(d2);
    if (stream_shape(d2, kind)) w = w > 256 * nc4_bucket(d2) ? w : 256 * nc4_bucket(d2);
    return w;
}

// Work-groups per problem of the merge after a sweep (4 columns per thread).
int merge_slices(int d2) { return (d2 + 4 * kMergeColsThreads - 1) / (4 * kMergeColsThreads); }

Layout layout(int B, int d1, int d2, int kind, int *R_out, int *RBS_out, int *JC_out) {
    int R, RBS;
    row_blocks(B, d1, d2, kind, &R, &RBS);
    const int JC = (d2 + kMergeThreads - 1) / kMergeThreads;
    const size_t d2p = padded_width(d2, kind);
    Layout L;
    size_t off = 0;
    L.bbuf = off;
    off = align256(off + sizeof(float) * 2 * (size_t)B * d2p);
    L.part = off;
    off = align256(off + sizeof(float) * 2 * (size_t)R * B * d2p);
    L.rowerr = off;
    off = align256(off + sizeof(float) * 3 * (size_t)R * B);
    L.lossp = off;
    off = align256(off + sizeof(float) * (size_t)R * B);
    L.state = off;  // state[B], sync[4]
    off = align256(off + sizeof(int32_t) * ((size_t)B + 4));
    L.order = off;  // order[B] then nlive
    if (kind == kKindShared) off = align256(off + sizeof(int32_t) * ((size_t)B + 1));
    L.a2 = off;
    if (stream_shape(d2, kind)) off = align256(off + sizeof(float) * (size_t)B * d1);
    L.ctr = off;
    if (kind == kKindPoints) off = align256(off + sizeof(float) * 4 * (size_t)B);
    L.stopacc = off;  // stopacc[B] (split merges only)
    if (merge_slices(d2) > 1) off = align256(off + sizeof(unsigned long long) * (size_t)B);
    L.total = off;
    if (R_out) *R_out = R;
    if (RBS_out) *RBS_out = RBS;
    if (JC_out) *JC_out = JC;
    return L;
}

// Raise a kernel's dynamic LDS limit when it needs more than the default 64 KB.
template <class Kernel>
hipError_t allow_lds(Kernel *kernel, size_t bytes) {
    if (bytes <= 64 * 1024) return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void *>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)bytes);
}

// The exact first v-update (a shared cost read once for 8 problems) and the
// closing kernel (1024 threads per problem above 1024 columns).
void launch_col_exact(const TiledArgs &T, hipStream_t st) {
    if (!T.c_batched && !T.X && T.B >= 8)
        hipLaunchKernelGGL(sk_tiled_col_exact<8>, dim3(T.JC, T.R, (T.B + 7) / 8), dim3(kMergeThreads), 0, st, T);
    else
        hipLaunchKernelGGL(sk_tiled_col_exact<1>, dim3(T.JC, T.R, T.B), dim3(kMergeThreads), 0, st, T);
}
// MS = ceil(d2 / 1024) work-groups of 256 threads per problem, plus the relist
// work-group of a compacted batch.
void launch_merge(const TiledArgs &T, int k, hipStream_t st) {
    hipLaunchKernelGGL(sk_tiled_merge_cols<kMergeColsThreads>, dim3(T.B + (T.order ? 1 : 0), T.MS),
                       dim3(kMergeColsThreads), 0, st, T, k);
}
void launch_final(const TiledArgs &T, hipStream_t st) {
    if (T.d2 > 1024)
        hipLaunchKernelGGL(sk_tiled_final<1024>, dim3(T.B), dim3(1024), 0, st, T);
    else
        hipLaunchKernelGGL(sk_tiled_final<256>, dim3(T.B), dim3(256), 0, st, T);
}

// Launch sequence of the wide rows: as run_sequence, each sweep being a rows
// pass and a columns pass.
hipError_t run_wide(const TiledArgs &T, hipStream_t st) {
    const dim3 blk(kThreads), rblk(64 * kWideRowWaves);
    const dim3 rg(T.R, T.B), cg(T.d2p / kThreads, T.R, T.B);
    hipLaunchKernelGGL(sk_tiled_init, dim3(512), blk, 0, st, T);
    if (T.n_iter > 0) {
        launch_col_exact(T, st);
        hipLaunchKernelGGL(sk_tiled_merge_exact, dim3(T.JC, T.B), dim3(kMergeThreads), 0, st, T);
        for (int k = 1; k <= T.n_iter; ++k) {
            hipLaunchKernelGGL(sk_wide_rows<false>, rg, rblk, 0, st, T, k);
            hipLaunchKernelGGL(sk_wide_cols<false>, cg, blk, 0, st, T, k);
            if (k < T.n_iter) launch_merge(T, k, st);
        }
    }
    hipLaunchKernelGGL(sk_wide_rows<true>, rg, rblk, 0, st, T, 0);
    hipLaunchKernelGGL(sk_wide_cols<true>, cg, blk, 0, st, T, 0);
    launch_final(T, st);
    return hipGetLastError();
}

// Launch sequence: init, exact first v-update (+ merge), n sweeps with a merge
// after each but the last, stats sweep, final.
template <class Sweep, class Stats>
hipError_t run_sequence(const TiledArgs &T, hipStream_t st, Sweep sweep, Stats stats) {
    const dim3 blk(kThreads);
    hipLaunchKernelGGL(sk_tiled_init, dim3(512), blk, 0, st, T);
    if (T.n_iter > 0) {
        launch_col_exact(T, st);
        const dim3 mblk(kMergeThreads);
        hipLaunchKernelGGL(sk_tiled_merge_exact, dim3(T.JC, T.B), mblk, 0, st, T);
        for (int k = 1; k <= T.n_iter; ++k) {
            sweep(k);
            if (k < T.n_iter) launch_merge(T, k, st);
        }
    }
    stats();
    launch_final(T, st);
    return hipGetLastError();
}

template <int NCW, bool BATCHED>
hipError_t run(const TiledArgs &T, hipStream_t st) {
    const size_t lds = sizeof(float) * kWaves * NCW * 64;
    const dim3 grid(T.R, T.B), blk(kThreads);
    return run_sequence(
        T, st, [&](int k) { hipLaunchKernelGGL((sk_tiled_sweep<NCW, false, BATCHED>), grid, blk, lds, st, T, k); },
        [&]() { hipLaunchKernelGGL((sk_tiled_sweep<NCW, true, BATCHED>), grid, blk, lds, st, T, 0); });
}

// Streaming sweep sequence: the merges are folded into the sweeps.
template <int NC4>
hipError_t run_stream(const TiledArgs &T, hipStream_t st) {
    constexpr int W = StreamShape<NC4>::W, NB = StreamShape<NC4>::NB;
    const size_t lds = sizeof(float) * W * NB * 256 * NC4;
    // Rings above 64 KB need the larger dynamic LDS limit (set on every call:
    // the library keeps no state of its own).
    hipError_t e = allow_lds(&sk_tiled_sweep_stream<NC4, false>, lds);
    if (e == hipSuccess) e = allow_lds(&sk_tiled_sweep_stream<NC4, true>, lds);
    if (e != hipSuccess) return e;
    const dim3 grid(T.R, T.B), blk(64 * W);
    hipLaunchKernelGGL(sk_tiled_init, dim3(512), dim3(kThreads), 0, st, T);
    if (T.n_iter > 0) {
        launch_col_exact(T, st);
        hipLaunchKernelGGL(sk_tiled_merge_exact, dim3(T.JC, T.B), dim3(kMergeThreads), 0, st, T);
        for (int k = 1; k <= T.n_iter; ++k)
            hipLaunchKernelGGL((sk_tiled_sweep_stream<NC4, false>), grid, blk, lds, st, T, k);
    }
    hipLaunchKernelGGL((sk_tiled_sweep_stream<NC4, true>), grid, blk, lds, st, T, 0);
    launch_final(T, st);
    return hipGetLastError();
}

// Rows per staged chunk and rows per reduction batch of the shared-cost sweep:
// wide rows keep fewer rows in flight (their plan entries live in registers
// until the row sum is known).
template <int NCW>
struct SharedShape {
    static constexpr int RB = NCW <= 16 ? 4 : (NCW <= 32 ? 2 : 1);
    static constexpr int RS = NCW <= 16 ? 8 : 4;
};

template <int NCW, int W, bool VEC4>
hipError_t run_shared(const TiledArgs &T, hipStream_t st) {
    constexpr int RS = SharedShape<NCW>::RS, RB = SharedShape<NCW>::RB;
    const size_t lds = sizeof(float) * 2 * RS * NCW * 64;
    // Chunk buffers above 64 KB need the larger dynamic LDS limit (set on
    // every call: the library keeps no state of its own).
    hipError_t e = allow_lds(&sk_tiled_sweep_shared<NCW, W, RS, RB, VEC4, false>, lds);
    if (e == hipSuccess) e = allow_lds(&sk_tiled_sweep_shared<NCW, W, RS, RB, VEC4, true>, lds);
    if (e != hipSuccess) return e;
    const dim3 grid(T.R, (T.B + W - 1) / W), blk(64 * W);
    return run_sequence(
        T, st,
        [&](int k) { hipLaunchKernelGGL((sk_tiled_sweep_shared<NCW, W, RS, RB, VEC4, false>), grid, blk, lds, st, T, k); },
        [&]() { hipLaunchKernelGGL((sk_tiled_sweep_shared<NCW, W, RS, RB, VEC4, true>), grid, blk, lds, st, T, 0); });
}

template <int NCW, int D>
hipError_t run_points(const TiledArgs &T, hipStream_t st) {
    const size_t lds = sizeof(float) * kWaves * NCW * 64;
    const dim3 grid(T.R, T.B), blk(kThreads);
    hipLaunchKernelGGL(sk_tiled_center, dim3(T.B), blk, 0, st, T);
    return run_sequence(
        T, st, [&](int k) { hipLaunchKernelGGL((sk_tiled_sweep_points<NCW, D, false>), grid, blk, lds, st, T, k); },
        [&]() { hipLaunchKernelGGL((sk_tiled_sweep_points<NCW, D, true>), grid, blk, lds, st, T, 0); });
}

template <int D>
hipError_t dispatch_points(const TiledArgs &T, int ncw, hipStream_t st) {
    if (ncw <= 4) return run_points<4, D>(T, st);
    if (ncw <= 8) return run_points<8, D>(T, st);
    if (ncw <= 13) return run_points<13, D>(T, st);
    if (ncw <= 16) return run_points<16, D>(T, st);
    return run_points<32, D>(T, st);
}

template <bool BATCHED>
hipError_t dispatch(const TiledArgs &T, int ncw, hipStream_t st) {
    if (ncw <= 4) return run<4, BATCHED>(T, st);
    if (ncw <= 8) return run<8, BATCHED>(T, st);
    if (ncw <= 13) return run<13, BATCHED>(T, st);
    if (ncw <= 16) return run<16, BATCHED>(T, st);
    if (ncw <= 32) return run<32, BATCHED>(T, st);
    return run<64, BATCHED>(T, st);
}

template <int W, bool VEC4>
hipError_t dispatch_shared(const TiledArgs &T, int ncw, hipStream_t st) {
    if (ncw <= 4) return run_shared<4, W, VEC4>(T, st);
    if (ncw <= 8) return run_shared<8, W, VEC4>(T, st);
    if (ncw <= 13) return run_shared<13, W, VEC4>(T, st);
    if (ncw <= 16) return run_shared<16, W, VEC4>(T, st);
    if (ncw <= 32) return run_shared<32, W, VEC4>(T, st);
    return run_shared<64, W, VEC4>(T, st);
}

// The row blocks of every chunk of a batch of B problems fit a grid dimension.
bool row_blocks_fit(int B, int d1, int d2, int kind) {
    int R, RBS;
    row_blocks(tiled_chunk(B), d1, d2, kind, &R, &RBS);
    if (R > 65535) return false;
    if (B > kTiledMaxBatch && B % kTiledMaxBatch) {
        row_blocks(B % kTiledMaxBatch, d1, d2, kind, &R, &RBS);
        if (R > 65535) return false;
    }
    return true;
}

}  // namespace

size_t tiled_workspace_bytes(int B, int d1, int d2, int c_batched) {
    return layout(tiled_chunk(B), d1, d2, tiled_kind(d2, c_batched), nullptr, nullptr, nullptr).total;
}

bool tiled_fits(int B, int d1, int d2, int c_batched) {
    return row_blocks_fit(B, d1, d2, tiled_kind(d2, c_batched));
}

bool tiled_points_fits(int B, int d1, int d2, int D) {
    return D >= 1 && D <= kPointsMaxD && d2 <= kPointsMaxD2 && row_blocks_fit(B, d1, d2, kKindPoints);
}

size_t tiled_points_workspace_bytes(int B, int d1, int d2) {
    return layout(tiled_chunk(B), d1, d2, kKindPoints, nullptr, nullptr, nullptr).total;
}

namespace {
// Workspace carving and scalar arguments common to every tiled launch.
TiledArgs tiled_args(const FwdArgs &a, int kind, void *ws, Layout *Lout) {
    TiledArgs T;
    int R, RBS, JC;
    const Layout L = layout(a.B, a.d1, a.d2, kind, &R, &RBS, &JC);
    *Lout = L;
    char *base = static_cast<char *>(ws);
    T.mu = a.mu;
    T.nu = a.nu;
    T.C = a.C;
    T.X = nullptr;
    T.Y = nullptr;
    T.ctr = nullptr;
    T.D = 0;
    T.rs = 0.f;
    T.a = a.alpha;
    T.a0 = a.alpha0;
    T.a2 = nullptr;
    T.bbuf = reinterpret_cast<float *>(base + L.bbuf);
    T.part = reinterpret_cast<float *>(base + L.part);
    T.rowerr = reinterpret_cast<float *>(base + L.rowerr);
    T.lossp = reinterpret_cast<float *>(base + L.lossp);
    T.state = reinterpret_cast<int32_t *>(base + L.state);
    T.sync = T.state + a.B;
    T.order = nullptr;
    T.nlive = nullptr;
    T.MS = merge_slices(a.d2);
    T.stopacc = T.MS > 1 ? reinterpret_cast<unsigned long long *>(base + L.stopacc) : nullptr;
    // Fixed point of the split merge's stop test: parts clamped to
    // fx_cap = 2^p >= max(8, 2 tol) at 2^(48 - p - ceil(log2 MS)) units per
    // unit of error, so that the sum of MS parts stays below 2^48 and never
    // carries into the count.
    int p = 3;
    while (p < 60 && std::ldexp(1.0, p) < 2.0 * (double)a.tol) ++p;
    int lms = 0;
    while ((1 << lms) < T.MS) ++lms;
    T.fx_cap = (float)std::ldexp(1.0, p);
    T.fx_scale = std::ldexp(1.0, kFxCountShift - 1 - p - lms);
    T.fx_tol = (double)a.tol * T.fx_scale;
    T.alpha_out = a.alpha;
    T.beta_out = a.beta;
    T.loss_out = a.loss;
    T.merr_out = a.marg_err;
    T.iters_out = a.iters;
    T.B = a.B;
    T.d1 = a.d1;
    T.d2 = a.d2;
    T.d2p = padded_width(a.d2, kind);
    T.R = R;
    T.RBS = RBS;
    T.JC = JC;
    T.n_iter = a.n_iter;
    T.c_batched = kind == kKindWide ? a.c_batched : kind != kKindShared;
    T.s = a.s;
    T.tol = a.tol;
    return T;
}
}  // namespace

namespace {
// One chunk (at most kTiledMaxBatch problems) of the points forward.
hipError_t launch_tiled_points_chunk(const FwdArgs &a, const float *X, const float *Y, int D, double rs, void *ws,
                                     hipStream_t st) {
    Layout L;
    TiledArgs T = tiled_args(a, kKindPoints, ws, &L);
    T.C = nullptr;
    T.X = X;
    T.Y = Y;
    T.ctr = reinterpret_cast<float *>(static_cast<char *>(ws) + L.ctr);
    T.D = D;
    T.rs = (float)rs;
    const int ncw = (a.d2 + 63) / 64;
    switch (D) {
        case 1: return dispatch_points<1>(T, ncw, st);
        case 2: return dispatch_points<2>(T, ncw, st);
        default: return dispatch_points<3>(T, ncw, st);
    }
}

// One chunk (at most kTiledMaxBatch problems) of the forward.
hipError_t launch_tiled_chunk(const FwdArgs &a, void *ws, hipStream_t st) {
    Layout L;
    const int kind = tiled_kind(a.d2, a.c_batched);
    TiledArgs T = tiled_args(a, kind, ws, &L);
    if (kind == kKindWide) return run_wide(T, st);
    char *base = static_cast<char *>(ws);
    const int ncw = (a.d2 + 63) / 64;
    const int W = shared_width(a.B, a.c_batched);
    // 16-byte global->LDS copies need 16-byte aligned cost rows.
    const bool vec4 = a.d2 % 4 == 0 && ((uintptr_t)a.C % 16) == 0;
    // Early stop with W problems per work-group: compact the running
    // problems before each sweep (unless sinkhorn_forward_select says not to).
    if (W && a.tol > 0.f && a.select != SK_SELECT_NO_COMPACTION) {
        T.order = reinterpret_cast<int32_t *>(base + L.order);
        T.nlive = T.order + a.B;
    }
    if (W == 8) return vec4 ? dispatch_shared<8, true>(T, ncw, st) : dispatch_shared<8, false>(T, ncw, st);
    if (W == 4) return vec4 ? dispatch_shared<4, true>(T, ncw, st) : dispatch_shared<4, false>(T, ncw, st);
    if (stream_shape(a.d2, a.c_batched ? kKindBatched : kKindShared) && ((uintptr_t)a.C % 16) == 0) {
        T.a2 = reinterpret_cast<float *>(base + L.a2);
        switch (stream_nc4(a.d2)) {
            case 1: return run_stream<1>(T, st);
            case 2: return run_stream<2>(T, st);
            case 3: return run_stream<3>(T, st);
            case 4: return run_stream<4>(T, st);
            case 5: return run_stream<5>(T, st);
            case 6: return run_stream<6>(T, st);
            case 7: return run_stream<7>(T, st);
            case 8: return run_stream<8>(T, st);
            case 9: return run_stream<9>(T, st);
            case 10: return run_stream<10>(T, st);
            case 11: return run_stream<11>(T, st);
            case 12: return run_stream<12>(T, st);
            case 13: return run_stream<13>(T, st);
            case 14: return run_stream<14>(T, st);
            case 15: return run_stream<15>(T, st);
            default: return run_stream<16>(T, st);
        }
    }
    if (a.c_batched) return dispatch<true>(T, ncw, st);
    return dispatch<false>(T, ncw, st);
}
}  // namespace

int tiled_describe(const FwdArgs &a, char *buf, size_t len) {
    const int B = tiled_chunk(a.B);
    const int kind = tiled_kind(a.d2, a.c_batched);
    int R, RBS, JC;
    const Layout L = layout(B, a.d1, a.d2, kind, &R, &RBS, &JC);
    const int W = shared_width(B, kind), ncw = ncw_bucket(a.d2);
    char sweep[192];
    bool merge = true;
    if (kind == kKindWide) {
        snprintf(sweep, sizeof sweep, "sk_wide_rows + sk_wide_cols (two passes over the cost per iteration)");
    } else if (W) {
        const int RB = ncw <= 16 ? 4 : (ncw <= 32 ? 2 : 1), RS = ncw <= 16 ? 8 : 4;
        snprintf(sweep, sizeof sweep,
                 "sk_tiled_sweep_shared<%d, %d, %d, %d> (%d problems per work-group, cost rows staged through LDS "
                 "%d at a time)",
                 ncw, W, RS, RB, W, RS);
    } else if (stream_shape(a.d2, kind)) {
        snprintf(sweep, sizeof sweep,
                 "sk_tiled_sweep_stream<%d> (the cost streamed once per iteration; "
                 "sk_tiled_sweep<%d> if its rows are not 16-byte aligned)",
                 stream_nc4(a.d2), ncw);
        merge = false;
    } else {
        snprintf(sweep, sizeof sweep, "sk_tiled_sweep<%d> (one problem per work-group)", ncw);
    }
    char mrg[128];
    if (merge)
        snprintf(mrg, sizeof mrg, "sk_tiled_merge_cols<%d> after each sweep (%d work-group%s per problem)",
                 kMergeColsThreads, merge_slices(a.d2), merge_slices(a.d2) == 1 ? "" : "s");
    else
        snprintf(mrg, sizeof mrg, "the merge folded into the next sweep");
    const bool compact = W && a.tol > 0.f && a.select != SK_SELECT_NO_COMPACTION;
    const int nchunk = (a.B + kTiledMaxBatch - 1) / kTiledMaxBatch;
    char chunks[64] = "";
    if (nchunk > 1) snprintf(chunks, sizeof chunks, "; %d chunks of at most %d problems", nchunk, kTiledMaxBatch);
    return snprintf(buf, len, "tiled: %s; %d row block%s of %d rows; %s%s%s; workspace %zu bytes", sweep, R,
                    R == 1 ? "" : "s", RBS, mrg, compact ? "; the running list rebuilt after stops" : "", chunks,
                    L.total);
}

hipError_t launch_tiled(const FwdArgs &a, void *ws, hipStream_t st) {
    return for_each_chunk(a.B, [&](int off, int n) { return launch_tiled_chunk(fwd_chunk(a, off, n), ws, st); });
}

// Per-sample clouds only (the on-the-fly sweep takes no shared clouds).
hipError_t launch_tiled_points(const FwdArgs &a, const float *X, const float *Y, int D, double rs, void *ws,
                               hipStream_t st) {
    return for_each_chunk(a.B, [&](int off, int n) {
        return launch_tiled_points_chunk(fwd_chunk(a, off, n), X + (size_t)off * a.d1 * D,
                                         Y + (size_t)off * a.d2 * D, D, rs, ws, st);
    });
}

}  // namespace sk
