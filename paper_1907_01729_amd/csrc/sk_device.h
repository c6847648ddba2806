// sk_device.h -- device helpers shared by the gfx950 Sinkhorn kernels.
//
// Base-2 arithmetic throughout: potentials are kept as a = alpha*log2(e),
// b = beta*log2(e) and the cost as cl = -C*log2(e)/lambda, so every plan
// entry P_ij = exp(alpha_i + beta_j - C_ij/lambda) is a single v_exp_f32 of
// (a_i + b_j + cl_ij).  Logarithms of sums use v_log_f32 (base 2).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sk {

constexpr float kLog2e = 1.44269504088896340736f;
constexpr float kLn2 = 0.69314718055994530942f;
// A sum of exponentials shifted by the previous potentials is trusted when it
// lies in [2^-64, 2^64]: each term it may have lost to underflow (< 2^-126) is
// then below 2^-62 of the sum.  Outside that range the exact
// max-then-sum logsumexp is used instead.
constexpr float kSumLo = 5.42101086242752217e-20f;  // 2^-64
constexpr float kSumHi = 1.84467440737095516e19f;   // 2^64

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }

// s_setprio with a level computed at run time or only after unrolling (0..3).
__device__ __forceinline__ void set_issue_priority(int p) {
    if (p <= 0)
        __builtin_amdgcn_s_setprio(0);
    else if (p == 1)
        __builtin_amdgcn_s_setprio(1);
    else if (p == 2)
        __builtin_amdgcn_s_setprio(2);
    else
        __builtin_amdgcn_s_setprio(3);
}

// Issue-priority base of iteration k of n in a kernel that runs a whole
// problem's iteration in one launch: 2 before the last eighth of the
// iterations, 0 in it.  Two wavefronts of different problems share a SIMD and
// have the same work; at equal priority the older one issues first, finishes
// early and leaves the younger alone on the SIMD for the rest.  A wavefront
// that reaches the last eighth first drops below the other until it gets
// there too, so both end nearly together.  Phases of an iteration add 0 or 1.
// (Measured on the log-domain kernel: 3 % on 1024 problems of 100 x 100; the
// plain-form kernels, whose iterations are short, ran slower with it.)
__device__ __forceinline__ int progress_priority(int k, int n) { return k < n - n / 8 ? 2 : 0; }

// v_exp_f32 / v_log_f32: base-2 hardware transcendentals.
__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float lg2(float x) { return __builtin_amdgcn_logf(x); }

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// DPP controls used below.
constexpr int kQuadXor1 = 0xB1;      // quad_perm [1,0,3,2]   : lane ^ 1
constexpr int kQuadXor2 = 0x4E;      // quad_perm [2,3,0,1]   : lane ^ 2
constexpr int kHalfMirror = 0x141;   // row_half_mirror       : lane -> 7 - lane (within 8)
constexpr int kRowRor8 = 0x128;      // row_ror:8             : lane ^ 8 (within 16)

// All-reduce over the 8 consecutive lanes 8p..8p+7.  Every butterfly step adds
// two values in both orders' IEEE-equal way, so all 8 lanes end bit-identical.
__device__ __forceinline__ float sum_q(float v) {
    v += dpp<kQuadXor1>(v);
    v += dpp<kQuadXor2>(v);
    v += dpp<kHalfMirror>(v);
    return v;
}
__device__ __forceinline__ float max_q(float v) {
    v = fmaxf(v, dpp<kQuadXor1>(v));
    v = fmaxf(v, dpp<kQuadXor2>(v));
    v = fmaxf(v, dpp<kHalfMirror>(v));
    return v;
}
// Exchange across DPP rows with gfx950's v_permlane{16,32}_swap: with both
// operands = x, lane l gets the pair (x[l & ~16], x[l | 16]) (resp. 32), the
// same ordered pair on lane l and lane l ^ 16 (resp. 32), so one swap plus one
// add is an all-reduce step whose result is bit-identical on both lanes.
struct LanePair {
    float lo, hi;
};
__device__ __forceinline__ LanePair swap16(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return {__uint_as_float(r[0]), __uint_as_float(r[1])};
}
__device__ __forceinline__ LanePair swap32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return {__uint_as_float(r[0]), __uint_as_float(r[1])};
}

// All-reduce over the 8 lanes q, q+8, ..., q+56 (same lane & 7).
__device__ __forceinline__ float sum_p(float v) {
    v += dpp<kRowRor8>(v);
    LanePair a = swap16(v);
    v = a.lo + a.hi;
    LanePair b = swap32(v);
    return b.lo + b.hi;
}
__device__ __forceinline__ float max_p(float v) {
    v = fmaxf(v, dpp<kRowRor8>(v));
    LanePair a = swap16(v);
    v = fmaxf(a.lo, a.hi);
    LanePair b = swap32(v);
    return fmaxf(b.lo, b.hi);
}
// Whole-wavefront all-reduce (bit-identical on every lane).
__device__ __forceinline__ float wave_sum(float v) { return sum_p(sum_q(v)); }
__device__ __forceinline__ float wave_max(float v) { return max_p(max_q(v)); }

// Pairwise (tree) sum of a register array: log-depth dependency chain instead
// of a serial one, so that few wavefronts per SIMD still keep the VALU busy.
template <int N>
__device__ __forceinline__ float tree_sum(const float *v) {
    if constexpr (N == 1) {
        return v[0];
    } else {
        constexpr int L = N / 2;
        return tree_sum<L>(v) + tree_sum<N - L>(v + L);
    }
}

// ---- register-resident products: lane (p, q) of a wavefront, p = lane & 7,
// q = lane >> 3, holds cells [p + 8r][q + 8t] of an 8-row by 8-column block
// grid ----

// Row totals through LDS: lane (p, q) holds partial sums x[r] of its rows
// p + 8r (r < NR) over its column blocks; lane (p, r), r < NR, gets the total
// of row r, summed over q in a fixed order (other lanes a copy of row
// NR - 1).  tb: the wavefront's own scratch of 8 x 72 floats, entry (p, r, q)
// at p * 72 + r * 8 + q, so that the 64 writes of one r fall on 64 distinct
// banks and each total is two 16-byte reads.  The LDS operations of one
// wavefront complete in order, so no barrier is needed, and the next call's
// writes cannot overtake this call's reads.
constexpr int kRowTotalsFloats = 8 * 72;
template <int NR>
__device__ __forceinline__ float row_totals(const float (&x)[NR], float *tb, int p, int q) {
    static_assert(NR <= 8, "one row per lane q");
    float *mine = tb + p * 72 + q;
#pragma unroll
    for (int r = 0; r < NR; ++r) mine[r * 8] = x[r];
    __builtin_amdgcn_wave_barrier();
    const float *row = tb + p * 72 + (q < NR ? q : NR - 1) * 8;
    const float4 a = *reinterpret_cast<const float4 *>(row);
    const float4 b = *reinterpret_cast<const float4 *>(row + 4);
    __builtin_amdgcn_wave_barrier();
    return ((a.x + a.y) + (a.z + a.w)) + ((b.x + b.y) + (b.z + b.w));
}

// Column partials of a two-wavefront work-group: lane (p, q) of wavefront w
// writes its partial sum of column q + 8t to cp[partial_at(w, p, q, t)]
// (64 consecutive floats per t); after a barrier column_total(cp, c) sums
// column c's 16 partials (8 lanes p, 2 wavefronts) in a fixed order.
// cp holds kColumnPartialsFloats floats (columns < 128), 16-byte aligned.
constexpr int kColumnPartialsFloats = 2 * 128 * 8;
__device__ __forceinline__ int partial_at(int w, int p, int q, int t) { return (w * 128 + q + 8 * t) * 8 + p; }
__device__ __forceinline__ float column_total(const float *cp, int c) {
    const float4 *v0 = reinterpret_cast<const float4 *>(cp + c * 8);
    const float4 *v1 = reinterpret_cast<const float4 *>(cp + (128 + c) * 8);
    const float4 a = v0[0], b = v0[1], e = v1[0], f = v1[1];
    return (((a.x + a.y) + (a.z + a.w)) + ((b.x + b.y) + (b.z + b.w))) +
           (((e.x + e.y) + (e.z + e.w)) + ((f.x + f.y) + (f.z + f.w)));
}

}  // namespace sk
