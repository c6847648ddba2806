// sk_resident.hip -- small problems (max(d1, d2) <= 128) entirely on-chip in
// the log domain: one work-group of two wavefronts per problem runs every
// iteration, the convergence check and the loss with the scaled cost in
// VGPRs (the iteration itself is in sk_resident_log.h).  HBM is touched only
// to load the inputs and store the outputs.  Used when the caller asks for
// the log domain alone and for n_iter = 0; the plain-form kernels run the same
// body in place for the problems they cannot keep in range.
#include "sk_resident_log.h"

namespace sk {
namespace {

template <int N>
__global__ __launch_bounds__(128) __attribute__((amdgpu_waves_per_eu(2))) void sk_resident_log_kernel(FwdArgs A) {
    __shared__ __attribute__((aligned(16))) float pool[kLogLdsFloats];
    resident_log_body<N>(A, pool);
}

template <int N>
hipError_t launch_n(const FwdArgs &a, hipStream_t st) {
    hipLaunchKernelGGL((sk_resident_log_kernel<N>), dim3(a.B), dim3(128), 0, st, a);
    return hipGetLastError();
}

}  // namespace

bool resident_fits(int d1, int d2) { return d1 <= kResidentMaxD && d2 <= kResidentMaxD; }

hipError_t launch_resident(const FwdArgs &a, hipStream_t st) {
    const int nb = ((a.d1 > a.d2 ? a.d1 : a.d2) + 7) / 8;
    if (nb <= 2) return launch_n<2>(a, st);
    if (nb <= 4) return launch_n<4>(a, st);
    if (nb <= 8) return launch_n<8>(a, st);
    if (nb <= 13) return launch_n<13>(a, st);
    return launch_n<16>(a, st);
}

}  // namespace sk
