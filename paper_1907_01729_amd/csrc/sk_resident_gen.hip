// sk_resident_gen.hip -- any cost (shared by the batch or one per problem)
// with max(d1, d2) <= 128: the general plain-form kernel, one work-group of
// two wavefronts per problem (the iteration itself is in sk_resident_gen.h).
#include "sk_resident_log.h"

namespace sk {
namespace {

template <int N>
__global__ __launch_bounds__(128) __attribute__((amdgpu_waves_per_eu(2))) void sk_resident_gen_kernel(FwdArgs A) {
    __shared__ __attribute__((aligned(16))) float pool[kGenLdsFloats > kLogLdsFloats ? kGenLdsFloats : kLogLdsFloats];
    if (resident_gen_body<N>(A, pool)) hand_over_to_log<N>(A, pool);
}

template <int N>
hipError_t launch_n(const FwdArgs &a, hipStream_t st) {
    hipLaunchKernelGGL((sk_resident_gen_kernel<N>), dim3(a.B), dim3(128), 0, st, a);
    return hipGetLastError();
}

}  // namespace

bool launch_resident_gen(const FwdArgs &a, hipStream_t st, hipError_t *err) {
    if (a.n_iter <= 0) return false;
    const int nb = ((a.d1 > a.d2 ? a.d1 : a.d2) + 7) / 8;
    if (nb <= 2) *err = launch_n<2>(a, st);
    else if (nb <= 4) *err = launch_n<4>(a, st);
    else if (nb <= 8) *err = launch_n<8>(a, st);
    else if (nb <= 13) *err = launch_n<13>(a, st);
    else if (nb <= 16) *err = launch_n<16>(a, st);
    else return false;
    return true;
}

}  // namespace sk
