// selfcheck.hip -- exhaustive check of the library's correctly rounded
// square root (sqrt_cr, cpe_common.hpp) over its whole input domain: every
// binary32 value x = fl32(S) of an integer S in [0, 2^32), i.e. 0 and every
// float in [1, 2^32), against the compiler's IEEE sqrtf.
#include <hip/hip_runtime.h>

#include "cpe_common.hpp"

namespace {

__global__ void k_clear_u64(unsigned long long *p) { *p = 0ull; }

__global__ void k_check_sqrt(unsigned long long *__restrict__ mismatches)
{
    constexpr uint32_t kN = 32u << 23;          // floats in [1, 2^32)
    unsigned long long bad = 0;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i <= kN; i += gridDim.x * blockDim.x) {
        const float x = i == kN ? 0.0f : __uint_as_float(0x3F800000u + i);
        bad += __float_as_uint(cpe::sqrt_cr(x)) != __float_as_uint(sqrtf(x));
    }
    if (bad) atomicAdd(mismatches, bad);
}

}  // namespace

extern "C" cpe_status cpe_check_sqrt(hipStream_t stream, unsigned long long *mismatches)
{
    if (!mismatches || ((uintptr_t)mismatches & 7u)) return CPE_ERR_INVALID_ARG;
    hipLaunchKernelGGL(k_clear_u64, dim3(1), dim3(1), 0, stream, mismatches);
    hipLaunchKernelGGL(k_check_sqrt, dim3(4096), dim3(256), 0, stream, mismatches);
    return hipGetLastError() == hipSuccess ? CPE_OK : CPE_ERR_HIP;
}
