// masks.hip -- binary instance masks M^_m (Eq8) from a label map.
//
// masks[m][p] = (labels[p] == first + m + 1) as one byte.  The work is one
// read of the labels per group of kMaskGroup masks and count * H * W bytes of
// mask stores, so it is bound by the HBM write rate.  When H * W is a
// multiple of 16 every mask starts 16-byte aligned and a thread handles 16
// consecutive pixels: one 64-byte label load, then one 16-byte store per
// mask, consecutive threads writing consecutive pieces of a mask.  The
// stores are non-temporal (the masks are not read back by this library).
// Other frame sizes take a one-pixel-per-thread kernel.
#include <hip/hip_runtime.h>

#include "cpe_decoder.hpp"

namespace cpe {
namespace {

constexpr int kMaskGroup = 8;     // masks per thread (grid.y = groups)
constexpr int kMaskThreads = 256;

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4m __attribute__((ext_vector_type(4)));

// byte j of the result = (v[j] == want)
__device__ __forceinline__ uint32_t eq_bytes(i32x4 v, int32_t want)
{
    return (uint32_t)(v.x == want) | ((uint32_t)(v.y == want) << 8) | ((uint32_t)(v.z == want) << 16) |
           ((uint32_t)(v.w == want) << 24);
}

__global__ __launch_bounds__(kMaskThreads) void k_masks16(const int32_t *__restrict__ labels, int64_t npix,
                                                         int32_t first, int32_t count, uint8_t *__restrict__ masks)
{
    const int64_t t = (int64_t)blockIdx.x * kMaskThreads + threadIdx.x;   // 16-pixel piece
    if (t * 16 >= npix) return;
    const i32x4 *src = reinterpret_cast<const i32x4 *>(labels + t * 16);
    const i32x4 l0 = src[0], l1 = src[1], l2 = src[2], l3 = src[3];
    const int m0 = (int)blockIdx.y * kMaskGroup;
    const int m1 = min(m0 + kMaskGroup, (int)count);
    for (int m = m0; m < m1; m++) {
        const int32_t want = first + m + 1;
        const u32x4m w = {eq_bytes(l0, want), eq_bytes(l1, want), eq_bytes(l2, want), eq_bytes(l3, want)};
        __builtin_nontemporal_store(w, reinterpret_cast<u32x4m *>(masks + (int64_t)m * npix + t * 16));
    }
}

__global__ __launch_bounds__(kMaskThreads) void k_masks1(const int32_t *__restrict__ labels, int64_t npix,
                                                        int32_t first, int32_t count, uint8_t *__restrict__ masks)
{
    const int64_t p = (int64_t)blockIdx.x * kMaskThreads + threadIdx.x;
    if (p >= npix) return;
    const int32_t l = labels[p];
    const int m0 = (int)blockIdx.y * kMaskGroup;
    const int m1 = min(m0 + kMaskGroup, (int)count);
    for (int m = m0; m < m1; m++) masks[(int64_t)m * npix + p] = (uint8_t)(l == first + m + 1);
}

}  // namespace

cpe_status launch_masks(hipStream_t stream, const int32_t *labels, int64_t npix, int32_t first, int32_t count,
                        uint8_t *masks)
{
    const unsigned groups = (unsigned)((count + kMaskGroup - 1) / kMaskGroup);
    if (npix % 16 == 0) {
        const int64_t pieces = npix / 16;
        const dim3 grid((unsigned)((pieces + kMaskThreads - 1) / kMaskThreads), groups);
        hipLaunchKernelGGL(k_masks16, grid, dim3(kMaskThreads), 0, stream, labels, npix, first, count, masks);
    } else {
        const dim3 grid((unsigned)((npix + kMaskThreads - 1) / kMaskThreads), groups);
        hipLaunchKernelGGL(k_masks1, grid, dim3(kMaskThreads), 0, stream, labels, npix, first, count, masks);
    }
    return hipGetLastError() == hipSuccess ? CPE_OK : CPE_ERR_HIP;
}

}  // namespace cpe
