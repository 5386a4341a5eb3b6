// cpe_common.hpp -- constants, device tables and arithmetic helpers shared by
// the decoder's kernels.  Every helper implements one step of the fixed-point
// contract stated in include/cpe_decode.h.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "cpe_decode.h"

namespace cpe {

constexpr int kWMant = 8;             // weight bucket: top 8 mantissa bits of fl32(S+1)
constexpr int kWKeys = 32 << kWMant;  // 8192 weight buckets (32 binades)
constexpr int kReplicas = 4;          // replicated global histograms (spread of the atomics)
constexpr int kMaxF = 16;             // harmonics per axis
constexpr int kMaxBins = 128;
constexpr int kCountCap = 1024;       // centroids whose pixel counts are privatised in LDS
constexpr int kMfmaBins = 32;         // bin grids up to 32 x 32 take the matrix-core path
constexpr int kPopKinds = 3;          // int8 palette operand kinds per axis (AxisOp in k_mfma.hpp)
constexpr int kMaxBinBlocks = (kMaxBins + kMfmaBins - 1) / kMfmaBins;   // blocks of 32 bins per axis
constexpr int kMaxSlices = 256;       // workgroups of the compaction (slices of the pixel list)
constexpr int64_t kFusedMaxPixels = 1LL << 21;   // frames the vote launch compacts itself (two launches)
constexpr int kFusedMaxSeg = 8192;               // listed pixels per workgroup of that launch (LDS)
constexpr int kFusedSteps = kFusedMaxSeg / 64;   // its 64-pixel steps per workgroup
static_assert(kFusedSteps <= 128, "two steps per lane in the folded compaction's prefix sum");

typedef short v2s __attribute__((ext_vector_type(2)));

// Device-resident constants built once by cpe_decode_create.
struct Tables {
    const int32_t *pal_x;     // [Bw][F]: harmonic k = (sin | cos << 16), int16 each, x4096
    const int32_t *pal_y;     // [Bh][F]
    const uint32_t *n2_x;     // [Bw] sum of squared palette entries
    const uint32_t *n2_y;     // [Bh]
    const uint16_t *wt;       // [kWKeys] 2^15 e^-d per 8-bit bucket (bucket order)
    const float *cx;          // [Bw] bin centres (pixels)
    const float *cy;          // [Bh]
    // matrix-core path (bins <= 32)
    const uint32_t *np1_x;    // [kMaxBinBlocks * 32] |P_w[bin]|^2 + 1 (1 for padded bins)
    const uint32_t *np1_y;    // [kMaxBinBlocks * 32]
    const uint32_t *pop;      // [axis][block][kind][64 lanes][4 words]: the int8 palette operand of
                              //   lane l (bin 32 block + (l & 31), K slots 16 (l >> 5) .. + 15);
                              //   see k_mfma.hpp
    const uint32_t *wt_pk;    // [kWKeys] weight as two fp16 limbs (q & 255) | (q >> 8) << 16,
                              //          at LDS position ((e + 31) & 31) * 256 + t
};

// Input to fixed point: rint(4096 clamp(v, -1.5, 1.5)), the input on the
// palette's grid of 1/4096; a NaN clamps to -1.5 (fmaxf/fminf return the
// non-NaN operand).
__device__ __forceinline__ int32_t to_fixed(float v)
{
    const float c = fminf(fmaxf(v, -1.5f), 1.5f);
    return (int32_t)rintf(c * 4096.0f);
}

// The Eq4 distance in units of 1/4096: the correctly rounded binary32 square
// root of x = fl32(S) (0 or at least 1).  The hardware square root is within
// one unit in the last place; the neighbours s - u and s + u of its result s
// are tested against x with exact residuals: x - s (s - u) is a multiple of
// u^2 and differs from x - (s - u/2)^2 by u^2/4, so its sign is that of x
// against the lower midpoint, and likewise x - s (s + u) for the upper
// midpoint (no midpoint is a root of a binary32 value).  For x = 0 both
// tests fail and 0 is returned.
__device__ __forceinline__ float sqrt_cr(float x)
{
    const float s = __builtin_amdgcn_sqrtf(x);
    const float sd = __uint_as_float(__float_as_uint(s) - 1u);
    const float su = __uint_as_float(__float_as_uint(s) + 1u);
    const float rd = __builtin_fmaf(-sd, s, x);
    const float ru = __builtin_fmaf(-su, s, x);
    float r = rd <= 0.0f ? sd : s;
    r = ru > 0.0f ? su : r;
    return r;
}

// min of two binary64 values that are never NaN (one instruction; the
// library's min also canonicalises its operands).
__device__ __forceinline__ double min_f64(double a, double b)
{
    double r;
    asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

__device__ __forceinline__ int32_t pack2(int32_t lo, int32_t hi)
{
    return (int32_t)(((uint32_t)lo & 0xffffu) | ((uint32_t)hi << 16));
}

__device__ __forceinline__ float half_bits_to_float(uint32_t bits)
{
    return (float)__builtin_bit_cast(_Float16, (uint16_t)bits);
}

template <typename T> __device__ __forceinline__ float load_scalar(const T *p);
template <> __device__ __forceinline__ float load_scalar<float>(const float *p) { return *p; }
template <> __device__ __forceinline__ float load_scalar<_Float16>(const _Float16 *p) { return (float)*p; }

// Foreground value of pixel p.  Without a foreground channel (fg == nullptr,
// a uniform branch) every pixel participates: +inf exceeds any finite
// threshold.
template <typename T>
__device__ __forceinline__ float fg_value(const T *fg, int64_t p)
{
    return fg ? load_scalar<T>(fg + p) : __builtin_huge_valf();
}

// S = |X|^2 + |P|^2 - 2 X.P is exact modulo 2^32 and lies in [0, 2^32).
__device__ __forceinline__ uint32_t axis_s(uint32_t nX, uint32_t nP, int32_t dot)
{
    return nX + nP - 2u * (uint32_t)dot;
}

// m-bit distance bucket: exponent and top m mantissa bits of fl32(S+1).
template <int M>
__device__ __forceinline__ int dist_key(uint32_t s)
{
    const uint32_t bits = __float_as_uint((float)(s + 1u));
    return (int)(bits >> (23 - M)) - (127 << M);
}

// Inclusive prefix sum of x over the 64 lanes of a wave with DPP moves:
// shifts by 1, 2, 4, 8 within each row of 16 lanes, then the last lane of
// row 0 added to row 1 (and of row 2 to row 3), then the last lane of row 1
// added to rows 2 and 3.  Every lane must be active.
__device__ __forceinline__ int wave_incl_sum(int x)
{
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true);   // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true);   // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, true);   // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, true);   // row_shr:8
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15 into rows 1, 3
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31 into rows 2, 3
    return x;
}

__device__ __forceinline__ int lane_prefix(unsigned long long mask)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
}

}  // namespace cpe
