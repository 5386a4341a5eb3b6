// k_compact.hpp -- the participating set S of Eq6 as a compact pixel list.
//
// One launch per frame before the vote: every lane tests 8 consecutive
// foreground values against the threshold, a wave prefix sum and one
// global reservation per workgroup give each participating pixel its slot,
// and its index is written to `list` (raster order within a workgroup's
// 2048 pixels; workgroups in the order of their reservations).  The
// non-participating pixels get their final outputs here: label 0 and, if a
// score map is requested, score 0.  The vote and assignment launches then
// stream equal shares of the list in full tiles, so their work does not
// depend on where in the frame the foreground lies.
//
// `count` must be 0 before the launch; afterwards it holds |S|.
#pragma once

#include "cpe_common.hpp"

namespace cpe {

constexpr int kCompactThreads = 256;
constexpr int kCompactPer = 8;                                   // pixels per lane
constexpr int kCompactSpan = kCompactThreads * kCompactPer;      // pixels per workgroup

// VEC: the foreground plane is 16-byte aligned (fp16) / 32-byte aligned
// (fp32), so a lane's 8 values are one or two vector loads.
template <typename T, bool VEC>
__global__ __launch_bounds__(kCompactThreads) void k_compact(const T *__restrict__ fg, int32_t npix, float fg_thr,
                                                             int32_t *__restrict__ list, int32_t *__restrict__ count,
                                                             int32_t *__restrict__ labels, float *__restrict__ score)
{
    __shared__ int s_wave[kCompactThreads / 64];
    __shared__ int s_base;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int p0 = (blockIdx.x * kCompactThreads + tid) * kCompactPer;

    float v[kCompactPer];
    if (VEC && p0 + kCompactPer <= npix) {
        if constexpr (sizeof(T) == 2) {
            const uint4 w = *reinterpret_cast<const uint4 *>(fg + p0);
            const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int i = 0; i < 4; i++) {
                v[2 * i] = half_bits_to_float(ww[i] & 0xffffu);
                v[2 * i + 1] = half_bits_to_float(ww[i] >> 16);
            }
        } else {
            const float4 a = *reinterpret_cast<const float4 *>(fg + p0);
            const float4 b = *reinterpret_cast<const float4 *>(fg + p0 + 4);
            v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
            v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < kCompactPer; i++) v[i] = p0 + i < npix ? load_scalar<T>(fg + p0 + i) : 0.0f;
    }
    uint32_t m = 0, valid = 0;
#pragma unroll
    for (int i = 0; i < kCompactPer; i++) {
        const bool in = p0 + i < npix;
        valid |= (in ? 1u : 0u) << i;
        m |= (in && v[i] > fg_thr ? 1u : 0u) << i;   // a NaN never exceeds the threshold
    }
    const int c = __popc(m);
    int incl = c;                                      // inclusive prefix over the wave
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int t = __shfl_up(incl, d);
        if (lane >= d) incl += t;
    }
    if (lane == 63) s_wave[wv] = incl;
    __syncthreads();
    if (tid == 0) {
        int tot = 0;
#pragma unroll
        for (int w = 0; w < kCompactThreads / 64; w++) tot += s_wave[w];
        s_base = tot ? atomicAdd(count, tot) : 0;
    }
    __syncthreads();
    int off = s_base + incl - c;
#pragma unroll
    for (int w = 0; w < kCompactThreads / 64; w++) off += w < wv ? s_wave[w] : 0;
#pragma unroll
    for (int i = 0; i < kCompactPer; i++)
        if ((m >> i) & 1u) list[off++] = p0 + i;

    // outputs of the pixels outside S
    const uint32_t bg = valid & ~m;
    if (bg == 0xffu) {
        const int4 z = {0, 0, 0, 0};
        reinterpret_cast<int4 *>(labels + p0)[0] = z;
        reinterpret_cast<int4 *>(labels + p0)[1] = z;
        if (score && ((uintptr_t)score & 15u) == 0) {
            const float4 zf = {0.0f, 0.0f, 0.0f, 0.0f};
            reinterpret_cast<float4 *>(score + p0)[0] = zf;
            reinterpret_cast<float4 *>(score + p0)[1] = zf;
        } else if (score) {
#pragma unroll
            for (int i = 0; i < kCompactPer; i++) score[p0 + i] = 0.0f;
        }
    } else if (bg) {
#pragma unroll
        for (int i = 0; i < kCompactPer; i++)
            if ((bg >> i) & 1u) {
                labels[p0 + i] = 0;
                if (score) score[p0 + i] = 0.0f;
            }
    }
}

}  // namespace cpe
