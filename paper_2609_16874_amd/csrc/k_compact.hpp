// k_compact.hpp -- the participating set S of Eq6 as a compact pixel list.
//
// One launch before the vote in frames of three launches (frames above
// kFusedMaxPixels pixels, grids above 32 x 32 bins; the vote launch lists
// the pixels itself otherwise).  Workgroup s of the grid owns the
// pixel range [s R, (s + 1) R) (R a multiple of 8192) and writes the indices
// of its participating pixels, in raster order, to its slice list[s R ..]
// and their number to counts[s]; every lane tests 8 consecutive foreground
// values against the threshold, a wave prefix sum gives the slots, and each
// step's entries are gathered in LDS and stored as one contiguous run.  No
// atomics: the consumers concatenate the slices through the prefix sum of
// the counts (slice_prefix / ListCursor).  The non-participating pixels get
// their final outputs here: label 0 and, if a score map is requested,
// score 0.  The launch also clears the next frame's vote histograms (this
// frame's were cleared before it).  The vote and assignment launches then
// stream equal shares of the list in full tiles, so their work does not
// depend on where in the frame the foreground lies.
#pragma once

#include "cpe_common.hpp"

namespace cpe {

constexpr int kCompactThreads = 1024;
constexpr int kCompactPer = 8;                                   // pixels per lane
constexpr int kCompactSpan = kCompactThreads * kCompactPer;      // pixels per workgroup and step
// Largest frame: every slice end (at most one slice, 2^23 pixels, past the
// frame) and every tile offset then stays below 2^31, so pixel and list
// positions are int32 throughout.
constexpr int64_t kMaxPixels = (1LL << 31) - (1LL << 23);

// Pixels per slice for a frame of npix pixels, and the number of slices.
__host__ __device__ constexpr int slice_pixels(int64_t npix)
{
    const int64_t steps = (npix + (int64_t)kMaxSlices * kCompactSpan - 1) / ((int64_t)kMaxSlices * kCompactSpan);
    return (int)(steps * kCompactSpan);
}
__host__ __device__ constexpr int slice_count(int64_t npix)
{
    const int64_t r = slice_pixels(npix);
    return (int)((npix + r - 1) / r);
}

// VEC: the foreground plane is 16-byte aligned, so a lane's 8 values are one
// (fp16) or two (fp32) vector loads.
template <typename T, bool VEC>
__global__ __launch_bounds__(kCompactThreads) void k_compact(const T *__restrict__ fg, int32_t npix, float fg_thr,
                                                             int32_t *__restrict__ list, int32_t *__restrict__ counts,
                                                             int32_t *__restrict__ labels, float *__restrict__ score,
                                                             unsigned long long *__restrict__ hclear, int32_t nclear)
{
    for (int i = blockIdx.x * kCompactThreads + threadIdx.x; i < nclear; i += gridDim.x * kCompactThreads)
        hclear[i] = 0ull;
    __shared__ int s_wave[kCompactThreads / 64];
    __shared__ int32_t s_out[kCompactSpan];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int R = slice_pixels(npix);
    const int begin = blockIdx.x * R;
    const int end = (int)min((int64_t)begin + R, (int64_t)npix);
    int32_t *out = list + begin;
    int base = 0;                                      // entries of the slice so far
    const bool score_vec = score && ((uintptr_t)score & 15u) == 0;

    for (int q0 = begin; q0 < end; q0 += kCompactSpan) {
        const int p0 = q0 + tid * kCompactPer;
        float v[kCompactPer];
        if (VEC && p0 + kCompactPer <= end) {
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
            for (int i = 0; i < kCompactPer; i++) v[i] = p0 + i < end ? load_scalar<T>(fg + p0 + i) : 0.0f;
        }
        uint32_t m = 0, valid = 0;
#pragma unroll
        for (int i = 0; i < kCompactPer; i++) {
            const bool in = p0 + i < end;
            valid |= (in ? 1u : 0u) << i;
            m |= (in && v[i] > fg_thr ? 1u : 0u) << i;   // a NaN never exceeds the threshold
        }
        const int c = __popc(m);
        const int incl = wave_incl_sum(c);
        if (lane == 63) s_wave[wv] = incl;
        __syncthreads();
        int off = incl - c, tot = 0;
#pragma unroll
        for (int w = 0; w < kCompactThreads / 64; w++) {
            const int n = s_wave[w];
            off += w < wv ? n : 0;
            tot += n;
        }
#pragma unroll
        for (int i = 0; i < kCompactPer; i++)
            if ((m >> i) & 1u) s_out[off++] = p0 + i;
        __syncthreads();                                   // s_wave and s_out are rewritten in the next step
        for (int i = tid; i < tot; i += kCompactThreads) out[base + i] = s_out[i];
        base += tot;

        // outputs of the pixels outside S
        const uint32_t bg = valid & ~m;
        if (bg == 0xffu) {
            const int4 z = {0, 0, 0, 0};
            reinterpret_cast<int4 *>(labels + p0)[0] = z;
            reinterpret_cast<int4 *>(labels + p0)[1] = z;
            if (score_vec) {
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
    if (tid == 0) counts[blockIdx.x] = base;
}

namespace {   // one private copy per translation unit that launches it

// Zero n words (the vote histograms of a frame without a compaction launch).
__global__ __launch_bounds__(256) __attribute__((unused)) void k_clear_u64(unsigned long long *__restrict__ p, int32_t n)
{
    for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0ull;
}

}  // namespace

// Exclusive prefix sums s_pref[0 .. nslices] of the slice counts (LDS),
// s_pref[nslices] = |S|, by the first wave: slice_load issues the loads
// (lane l holds slices 4 l .. 4 l + 3), slice_scan writes the sums.  Split
// so that the caller can issue its other loads in between; the caller's
// barrier publishes s_pref.
struct SliceLoad {
    int c[kMaxSlices / 64];
};
__device__ __forceinline__ void slice_load(const int32_t *__restrict__ counts, int nslices, SliceLoad &sl)
{
    const int tid = threadIdx.x;
    if (tid < 64) {
#pragma unroll
        for (int k = 0; k < kMaxSlices / 64; k++) {
            const int s = 4 * tid + k;
            sl.c[k] = s < nslices ? counts[s] : 0;
        }
    }
}
__device__ __forceinline__ void slice_scan(const SliceLoad &sl, int nslices, int *s_pref)
{
    const int tid = threadIdx.x;
    if (tid < 64) {
        int sum = 0;
#pragma unroll
        for (int k = 0; k < kMaxSlices / 64; k++) sum += sl.c[k];
        const int incl = wave_incl_sum(sum);
        int run = incl - sum;
#pragma unroll
        for (int k = 0; k < kMaxSlices / 64; k++) {
            const int s = 4 * tid + k;
            if (s <= nslices) s_pref[s] = run;
            run += sl.c[k];
        }
        // the lanes' slices end at kMaxSlices - 1: the total for nslices == kMaxSlices
        if (tid == 63) s_pref[nslices] = incl;
    }
}

// The concatenated slices seen by one lane whose positions never decrease:
// entry i is list[s R + i - pref[s]] for the slice s with pref[s] <= i <
// pref[s + 1].  start() locates the slice of a wave-uniform position i0 (no
// larger than any position the lane asks for) by counting the prefix sums
// <= i0 with ballots; pixel() then steps forward.  Without a list (every
// pixel participates) entry i is pixel i.
struct ListCursor {
    const int32_t *list;
    const int *pref;          // LDS, pref[0 .. nslices]
    int R, s, lo, hi;

    // Called by every lane of the wave; i0 < pref[nslices] unless the lane
    // asks for no entry.
    __device__ __forceinline__ void start(const int32_t *list_, const int *pref_, int nslices, int R_, int i0)
    {
        list = list_;
        pref = pref_;
        R = R_;
        if (!list) return;
        const int lane = threadIdx.x & 63;
        int cnt = 0;              // slices s < nslices with pref[s] <= i0 (pref is non-decreasing)
#pragma unroll
        for (int k = 0; k < kMaxSlices / 64; k++) {
            const int q = 64 * k + lane;
            cnt += __popcll(__ballot(q < nslices && pref[q] <= i0));
        }
        s = cnt > 0 ? cnt - 1 : 0;
        lo = pref[s];
        hi = pref[s + 1];
    }
    __device__ __forceinline__ int pixel(int i)
    {
        if (!list) return i;
        while (i >= hi) {
            s++;
            lo = hi;
            hi = pref[s + 1];
        }
        return list[(size_t)s * R + (i - lo)];
    }
};

}  // namespace cpe
