// k_generic.hpp -- the assignment kernel for bin grids above 32 x 32 (up to
// 128 x 128).
//
// One thread per foreground pixel computes the per-axis squared distances to
// every palette entry with packed 16-bit dot products (Eq4/Eq10), turns them
// into distances sqrt_cr(fl32(S)), assigns the pixel to the candidate with
// the smallest exact distance sum (Eq7, lowest index on ties), writes its
// label and score and counts it.  The candidates come from the stand-alone
// peak kernel (k_peaks.hpp); the votes of every grid are cast by the
// matrix-core kernel of k_mfma.hpp, and grids up to 32 x 32 also take its
// matrix-core assignment.
#pragma once

#include "cpe_common.hpp"
#include "k_compact.hpp"
#include "k_peaks.hpp"

namespace cpe {

// Load one axis block (2F channels) of a pixel and pack it as F int16 pairs.
template <typename T, int F, int ALIGN>
__device__ __forceinline__ void load_block(const T *blk, int32_t (&pk)[F])
{
    if constexpr (sizeof(T) == 4) {
        const float *p = reinterpret_cast<const float *>(__builtin_assume_aligned(blk, ALIGN));
#pragma unroll
        for (int k = 0; k < F; k++) pk[k] = pack2(to_fixed(p[2 * k]), to_fixed(p[2 * k + 1]));
    } else {
        const uint32_t *p = reinterpret_cast<const uint32_t *>(__builtin_assume_aligned(blk, ALIGN));
#pragma unroll
        for (int k = 0; k < F; k++) {
            uint32_t w = p[k];
            pk[k] = pack2(to_fixed(half_bits_to_float(w & 0xffffu)), to_fixed(half_bits_to_float(w >> 16)));
        }
    }
}

template <int F>
__device__ __forceinline__ int32_t dot_pk(const int32_t (&x)[F], const int32_t *p)
{
    int32_t acc = 0;
#pragma unroll
    for (int k = 0; k < F; k++)
        acc = __builtin_amdgcn_sdot2(__builtin_bit_cast(v2s, x[k]), __builtin_bit_cast(v2s, p[k]), acc, false);
    return acc;
}

// Alignment of a pixel's axis blocks in the layout with D = 4F channels; a
// longer encoding (D > 4F) has 16-byte aligned rows and y blocks, which
// satisfies the same bounds.
template <typename T, int F>
struct PixelLayout {
    static constexpr int kRowBytes = 4 * F * (int)sizeof(T);
    static constexpr int kAlignX = (kRowBytes % 16 == 0) ? 16 : 4;
    static constexpr int kAlignY = (kAlignX == 16 && (2 * F * (int)sizeof(T)) % 16 == 0) ? 16 : 4;
};

// ---------------------------------------------------------------------------
// S4 + S5: assignment, label write-out, counts
// ---------------------------------------------------------------------------
// LDS bytes of k_assign_generic before its per-pixel distances: palettes,
// norms, counts, candidate slots, the slots' bins, the candidate rows'
// first candidates and the slice prefix.
__host__ __device__ constexpr size_t generic_assign_fixed(int Bw, int Bh, int F, int kmax)
{
    return ((size_t)(Bw + Bh) * F * 4 + (size_t)(Bw + Bh) * 4 + (size_t)kCountCap * 4 + (size_t)kmax * 4 +
            2 * (size_t)kMaxBins * 2 + 2 * (size_t)kMaxBins / 8 + 2 * (size_t)kMaxBins * 2 +
            (size_t)(kMaxBins + 1) * 4 + (size_t)(kMaxSlices + 1) * 4 + 64 + 15) &
           ~(size_t)15;
}

// One thread per participating pixel (entries of the compact list written by
// k_compact, or every pixel without a foreground channel).  The candidate
// columns and rows are numbered in ascending order (slots); each thread
// computes its pixel's distances to the slots' palette entries only, then
// scans the candidate rows in order: the candidates are in bin order, so
// each row's candidates are a contiguous run of indices, and within a row
// the smallest sum r_y + r_x belongs to the smallest r_x (the binary64 sum
// of two binary32 values is exact, hence strictly increasing in r_x).  The
// first row with the smallest sum, and in it the first candidate with that
// row's smallest r_x, is the lowest index attaining the minimum (Eq7).
template <typename T, int F>
__global__ __launch_bounds__(256) void k_assign_generic(const T *__restrict__ emb, int32_t dstride, int32_t yoff,
                                                const int32_t *__restrict__ list, const int32_t *__restrict__ counts,
                                                int32_t nslices, int32_t slice_px, int32_t npix,
                                                double tau4096, Tables tb, int32_t Bw, int32_t Bh,
                                                const int32_t *__restrict__ peaks, const int32_t *__restrict__ kinfo,
                                                cpe_centroid *__restrict__ cents, int32_t *__restrict__ labels,
                                                float *__restrict__ score_map)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int TP = blockDim.x;
    const int tid = threadIdx.x;
    const int kmax = max_peaks(Bw, Bh);
    int32_t *s_px = reinterpret_cast<int32_t *>(smem);
    int32_t *s_py = s_px + Bw * F;
    uint32_t *s_nx = reinterpret_cast<uint32_t *>(s_py + Bh * F);
    uint32_t *s_ny = s_nx + Bw;
    int32_t *s_cnt = reinterpret_cast<int32_t *>(s_ny + Bh);     // [kCountCap]
    int32_t *s_pk = s_cnt + kCountCap;                           // [kmax] column slot | row slot << 16
    uint16_t *s_slot = reinterpret_cast<uint16_t *>(s_pk + kmax); // [2][kMaxBins] bin -> slot
    uint32_t *s_mask = reinterpret_cast<uint32_t *>(s_slot + 2 * kMaxBins);   // [2][kMaxBins / 32]
    uint16_t *s_sbin = reinterpret_cast<uint16_t *>(s_mask + 2 * kMaxBins / 32);  // [2][kMaxBins] slot -> bin
    int *s_rfirst = reinterpret_cast<int *>(s_sbin + 2 * kMaxBins);          // [kMaxBins + 1] first candidate of a row slot
    int *s_pref = s_rfirst + kMaxBins + 1;                                   // [kMaxSlices + 1]
    int *s_ns = s_pref + kMaxSlices + 1;                                     // [2] candidate columns, rows
    float *s_r = reinterpret_cast<float *>(smem + generic_assign_fixed(Bw, Bh, F, kmax));  // [column slots][TP]

    const int Kc = kinfo[0];
    const int ncnt = Kc < kCountCap ? Kc : kCountCap;
    SliceLoad sl;
    if (list) slice_load(counts, nslices, sl);
    for (int i = tid; i < Bw * F; i += TP) s_px[i] = tb.pal_x[i];
    for (int i = tid; i < Bh * F; i += TP) s_py[i] = tb.pal_y[i];
    for (int i = tid; i < Bw; i += TP) s_nx[i] = tb.n2_x[i];
    for (int i = tid; i < Bh; i += TP) s_ny[i] = tb.n2_y[i];
    for (int i = tid; i < ncnt; i += TP) s_cnt[i] = 0;
    for (int i = tid; i < 2 * kMaxBins / 32; i += TP) s_mask[i] = 0u;
    if (list) slice_scan(sl, nslices, s_pref);
    __syncthreads();
    // candidate columns and rows as bit masks, then their slots in ascending order
    for (int k = tid; k < Kc; k += TP) {
        const int32_t pk = peaks[k], a = pk & 0xffff, b = pk >> 16;
        atomicOr(&s_mask[a >> 5], 1u << (a & 31));
        atomicOr(&s_mask[kMaxBins / 32 + (b >> 5)], 1u << (b & 31));
    }
    __syncthreads();
    for (int i = tid; i < 2 * kMaxBins; i += TP) {
        const int ax = i / kMaxBins, bin = i % kMaxBins;
        const uint32_t *m = s_mask + ax * (kMaxBins / 32);
        int below = __popc(m[bin >> 5] & ((1u << (bin & 31)) - 1u));
        for (int w = 0; w < (bin >> 5); w++) below += __popc(m[w]);
        s_slot[i] = (uint16_t)below;
        if ((m[bin >> 5] >> (bin & 31)) & 1u) s_sbin[ax * kMaxBins + below] = (uint16_t)bin;
        if (bin == kMaxBins - 1) s_ns[ax] = below + (int)((m[bin >> 5] >> 31) & 1u);
    }
    __syncthreads();
    for (int k = tid; k < Kc; k += TP) {
        const int32_t pk = peaks[k];
        const int rs = s_slot[kMaxBins + (pk >> 16)];
        s_pk[k] = (int32_t)s_slot[pk & 0xffff] | (rs << 16);
        // candidates are in bin order: a row slot's candidates are a run of indices
        if (k == 0 || (peaks[k - 1] >> 16) != (pk >> 16)) s_rfirst[rs] = k;
    }
    if (tid == 0) s_rfirst[s_ns[1]] = Kc;
    __syncthreads();
    const int ncol = s_ns[0], nrow = s_ns[1];

    using L = PixelLayout<T, F>;
    const int n = list ? s_pref[nslices] : npix;
    const int stride = gridDim.x * TP;
    const int first = blockIdx.x * TP + (tid & ~63);             // the wave's first entry
    ListCursor cur;
    cur.start(list, s_pref, nslices, slice_px, first < n ? first : 0);
    for (int i = blockIdx.x * TP + tid; i - tid + (tid & ~63) < n; i += stride) {
        if (i < n) {
            const int32_t pp = cur.pixel(i);
            if (Kc == 0) {
                labels[pp] = 0;
                if (score_map) score_map[pp] = 0.0f;
                continue;
            }
            const T *row = emb + (size_t)pp * dstride;
            int32_t xk[F], yk[F];
            load_block<T, F, L::kAlignX>(row, xk);
            load_block<T, F, L::kAlignY>(row + yoff, yk);
            const uint32_t nX = (uint32_t)dot_pk<F>(xk, xk);
            const uint32_t nY = (uint32_t)dot_pk<F>(yk, yk);
            // distances of the candidate columns (the column slots' bins)
            for (int s = 0; s < ncol; s++) {
                const int a = s_sbin[s];
                s_r[s * TP + tid] = sqrt_cr((float)axis_s(nX, s_nx[a], dot_pk<F>(xk, s_px + a * F)));
            }
            // Eq7 by rows: the smallest column distance of each row's run (the
            // binary32 bits of distances >= 0 order like their values), plus the
            // row's distance (computed here, once per row), summed exactly in
            // binary64; strict < keeps the first row
            const uint32_t *s_rb = reinterpret_cast<const uint32_t *>(s_r);
            double bd = __builtin_inf();
            int brow = 0;
            uint32_t bm = 0u;
            for (int r = 0, k = 0; r < nrow; r++) {
                const int kend = s_rfirst[r + 1];
                uint32_t m = 0xffffffffu;
                for (; k < kend; k++) m = min(m, s_rb[(s_pk[k] & 0xffff) * TP + tid]);
                const int b = s_sbin[kMaxBins + r];
                const float ry = sqrt_cr((float)axis_s(nY, s_ny[b], dot_pk<F>(yk, s_py + b * F)));
                const double d = (double)__uint_as_float(m) + (double)ry;
                if (d < bd) {
                    bd = d;
                    brow = r;
                    bm = m;
                }
            }
            // the first candidate of that row with its smallest column distance
            int best = s_rfirst[brow];
            const int blast = s_rfirst[brow + 1] - 1;
            while (best < blast && s_rb[(s_pk[best] & 0xffff) * TP + tid] != bm) best++;
            if (bd < tau4096) {     // Eq8
                labels[pp] = best + 1;
                if (score_map) score_map[pp] = expf(-(float)(bd * 0x1p-12));
                if (best < kCountCap)
                    atomicAdd(s_cnt + best, 1);
                else
                    atomicAdd(&cents[best].npix, 1);
            } else {
                labels[pp] = 0;
                if (score_map) score_map[pp] = 0.0f;
            }
        }
    }
    __syncthreads();
    for (int i = tid; i < ncnt; i += TP)
        if (s_cnt[i]) atomicAdd(&cents[i].npix, s_cnt[i]);
}


}  // namespace cpe
